// dps_device.h -- device-side helpers shared by the libdps kernels (gfx950).
//
// Residual addressing (Sec. IV-B "Shared Region"): the residual bytes of a
// weight form a logical stream in row-major element order, cut into chunks
// of C = 2^log2c bytes; chunk c lives in pool slot slots[c].  Every access the
// kernels make is a 16-byte vector at a 16-byte-aligned logical offset, and
// C >= 16, so a vector never straddles two chunks.
//
// Merge (Sec. IV-C "Overall concept"; nestings of Sec. IV-B "Persistent
// Region"): with the E5M2 nesting an FP16 word is (upper byte << 8) |
// residual byte; with the E4M3 nesting the upper byte holds the sign, the
// four low exponent bits and three mantissa bits, the exponent MSB is zero
// and the residual byte's seven low bits are the rest of the mantissa.  The
// kernels build FP16 operands in registers with one byte permute per two
// weights (plus three bit operations for E4M3).  The fast-mode weight is the
// FP16 word with its residual bits cleared -- E5M2(hi), or E4M3(hi) * 2^-8 --
// so a fast-mode product is bit-identical to a full-mode product whose
// residual bytes are all zero.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dps {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int32_t i32x8 __attribute__((ext_vector_type(8)));

enum { MODE_FULL = 0, MODE_FAST = 1 };
enum { ENC_E5M2 = 0, ENC_E4M3 = 1 };

// Kernel-argument form of a residual descriptor.
struct ResidualView {
    const uint8_t *pool;
    const int32_t *slots;
    int64_t n_pool_slots;  // pool_bytes >> log2c
    int64_t n_chunks;
    int32_t log2c;
};

// Physical byte offset of logical residual byte li, or -1 when its chunk is
// beyond the table or its slot is outside the pool.  Branch-free: the table
// read is always issued (entry 0 stands in for an out-of-range chunk;
// n_chunks >= 1 whenever a residual is read).
__device__ __forceinline__ int64_t residual_offset(const ResidualView &r, int64_t li)
{
    const int64_t c = li >> r.log2c;
    const bool cin = c >= 0 && c < r.n_chunks;
    const int64_t s = r.slots[cin ? c : 0];
    const bool sin = cin && s >= 0 && s < r.n_pool_slots;
    return sin ? ((s << r.log2c) | (li & ((int64_t(1) << r.log2c) - 1))) : -1;
}

// Addressing for one contiguous logical range [lbegin, lend) that spans at
// most two chunks (the range is no longer than one chunk).  Logical byte li
// of the range lives at pool + delta[li >= bnd] + li.
struct RangeResidual {
    int64_t delta0, delta1;
    int64_t bnd;
    bool ok0, ok1;
};

__device__ __forceinline__ void slot_delta(const ResidualView &r, int64_t c, int64_t &delta,
                                           bool &ok)
{
    ok = false;
    delta = 0;
    if (c >= 0 && c < r.n_chunks) {
        const int64_t s = r.slots[c];
        if (s >= 0 && s < r.n_pool_slots) {
            ok = true;
            delta = (s - c) << r.log2c;
        }
    }
}

__device__ __forceinline__ RangeResidual range_residual(const ResidualView &r, int64_t lbegin,
                                                        int64_t lend)
{
    RangeResidual rr;
    const int64_t c0 = lbegin >> r.log2c;
    const int64_t c1 = (lend - 1) >> r.log2c;
    slot_delta(r, c0, rr.delta0, rr.ok0);
    slot_delta(r, c1, rr.delta1, rr.ok1);
    rr.bnd = c1 << r.log2c;
    return rr;
}

__device__ __forceinline__ u32x4 load16(const void *p)
{
    return *reinterpret_cast<const u32x4 *>(p);
}

// 16 residual bytes at logical offset li: two-chunk fast path.
__device__ __forceinline__ u32x4 load_lo_range(const ResidualView &r, const RangeResidual &rr,
                                               int64_t li)
{
    const bool second = li >= rr.bnd;
    const bool ok = second ? rr.ok1 : rr.ok0;
    const int64_t d = second ? rr.delta1 : rr.delta0;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (ok)
        v = load16(r.pool + (d + li));
    return v;
}

// 16 residual bytes at logical offset li: per-vector table lookup.
__device__ __forceinline__ u32x4 load_lo_lookup(const ResidualView &r, int64_t li)
{
    const int64_t off = residual_offset(r, li);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (off >= 0)
        v = load16(r.pool + off);
    return v;
}

// Two E4M3-nested words t = (hi << 8 | lo) per 16-bit half -> FP16 words:
// the sign stays at bit 15, the seven bits below it move down one place
// (the exponent MSB becomes 0) and the residual keeps its seven low bits.
__device__ __forceinline__ uint32_t e4m3_words(uint32_t t)
{
    return (t & 0x807F807Fu) | ((t >> 1) & 0x3F803F80u);
}

// Four FP16 words from four upper bytes (hi4) and four residual bytes (lo4):
// first word j = hi byte j << 8 | lo byte j (v_perm_b32 picks bytes 0-3 from
// its second source and 4-7 from its first), then the E4M3 field move.
template <int ENC>
__device__ __forceinline__ u32x2 merge4(uint32_t hi4, uint32_t lo4)
{
    u32x2 t = {__builtin_amdgcn_perm(hi4, lo4, 0x05010400u),
               __builtin_amdgcn_perm(hi4, lo4, 0x07030602u)};
    if (ENC == ENC_E4M3) {
        t.x = e4m3_words(t.x);
        t.y = e4m3_words(t.y);
    }
    return t;
}

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

// merge4 as the linear kernels take it.  E4M3: gfx950's packed E4M3 -> FP16
// conversion with scale 2^-8 gives the word with a zero residual (see fast4),
// and the residual's seven low bits go into the low byte of each word: three
// instructions per two words against the bit moves' four (on MI355X the
// E4M3 full-mode decode step 0.97x the time, gate+up at 256 tokens 0.92x).
// Exact on every upper byte but the two E4M3 NaN codes, which no layer that
// dps_select_enc admits for E4M3 holds; the standalone merge keeps merge4.
template <int ENC>
__device__ __forceinline__ u32x2 merge4_lin(uint32_t hi4, uint32_t lo4)
{
    if (ENC == ENC_E4M3) {
        const half2v a = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(hi4, 0.00390625f, false);
        const half2v b = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(hi4, 0.00390625f, true);
        const uint32_t l01 = __builtin_amdgcn_perm(0u, lo4, 0x0c010c00u);  // 0, lo1, 0, lo0
        const uint32_t l23 = __builtin_amdgcn_perm(0u, lo4, 0x0c030c02u);  // 0, lo3, 0, lo2
        return u32x2{(l01 & 0x007F007Fu) | __builtin_bit_cast(uint32_t, a),
                     (l23 & 0x007F007Fu) | __builtin_bit_cast(uint32_t, b)};
    }
    return merge4<ENC>(hi4, lo4);
}

// Eight FP16 operands (one MFMA f16 operand) from 8 upper + 8 residual bytes.
template <int ENC>
__device__ __forceinline__ half8 merge8(uint32_t h0, uint32_t h1, uint32_t l0, uint32_t l1)
{
    const u32x2 p = merge4_lin<ENC>(h0, l0);
    const u32x2 q = merge4_lin<ENC>(h1, l1);
    const u32x4 w = {p.x, p.y, q.x, q.y};
    return __builtin_bit_cast(half8, w);
}

// Fast-mode FP16 words of four upper bytes.  E5M2: the byte is the word's
// upper byte (the merge with zero residual bytes).  E4M3: gfx950's packed
// E4M3 -> FP16 conversion with scale 2^-8, one instruction per two words; it
// is exact for every E4M3 number (E4M3 subnormals land on FP16 subnormals)
// and gives the same words as the merge with zero residual bytes, except
// for the E4M3 NaN pattern, which no layer chosen for E4M3 holds.
template <int ENC>
__device__ __forceinline__ u32x2 fast4(uint32_t hi4)
{
    if (ENC == ENC_E4M3) {
        const half2v a = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(hi4, 0.00390625f, false);
        const half2v b = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(hi4, 0.00390625f, true);
        return u32x2{__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b)};
    }
    return merge4<ENC>(hi4, 0u);
}

// One MFMA f16 operand (eight weights) of the mode: merged from upper and
// residual bytes (full) or from the upper bytes alone (fast).
template <int MODE, int ENC>
__device__ __forceinline__ half8 weight8(uint32_t h0, uint32_t h1, uint32_t l0, uint32_t l1)
{
    if (MODE == MODE_FULL)
        return merge8<ENC>(h0, h1, l0, l1);
    const u32x2 p = fast4<ENC>(h0);
    const u32x2 q = fast4<ENC>(h1);
    const u32x4 w = {p.x, p.y, q.x, q.y};
    return __builtin_bit_cast(half8, w);
}

__device__ __forceinline__ half8 as_half8(u32x4 v)
{
    return __builtin_bit_cast(half8, v);
}

// D += A.B on a 16x16 fp32 tile, K = 32 FP16 (v_mfma_f32_16x16x32_f16).
// Lane l holds A[l%16][8*(l/16) .. +7], B[8*(l/16) .. +7][l%16] and
// D[4*(l/16) .. +3][l%16].
__device__ __forceinline__ f32x4 mfma16x16x32(half8 a, half8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// D += A.B on a 16x16 fp32 tile, K = 128 FP8: A (the upper bytes) in E5M2
// (format 1) or OCP E4M3 (format 0), B in OCP E4M3; 32 bytes of each operand
// per lane.  With both scale operands zero the compiler emits the unscaled
// v_mfma_f32_16x16x128_f8f6f4 (cbsz selects the A format).
template <int ENC>
__device__ __forceinline__ f32x4 mfma16x16x128_fp8(i32x8 a, i32x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, ENC == ENC_E5M2 ? 1 : 0, 0,
                                                             0, 0, 0, 0);
}

}  // namespace dps
