// dps_device.h -- device-side helpers shared by the libdps kernels (gfx950).
//
// Residual addressing (Sec. IV-B "Shared Region"): the residual bytes of a
// weight form a logical stream in row-major element order, cut into chunks
// of C = 2^log2c bytes; chunk c lives in pool slot slots[c].  Every access the
// kernels make is a 16-byte vector at a 16-byte-aligned logical offset, and
// C >= 16, so a vector never straddles two chunks.
//
// Merge (Sec. IV-C "Overall concept"): an FP16 word is (upper byte << 8) |
// residual byte.  The kernels build FP16 operands in registers with one byte
// permute per two weights; fast mode feeds zero residual bytes through the
// same permute, so a fast-mode product is bit-identical to a full-mode
// product whose residual bytes are all zero.
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

// Four FP16 words from four upper bytes (hi4) and four residual bytes (lo4):
// word j = hi byte j << 8 | lo byte j.  v_perm_b32 picks bytes 0-3 from its
// second source and 4-7 from its first.
__device__ __forceinline__ u32x2 merge4(uint32_t hi4, uint32_t lo4)
{
    return u32x2{__builtin_amdgcn_perm(hi4, lo4, 0x05010400u),
                 __builtin_amdgcn_perm(hi4, lo4, 0x07030602u)};
}

// Eight FP16 operands (one MFMA f16 operand) from 8 upper + 8 residual bytes.
__device__ __forceinline__ half8 merge8(uint32_t h0, uint32_t h1, uint32_t l0, uint32_t l1)
{
    const u32x2 p = merge4(h0, l0);
    const u32x2 q = merge4(h1, l1);
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

// D += A.B on a 16x16 fp32 tile, K = 128 FP8: A in E5M2 (format 1), B in
// OCP E4M3 (format 0); 32 bytes of each operand per lane.
__device__ __forceinline__ f32x4 mfma16x16x128_bf8_fp8(i32x8 a, i32x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 1, 0, 0, 0, 0, 0);
}

}  // namespace dps
