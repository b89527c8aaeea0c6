// dps_elementwise.hip -- split, merge, the per-layer encoding choice, FP8 row
// quantization and the split-K reduction (gfx950).  All are bandwidth-bound
// streams of 16-byte vectors.
#include "dps_internal.h"

namespace dps {

namespace {

constexpr int kThreads = 256;

// Upper bytes and lower bytes of the four FP16 words held in two dwords.
__device__ __forceinline__ uint32_t high_bytes(uint32_t d0, uint32_t d1)
{
    return __builtin_amdgcn_perm(d1, d0, 0x07050301u);
}
__device__ __forceinline__ uint32_t low_bytes(uint32_t d0, uint32_t d1)
{
    return __builtin_amdgcn_perm(d1, d0, 0x06040200u);
}

// Two FP16 words per dword -> E4M3-nested words (per 16-bit half: upper byte
// = sign | exponent bits 3..0 | mantissa bits 9..7, low byte = mantissa bits
// 6..0).  The inverse of e4m3_words; bit 14 (the exponent MSB) is dropped.
__device__ __forceinline__ uint32_t e4m3_nest(uint32_t d)
{
    return (d & 0x807F807Fu) | ((d << 1) & 0x7F007F00u);
}

// FP16 magnitude bits below 0x3F80 (1.875): the exponent MSB is zero and the
// E4M3 part is a number (0x3F80 and up would give the E4M3 NaN pattern or
// lose the exponent MSB; infinities and NaNs are above).
__device__ __forceinline__ bool e4m3_fits(uint32_t word16)
{
    return (word16 & 0x7FFFu) < 0x3F80u;
}

int64_t grid_for(int64_t items)
{
    int64_t blocks = (items + kThreads - 1) / kThreads;
    if (blocks < 1)
        blocks = 1;
    if (blocks > 65536)
        blocks = 65536;
    return blocks;
}

// Sec. IV-A / IV-B "Persistent Region": E5M2 keeps hi = w >> 8 (truncation)
// and residual = w & 0xFF; E4M3 keeps sign, exponent bits 3..0 and mantissa
// bits 9..7 in hi and mantissa bits 6..0 in the residual byte.
template <int ENC>
__global__ __launch_bounds__(kThreads) void split_kernel(const uint16_t *__restrict__ w,
                                                         int64_t numel, uint8_t *__restrict__ hi,
                                                         ResidualView res)
{
    uint8_t *pool = const_cast<uint8_t *>(res.pool);
    const int64_t nvec = numel >> 4;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t v = (int64_t)blockIdx.x * kThreads + threadIdx.x; v < nvec; v += stride) {
        const int64_t i0 = v << 4;
        u32x4 a = load16(w + i0);
        u32x4 b = load16(w + i0 + 8);
        if (ENC == ENC_E4M3) {
            a = u32x4{e4m3_nest(a.x), e4m3_nest(a.y), e4m3_nest(a.z), e4m3_nest(a.w)};
            b = u32x4{e4m3_nest(b.x), e4m3_nest(b.y), e4m3_nest(b.z), e4m3_nest(b.w)};
        }
        u32x4 h, l;
        h.x = high_bytes(a.x, a.y);
        h.y = high_bytes(a.z, a.w);
        h.z = high_bytes(b.x, b.y);
        h.w = high_bytes(b.z, b.w);
        l.x = low_bytes(a.x, a.y);
        l.y = low_bytes(a.z, a.w);
        l.z = low_bytes(b.x, b.y);
        l.w = low_bytes(b.z, b.w);
        *reinterpret_cast<u32x4 *>(hi + i0) = h;
        const int64_t off = residual_offset(res, i0);
        if (off >= 0)
            *reinterpret_cast<u32x4 *>(pool + off) = l;
    }
    // ragged tail (< 16 words), one thread
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        for (int64_t i = nvec << 4; i < numel; ++i) {
            const uint16_t word = ENC == ENC_E4M3 ? (uint16_t)e4m3_nest(w[i]) : w[i];
            hi[i] = (uint8_t)(word >> 8);
            const int64_t off = residual_offset(res, i);
            if (off >= 0)
                pool[off] = (uint8_t)(word & 0xFF);
        }
    }
}

// Sec. IV-C "Overall concept": the FP16 word rebuilt from hi and the residual
// byte (merge4 holds both nestings).
template <int ENC>
__global__ __launch_bounds__(kThreads) void merge_kernel(const uint8_t *__restrict__ hi,
                                                         ResidualView res, int64_t numel,
                                                         uint16_t *__restrict__ w)
{
    const int64_t nvec = numel >> 4;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t v = (int64_t)blockIdx.x * kThreads + threadIdx.x; v < nvec; v += stride) {
        const int64_t i0 = v << 4;
        const u32x4 h = load16(hi + i0);
        const u32x4 l = load_lo_lookup(res, i0);
        const u32x2 p0 = merge4<ENC>(h.x, l.x), p1 = merge4<ENC>(h.y, l.y);
        const u32x2 p2 = merge4<ENC>(h.z, l.z), p3 = merge4<ENC>(h.w, l.w);
        const u32x4 a = {p0.x, p0.y, p1.x, p1.y};
        const u32x4 b = {p2.x, p2.y, p3.x, p3.y};
        *reinterpret_cast<u32x4 *>(w + i0) = a;
        *reinterpret_cast<u32x4 *>(w + i0 + 8) = b;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        for (int64_t i = nvec << 4; i < numel; ++i) {
            const int64_t off = residual_offset(res, i);
            const uint16_t lo = off >= 0 ? res.pool[off] : 0;
            const uint32_t t = ((uint32_t)hi[i] << 8) | lo;
            w[i] = (uint16_t)(ENC == ENC_E4M3 ? e4m3_words(t) : t);
        }
    }
}

// Per-layer encoding choice (Sec. IV-C, "Dual-mode serving" paragraph): a
// block stores E5M2 into *out if any of its words does not fit E4M3; *out was
// set to E4M3 by set_enc_kernel just before on the same stream.  Every
// writer stores the same value, so the unordered stores need no atomics.
__global__ void set_enc_kernel(int32_t *out)
{
    *out = ENC_E4M3;
}

__global__ __launch_bounds__(kThreads) void select_enc_kernel(const uint16_t *__restrict__ w,
                                                              int64_t numel, int32_t *out)
{
    const int64_t nvec = numel >> 3;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    bool bad = false;
    for (int64_t v = (int64_t)blockIdx.x * kThreads + threadIdx.x; v < nvec; v += stride) {
        const u32x4 a = load16(w + (v << 3));
        const uint32_t d[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
        for (int j = 0; j < 4; ++j)
            bad |= !e4m3_fits(d[j]) || !e4m3_fits(d[j] >> 16);
    }
    if (blockIdx.x == 0 && threadIdx.x == 0)
        for (int64_t i = nvec << 3; i < numel; ++i)
            bad |= !e4m3_fits(w[i]);
    if (__syncthreads_or(bad) && threadIdx.x == 0)
        *out = ENC_E5M2;
}

// Nearest OCP E4M3 code to v (|v| <= 448), ties to even, written from the
// format: 4 exponent bits (bias 7), 3 mantissa bits, subnormal step 2^-9.
__device__ __forceinline__ uint32_t e4m3_rne(float v)
{
    const uint32_t b = __float_as_uint(v);
    const uint32_t sign = (b >> 24) & 0x80u;
    const uint32_t a = b & 0x7fffffffu;
    const float av = __uint_as_float(a);
    uint32_t code;
    if (av < 0.015625f) {
        // below 2^-6: multiples of 2^-9; 8 * 2^-9 = 2^-6 is code 0x08
        code = (uint32_t)__builtin_rintf(av * 512.0f);
    } else {
        // keep 3 of the 23 fp32 mantissa bits, round to nearest even
        uint32_t q = a >> 20;
        const uint32_t rem = a & 0xFFFFFu;
        q += (rem > 0x80000u) | ((rem == 0x80000u) & (q & 1u));
        code = q - (120u << 3);  // exponent bias 127 -> 7
    }
    return code | sign;
}

__device__ __forceinline__ float half_bits_abs(uint32_t bits16)
{
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(bits16 & 0x7fffu));
}

// One block per row: amax, power-of-two scale, E4M3 codes.
__global__ __launch_bounds__(kThreads) void quant_rows_kernel(const uint16_t *__restrict__ x,
                                                              int64_t k, uint8_t *__restrict__ xq,
                                                              float *__restrict__ scale)
{
    __shared__ float wave_max[kThreads / 64];
    const int64_t r = blockIdx.x;
    const uint16_t *row = x + r * k;
    const int64_t nvec = k >> 4;
    float amax = 0.f;
    for (int64_t v = threadIdx.x; v < nvec; v += kThreads) {
        const u32x4 a = load16(row + (v << 4));
        const u32x4 b = load16(row + (v << 4) + 8);
        const uint32_t d[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            amax = fmaxf(amax, half_bits_abs(d[j]));
            amax = fmaxf(amax, half_bits_abs(d[j] >> 16));
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        amax = fmaxf(amax, __shfl_xor(amax, off, 64));
    if ((threadIdx.x & 63) == 0)
        wave_max[threadIdx.x >> 6] = amax;
    __syncthreads();
    amax = wave_max[0];
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w)
        amax = fmaxf(amax, wave_max[w]);

    // smallest e with amax <= 448 * 2^e; amax = f * 2^E, f in [0.5, 1),
    // 448 = 0.875 * 2^9  =>  e = E - 9, plus one when f > 0.875.
    int e = 0;
    if (amax > 0.f) {
        int E;
        const float f = frexpf(amax, &E);
        e = E - 9 + (f > 0.875f ? 1 : 0);
    }
    if (threadIdx.x == 0)
        scale[r] = ldexpf(1.0f, e);

    uint8_t *qrow = xq + r * k;
    for (int64_t v = threadIdx.x; v < nvec; v += kThreads) {
        const u32x4 a = load16(row + (v << 4));
        const u32x4 b = load16(row + (v << 4) + 8);
        const uint32_t d[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
        uint32_t out[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            uint32_t q = 0;
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const uint32_t bits = (d[2 * j + (h >> 1)] >> (16 * (h & 1))) & 0xffffu;
                const float val = (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
                q |= e4m3_rne(ldexpf(val, -e)) << (8 * h);
            }
            out[j] = q;
        }
        u32x4 o = {out[0], out[1], out[2], out[3]};
        *reinterpret_cast<u32x4 *>(qrow + (v << 4)) = o;
    }
}

// One wave per row, the row held in registers (NV 16-element vectors per
// lane, K <= 1024 NV): one load round trip, the amax reduced across the wave
// without a block barrier, then the same scale and codes as quant_rows_kernel.
// The codes come from gfx950's packed f32 -> E4M3 conversion, which rounds to
// nearest even like e4m3_rne (the values are exact multiples of the scale
// and at most 448, so neither saturation nor a second rounding occurs);
// checked against the oracle on every FP16 value.
template <int NV>
__global__ __launch_bounds__(kThreads) void quant_rows_wave_kernel(const uint16_t *__restrict__ x,
                                                                   int64_t m, int64_t k,
                                                                   uint8_t *__restrict__ xq,
                                                                   float *__restrict__ scale)
{
    const int lane = threadIdx.x & 63;
    const int64_t r = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (r >= m)
        return;  // the whole wave
    const uint16_t *row = x + r * k;
    const int64_t nvec = k >> 4;
    u32x4 lo[NV], hi[NV];
    float amax = 0.f;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const int64_t idx = (int64_t)v * 64 + lane;
        lo[v] = hi[v] = u32x4{0u, 0u, 0u, 0u};
        if (idx < nvec) {
            lo[v] = load16(row + (idx << 4));
            hi[v] = load16(row + (idx << 4) + 8);
        }
    }
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const uint32_t d[8] = {lo[v].x, lo[v].y, lo[v].z, lo[v].w,
                               hi[v].x, hi[v].y, hi[v].z, hi[v].w};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            amax = fmaxf(amax, half_bits_abs(d[j]));
            amax = fmaxf(amax, half_bits_abs(d[j] >> 16));
        }
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        amax = fmaxf(amax, __shfl_xor(amax, off, 64));
    // smallest e with amax <= 448 * 2^e (as in quant_rows_kernel)
    int e = 0;
    if (amax > 0.f) {
        int E;
        const float f = frexpf(amax, &E);
        e = E - 9 + (f > 0.875f ? 1 : 0);
    }
    if (lane == 0)
        scale[r] = ldexpf(1.0f, e);
    uint8_t *qrow = xq + r * k;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const int64_t idx = (int64_t)v * 64 + lane;
        if (idx >= nvec)
            continue;
        const uint32_t d[8] = {lo[v].x, lo[v].y, lo[v].z, lo[v].w,
                               hi[v].x, hi[v].y, hi[v].z, hi[v].w};
        uint32_t out[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float f4[4];
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const uint32_t bits = (d[2 * j + (h >> 1)] >> (16 * (h & 1))) & 0xffffu;
                f4[h] = ldexpf((float)__builtin_bit_cast(_Float16, (uint16_t)bits), -e);
            }
            int q = __builtin_amdgcn_cvt_pk_fp8_f32(f4[0], f4[1], 0, false);
            q = __builtin_amdgcn_cvt_pk_fp8_f32(f4[2], f4[3], q, true);
            out[j] = (uint32_t)q;
        }
        *reinterpret_cast<u32x4 *>(qrow + (idx << 4)) = u32x4{out[0], out[1], out[2], out[3]};
    }
}

template <int VEC>
__global__ __launch_bounds__(kThreads) void splitk_reduce_kernel(const float *__restrict__ partial,
                                                                 int splits, int64_t rows,
                                                                 int64_t n,
                                                                 uint16_t *__restrict__ y)
{
    const int64_t total = rows * n / VEC;
    const int64_t plane = rows * n;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t v = (int64_t)blockIdx.x * kThreads + threadIdx.x; v < total; v += stride) {
        const int64_t i = v * VEC;
        if (VEC == 4) {
            f32x4 acc = *reinterpret_cast<const f32x4 *>(partial + i);
            for (int s = 1; s < splits; ++s) {
                const f32x4 p = *reinterpret_cast<const f32x4 *>(partial + s * plane + i);
                acc += p;
            }
            typedef _Float16 half4 __attribute__((ext_vector_type(4)));
            half4 h = {(_Float16)acc.x, (_Float16)acc.y, (_Float16)acc.z, (_Float16)acc.w};
            *reinterpret_cast<half4 *>(y + i) = h;
        } else {
            float acc = partial[i];
            for (int s = 1; s < splits; ++s)
                acc += partial[s * plane + i];
            y[i] = __builtin_bit_cast(uint16_t, (_Float16)acc);
        }
    }
}

}  // namespace

hipError_t launch_split(int enc, const uint16_t *w, int64_t numel, uint8_t *hi,
                        const ResidualView &res, hipStream_t stream)
{
    const dim3 grid((unsigned)grid_for(numel >> 4));
    if (enc == ENC_E4M3)
        hipLaunchKernelGGL(split_kernel<ENC_E4M3>, grid, dim3(kThreads), 0, stream, w, numel, hi,
                           res);
    else
        hipLaunchKernelGGL(split_kernel<ENC_E5M2>, grid, dim3(kThreads), 0, stream, w, numel, hi,
                           res);
    return hipGetLastError();
}

hipError_t launch_merge(int enc, const uint8_t *hi, const ResidualView &res, int64_t numel,
                        uint16_t *w_out, hipStream_t stream)
{
    const dim3 grid((unsigned)grid_for(numel >> 4));
    if (enc == ENC_E4M3)
        hipLaunchKernelGGL(merge_kernel<ENC_E4M3>, grid, dim3(kThreads), 0, stream, hi, res, numel,
                           w_out);
    else
        hipLaunchKernelGGL(merge_kernel<ENC_E5M2>, grid, dim3(kThreads), 0, stream, hi, res, numel,
                           w_out);
    return hipGetLastError();
}

hipError_t launch_select_enc(const uint16_t *w, int64_t numel, int32_t *enc_out,
                             hipStream_t stream)
{
    hipLaunchKernelGGL(set_enc_kernel, dim3(1), dim3(1), 0, stream, enc_out);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || numel == 0)
        return e;
    int64_t blocks = grid_for(numel >> 3);
    blocks = blocks < 1024 ? blocks : 1024;  // at most 1024 stores of the verdict
    hipLaunchKernelGGL(select_enc_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, w,
                       numel, enc_out);
    return hipGetLastError();
}

template <int NV>
hipError_t launch_quant_wave(const uint16_t *x, int64_t m, int64_t k, uint8_t *xq, float *scale,
                             hipStream_t stream)
{
    const int64_t rows_per_block = kThreads / 64;
    hipLaunchKernelGGL(quant_rows_wave_kernel<NV>,
                       dim3((unsigned)((m + rows_per_block - 1) / rows_per_block)),
                       dim3(kThreads), 0, stream, x, m, k, xq, scale);
    return hipGetLastError();
}

hipError_t launch_quant_rows(const uint16_t *x, int64_t m, int64_t k, uint8_t *xq, float *scale,
                             hipStream_t stream)
{
    // rows of up to 16384 elements: one wave per row from registers
    switch ((k + 1023) / 1024) {
    case 1: return launch_quant_wave<1>(x, m, k, xq, scale, stream);
    case 2: return launch_quant_wave<2>(x, m, k, xq, scale, stream);
    case 3:
    case 4: return launch_quant_wave<4>(x, m, k, xq, scale, stream);
    case 5:
    case 6:
    case 7:
    case 8: return launch_quant_wave<8>(x, m, k, xq, scale, stream);
    case 9:
    case 10:
    case 11:
    case 12: return launch_quant_wave<12>(x, m, k, xq, scale, stream);
    case 13:
    case 14:
    case 15:
    case 16: return launch_quant_wave<16>(x, m, k, xq, scale, stream);
    default:
        hipLaunchKernelGGL(quant_rows_kernel, dim3((unsigned)m), dim3(kThreads), 0, stream, x, k,
                           xq, scale);
        return hipGetLastError();
    }
}

hipError_t launch_splitk_reduce(const float *partial, int splits, int64_t rows, int64_t n,
                                uint16_t *y, hipStream_t stream)
{
    if (n % 4 == 0)
        hipLaunchKernelGGL(splitk_reduce_kernel<4>, dim3((unsigned)grid_for(rows * n / 4)),
                           dim3(kThreads), 0, stream, partial, splits, rows, n, y);
    else
        hipLaunchKernelGGL(splitk_reduce_kernel<1>, dim3((unsigned)grid_for(rows * n)),
                           dim3(kThreads), 0, stream, partial, splits, rows, n, y);
    return hipGetLastError();
}

}  // namespace dps
