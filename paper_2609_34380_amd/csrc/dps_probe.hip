// dps_probe.hip -- measured ceilings of the MI355X (gfx950) units the nested
// linear layer is bound by, for the benchmark's roofline fractions.  Not part
// of the nested-linear path: a separate library (libdps_probe.so).
//
//   - stream_read_kernel: every byte of a buffer read once with 16-byte loads
//     (1 KiB per wave instruction, the load shape the decode kernels stream
//     weights with), each block over a contiguous chunk of its own, folded
//     into one word per block so no load is dead.
//   - mfma_loop_kernel: back-to-back MFMAs on register operands, eight
//     independent accumulator chains per wave, FP16 16x16x32 or FP8
//     16x16x128, nothing from memory inside the loop.
//   - lds_fill_kernel: the GEMMs' global -> LDS fill alone: one block per
//     CU, NL waves issuing direct-to-LDS loads of 8 rows x 128 bytes per
//     instruction (rows 4 KiB apart, the weight planes' pitch at K = 4096)
//     into 64 KiB stages of a two-slot ring, one barrier per stage.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dps_probe.h"

#define DPS_PROBE_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x8 __attribute__((ext_vector_type(8)));

constexpr int kThreads = 256;

template <bool NT>
__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4 *__restrict__ src,
                                                               int64_t n16, int64_t chunk16,
                                                               uint32_t *out)
{
    // block b reads the 16-byte vectors [b * chunk16, (b+1) * chunk16): 4 KiB
    // per block instruction (1 KiB per wave), four instructions in flight
    constexpr int U = 4;
    u32x4 acc = {0u, 0u, 0u, 0u};
    const int64_t b0 = (int64_t)blockIdx.x * chunk16;
    const int64_t b1 = b0 + chunk16 < n16 ? b0 + chunk16 : n16;
    for (int64_t base = b0 + threadIdx.x; base < b1; base += (int64_t)kThreads * U) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + (int64_t)u * kThreads;
            const int64_t j = i < b1 ? i : b1 - 1;  // in bounds; the duplicate is harmless
            v[u] = NT ? __builtin_nontemporal_load(src + j) : src[j];
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            acc ^= v[u];
    }
    uint32_t w = acc.x ^ acc.y ^ acc.z ^ acc.w;
    for (int off = 32; off > 0; off >>= 1)
        w ^= __shfl_xor(w, off);
    __shared__ uint32_t part[kThreads / 64];
    if ((threadIdx.x & 63) == 0)
        part[threadIdx.x >> 6] = w;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
        for (int j = 0; j < kThreads / 64; ++j)
            t ^= part[j];
        out[blockIdx.x] = t;
    }
}

// Launched with 256 threads, bounded at 512: with the looser bound the
// compiler keeps the accumulators in AGPRs and moves them through VGPRs on
// every trip (over a hundred accvgpr moves per eight MFMAs, half the rate);
// at 512 the chains stay in place and the loop is the eight MFMAs alone.
template <int FP8>
__global__ __launch_bounds__(512) void mfma_loop_kernel(int iters, float seed, float *out)
{
    constexpr int NACC = 8;  // independent accumulator chains per wave
    f32x4 acc[NACC];
#pragma unroll
    for (int j = 0; j < NACC; ++j)
        acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int lane = threadIdx.x & 63;
    if (FP8) {
        i32x8 a, b;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            a[i] = (int)(seed * 3.f) + lane * 7 + i;
            b[i] = i * 3 + 0x3c3c3c3c;
        }
        for (int it = 0; it < iters; ++it) {
#pragma unroll
            for (int j = 0; j < NACC; ++j)
                acc[j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, acc[j], 0, 0, 0, 0,
                                                                          0, 0);
        }
    } else {
        half8 a, b;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            a[i] = (_Float16)(seed + 0.001f * lane + i);
            b[i] = (_Float16)(0.5f * i);
        }
        for (int it = 0; it < iters; ++it) {
#pragma unroll
            for (int j = 0; j < NACC; ++j)
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc[j], 0, 0, 0);
        }
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NACC; ++j)
        s += acc[j].x + acc[j].y + acc[j].z + acc[j].w;
    out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = s;
}

// NL loader waves fill 64 KiB per stage (64 / NL instructions each) into
// slot t & 1 while the previous stage's slot is free; every wave waits for
// its own loads and meets the others at one barrier per stage.  Stage t of
// block b covers rows b * 2048 + 512 t (mod the window's rows) at byte column
// 128 (t mod 32) of each 4 KiB row: every address stays inside the window.
template <int NL>
__global__ __launch_bounds__(NL * 64) void lds_fill_kernel(const uint8_t *src, int64_t rows,
                                                           int iters, uint32_t *out)
{
    constexpr int G = 64 / NL;
    __shared__ __attribute__((aligned(16))) uint8_t ring[2][65536];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    auto issue = [&](int t) {
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int ins = wave * G + j;  // 0 .. 63
            const int64_t row =
                ((int64_t)blockIdx.x * 2048 + (int64_t)t * 512 + ins * 8) % (rows - 8) + (lane >> 3);
            const uint8_t *g = src + row * 4096 + (t & 31) * 128 + (lane & 7) * 16;
            __builtin_amdgcn_global_load_lds(
                g, (__attribute__((address_space(3))) void *)&ring[t & 1][ins * 1024], 16, 0, 0);
        }
    };
    issue(0);
    for (int t = 0; t < iters; ++t) {
        __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of stage t have landed
        __syncthreads();
        if (t + 1 < iters)
            issue(t + 1);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0)
        out[blockIdx.x] = *reinterpret_cast<const uint32_t *>(&ring[(iters - 1) & 1][0]);
}

}  // namespace

DPS_PROBE_EXPORT int dps_probe_stream_read(const void *buf, int64_t bytes, int nontemporal,
                                           uint32_t *out, int64_t blocks, void *stream)
{
    if (buf == nullptr || out == nullptr || bytes < 16 || bytes % 16 != 0 || blocks < 1 ||
        blocks > (1 << 20) || ((uintptr_t)buf & 15) != 0)
        return 1;
    const dim3 grid((unsigned)blocks);
    const int64_t n16 = bytes / 16;
    const int64_t chunk16 = (n16 + blocks - 1) / blocks;
    if (nontemporal)
        hipLaunchKernelGGL(stream_read_kernel<true>, grid, dim3(kThreads), 0, (hipStream_t)stream,
                           static_cast<const u32x4 *>(buf), n16, chunk16, out);
    else
        hipLaunchKernelGGL(stream_read_kernel<false>, grid, dim3(kThreads), 0,
                           (hipStream_t)stream, static_cast<const u32x4 *>(buf), n16, chunk16, out);
    return hipGetLastError() == hipSuccess ? 0 : 5;
}

DPS_PROBE_EXPORT int dps_probe_mfma(int fp8, int iters, int64_t blocks, float *out, void *stream)
{
    if (out == nullptr || iters < 1 || blocks < 1 || blocks > (1 << 20))
        return 1;
    const dim3 grid((unsigned)blocks);
    if (fp8)
        hipLaunchKernelGGL(mfma_loop_kernel<1>, grid, dim3(kThreads), 0, (hipStream_t)stream,
                           iters, 0.5f, out);
    else
        hipLaunchKernelGGL(mfma_loop_kernel<0>, grid, dim3(kThreads), 0, (hipStream_t)stream,
                           iters, 0.5f, out);
    return hipGetLastError() == hipSuccess ? 0 : 5;
}

DPS_PROBE_EXPORT int dps_probe_lds_fill(const void *buf, int64_t window_bytes, int loaders,
                                        int iters, int64_t blocks, uint32_t *out, void *stream)
{
    if (buf == nullptr || out == nullptr || window_bytes < (int64_t(1) << 20) ||
        window_bytes % 4096 != 0 || iters < 1 || blocks < 1 || blocks > (1 << 20) ||
        ((uintptr_t)buf & 15) != 0)
        return 1;
    const dim3 grid((unsigned)blocks);
    const int64_t rows = window_bytes / 4096;
    const uint8_t *src = static_cast<const uint8_t *>(buf);
    switch (loaders) {
    case 4:
        hipLaunchKernelGGL(lds_fill_kernel<4>, grid, dim3(256), 0, (hipStream_t)stream, src, rows,
                           iters, out);
        break;
    case 8:
        hipLaunchKernelGGL(lds_fill_kernel<8>, grid, dim3(512), 0, (hipStream_t)stream, src, rows,
                           iters, out);
        break;
    case 16:
        hipLaunchKernelGGL(lds_fill_kernel<16>, grid, dim3(1024), 0, (hipStream_t)stream, src,
                           rows, iters, out);
        break;
    default:
        return 1;
    }
    return hipGetLastError() == hipSuccess ? 0 : 5;
}
