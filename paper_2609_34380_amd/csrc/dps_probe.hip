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
//   - mfma_lds_kernel: the FP16 GEMMs' compute loop alone: per 64-element
//     stage each wave reads its weight fragments (b128, optionally a second
//     plane merged byte by byte as full mode does) and its token fragments
//     from LDS and runs the MFMAs of its wave tile, optionally ending the
//     stage at a block barrier; no global memory inside the loop.
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

__device__ __forceinline__ int probe_swz8(int r) { return (r >> 1) & 7; }

// NW waves of TN x TM tiles over a 256-row tile; LDS holds one 32 KiB stage
// of each operand, read with the 128-byte-row swizzle of the GEMMs (every
// address modulo 32 KiB).  MERGE: weight fragments come from two planes 64
// bytes apart and are interleaved into FP16 words with v_perm.  BAR: a block
// barrier ends every stage.
template <int NW, int TN, int TM, bool MERGE, bool BAR>
__global__ __launch_bounds__(NW * 64) void mfma_lds_kernel(int iters, float *out)
{
    __shared__ __attribute__((aligned(16))) unsigned char A[32768], B[32768];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int li = lane & 15, lg = lane >> 4;
    for (int i = threadIdx.x; i < 32768 / 16; i += NW * 64) {
        reinterpret_cast<u32x4 *>(A)[i] = u32x4{0x3c003c00u + i, 0x3c003c00u, 0x3c003c00u, 0x3c003c00u};
        reinterpret_cast<u32x4 *>(B)[i] = u32x4{0x3c003c00u, 0x3c003c00u + i, 0x3c003c00u, 0x3c003c00u};
    }
    __syncthreads();
    constexpr int NT = TN / 16, MT = TM / 16, WN = 256 / TN;
    const int wn = wave % WN, wm = wave / WN;
    f32x4 acc[NT][MT];
#pragma unroll
    for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int j = 0; j < MT; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int aoff = ((wn * TN + li) * 128 + ((lg ^ probe_swz8(li)) << 4)) % 32768;
    const int boff0 = ((wm * TM + li) * 128 + ((lg ^ probe_swz8(li)) << 4)) % 32768;
    const int boff1 = ((wm * TM + li) * 128 + (((lg + 4) ^ probe_swz8(li)) << 4)) % 32768;
    for (int it = 0; it < iters; ++it) {
        if (BAR) {
            __builtin_amdgcn_s_waitcnt(0xC07F);
            __builtin_amdgcn_s_barrier();
        }
        half8 av[2][NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const u32x4 h = *reinterpret_cast<const u32x4 *>(A + (aoff + nt * 2048) % 32768);
            if (MERGE) {
                const u32x4 l = *reinterpret_cast<const u32x4 *>(A + (aoff + nt * 2048 + 64) % 32768);
                av[0][nt] = __builtin_bit_cast(
                    half8, u32x4{__builtin_amdgcn_perm(h.x, l.x, 0x05010400u),
                                 __builtin_amdgcn_perm(h.x, l.x, 0x07030602u),
                                 __builtin_amdgcn_perm(h.y, l.y, 0x05010400u),
                                 __builtin_amdgcn_perm(h.y, l.y, 0x07030602u)});
                av[1][nt] = __builtin_bit_cast(
                    half8, u32x4{__builtin_amdgcn_perm(h.z, l.z, 0x05010400u),
                                 __builtin_amdgcn_perm(h.z, l.z, 0x07030602u),
                                 __builtin_amdgcn_perm(h.w, l.w, 0x05010400u),
                                 __builtin_amdgcn_perm(h.w, l.w, 0x07030602u)});
            } else {
                av[0][nt] = __builtin_bit_cast(half8, u32x4{h.x, h.y, h.x, h.y});
                av[1][nt] = __builtin_bit_cast(half8, u32x4{h.z, h.w, h.z, h.w});
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const half8 b0 = *reinterpret_cast<const half8 *>(B + (boff0 + mt * 2048) % 32768);
            const half8 b1 = *reinterpret_cast<const half8 *>(B + (boff1 + mt * 2048) % 32768);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av[0][nt], b0, acc[nt][mt], 0, 0, 0);
                acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av[1][nt], b1, acc[nt][mt], 0, 0, 0);
            }
        }
    }
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int j = 0; j < MT; ++j)
            sum += acc[i][j].x + acc[i][j].w;
    out[(int64_t)blockIdx.x * NW * 64 + threadIdx.x] = sum;
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

DPS_PROBE_EXPORT int dps_probe_mfma_lds(int shape, int merge, int barrier, int iters,
                                        int64_t blocks, float *out, void *stream)
{
    if (out == nullptr || iters < 1 || blocks < 1 || blocks > (1 << 20) || shape < 0 ||
        shape > 1)
        return 1;
    const dim3 grid((unsigned)blocks);
    hipStream_t st = (hipStream_t)stream;
    const int sel = shape * 4 + (merge ? 2 : 0) + (barrier ? 1 : 0);
    switch (sel) {
    case 0: hipLaunchKernelGGL((mfma_lds_kernel<8, 64, 128, false, false>), grid, dim3(512), 0, st, iters, out); break;
    case 1: hipLaunchKernelGGL((mfma_lds_kernel<8, 64, 128, false, true>), grid, dim3(512), 0, st, iters, out); break;
    case 2: hipLaunchKernelGGL((mfma_lds_kernel<8, 64, 128, true, false>), grid, dim3(512), 0, st, iters, out); break;
    case 3: hipLaunchKernelGGL((mfma_lds_kernel<8, 64, 128, true, true>), grid, dim3(512), 0, st, iters, out); break;
    case 4: hipLaunchKernelGGL((mfma_lds_kernel<4, 128, 64, false, false>), grid, dim3(256), 0, st, iters, out); break;
    case 5: hipLaunchKernelGGL((mfma_lds_kernel<4, 128, 64, false, true>), grid, dim3(256), 0, st, iters, out); break;
    case 6: hipLaunchKernelGGL((mfma_lds_kernel<4, 128, 64, true, false>), grid, dim3(256), 0, st, iters, out); break;
    default: hipLaunchKernelGGL((mfma_lds_kernel<4, 128, 64, true, true>), grid, dim3(256), 0, st, iters, out); break;
    }
    return hipGetLastError() == hipSuccess ? 0 : 5;
}
