// dps_gemv.hip -- decode-shaped nested linear for one to four tokens on the
// vector ALUs (gfx950).
//
// A product of a few tokens leaves the matrix cores mostly idle and is bound by
// the weight stream, so this kernel streams each weight row in the fastest
// load shape the part has: one wave instruction = 1 KiB of one row, 64 lanes
// x 16 contiguous bytes (nontemporal), measured at 7.2-7.9 TB/s from HBM
// against 5-6 TB/s for 4-8-row shapes.  Each wave owns R whole rows, K
// included, so K is never split and no second kernel sums partials:
//   - the block stages X [M][K] (FP16) in LDS once; lane l of a 1 KiB chunk
//     reads the 16 activations of every token that pair with its 16 weights
//     (32 contiguous bytes per token, a linear pattern);
//   - the upper bytes (and, in full mode, the residual bytes, through the
//     chunk table) are merged into FP16 words in registers exactly as in the
//     matrix-core kernels, and each lane accumulates its 16 products per row
//     and token in fp32 with v_dot2_f32_f16;
//   - chunks are prefetched D deep in registers, so D KiB per row are in
//     flight per wave;
//   - at the end a butterfly over the 64 lanes sums each (row, token) in a
//     fixed order, and the FP16 result is written.
// Fast mode runs the same code on zero residual bytes' words, so fast equals
// full over a zero residual bit for bit.
#include "dps_internal.h"

namespace dps {

namespace {

constexpr int kGemvDepth = 4;  // chunks in flight per row
constexpr int kChunk = 1024;   // K elements (= upper bytes) per wave instruction

struct GemvArgs {
    const uint16_t *x;  // FP16 [m][k]
    int m;              // tokens (<= the kernel's M)
    const uint8_t *hi;
    ResidualView res;
    int64_t n, k;
    uint16_t *y;        // FP16 [m][n]
};

__device__ __forceinline__ u32x4 load_nt16(const void *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

__device__ __forceinline__ u32x4 keep16(bool keep, u32x4 v)
{
    const uint32_t msk = 0u - (uint32_t)keep;
    return v & u32x4{msk, msk, msk, msk};
}

// Eight FP16 pairs (16 weights) of the mode from 16 upper and 16 residual bytes.
template <int MODE, int ENC>
__device__ __forceinline__ void words16(u32x4 h, u32x4 l, uint32_t (&w)[8])
{
    const uint32_t hh[4] = {h.x, h.y, h.z, h.w};
    const uint32_t ll[4] = {l.x, l.y, l.z, l.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const u32x2 p = MODE == MODE_FULL ? merge4_lin<ENC>(hh[j], ll[j]) : fast4<ENC>(hh[j]);
        w[2 * j] = p.x;
        w[2 * j + 1] = p.y;
    }
}

// M: token slots (1, 2 or 4); a.m <= M tokens are live, the others read
// zeros and write nothing.  W waves per block share one staged copy of X.
template <int MODE, int ENC, int M, int R, int W, bool RANGE>
__global__ __launch_bounds__(W * 64) void gemv_kernel(GemvArgs a)
{
    extern __shared__ __attribute__((aligned(16))) uint16_t xs[];  // X [a.m][k]
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    const int64_t r0 = ((int64_t)blockIdx.x * W + wave) * R;
    const bool has_rows = r0 < a.n;  // uniform per wave

    const uint8_t *hrow[R];
    int64_t lrow[R];
    bool rok[R];
    RangeResidual rr[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        rok[r] = r0 + r < a.n;
        lrow[r] = (rok[r] ? r0 + r : r0) * a.k;
        hrow[r] = a.hi + lrow[r];
        rr[r].ok0 = rr[r].ok1 = false;
        rr[r].delta0 = rr[r].delta1 = 0;
        rr[r].bnd = 0;
        if (MODE == MODE_FULL && RANGE)
            rr[r] = range_residual(a.res, lrow[r], lrow[r] + a.k);
    }

    const int64_t nchunks = (a.k + kChunk - 1) / kChunk;
    // loaded vectors and their keep masks; the masks are applied only where
    // the vectors are used, so the loads of later chunks stay in flight
    u32x4 hb[kGemvDepth][R], lb[kGemvDepth][R];
    bool hk[kGemvDepth][R], lk[kGemvDepth][R];

    // chunk c of every row into slot `slot`; chunks past K (or lanes past K in
    // the last one) load from the row's start and are masked to zeros
    auto load = [&](int slot, int64_t c) {
        const int64_t kk = c * kChunk + lane * 16;
        const bool kin = c < nchunks && kk < a.k;
        const int64_t ks = kin ? kk : 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            hb[slot][r] = load_nt16(hrow[r] + ks);
            hk[slot][r] = kin && rok[r];
            if (MODE == MODE_FULL) {
                const int64_t li = lrow[r] + ks;
                int64_t off;
                bool ok;
                if (RANGE) {
                    const bool second = li >= rr[r].bnd;
                    ok = second ? rr[r].ok1 : rr[r].ok0;
                    off = (second ? rr[r].delta1 : rr[r].delta0) + li;
                } else {
                    off = residual_offset(a.res, li);
                    ok = off >= 0;
                }
                lb[slot][r] = load_nt16(a.res.pool + (ok ? off : 0));
                lk[slot][r] = kin && rok[r] && ok;
            } else {
                lb[slot][r] = u32x4{0u, 0u, 0u, 0u};
                lk[slot][r] = false;
            }
        }
    };

    float acc[R][M];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int m = 0; m < M; ++m)
            acc[r][m] = 0.f;

    auto compute = [&](int slot, int64_t c) {
        const int64_t kk = c * kChunk + lane * 16;
        const bool kin = c < nchunks && kk < a.k;
        const int64_t ks = kin ? kk : 0;
        uint32_t xv[M][8];
#pragma unroll
        for (int m = 0; m < M; ++m) {
            const bool live = kin && m < a.m;
            const int64_t xo = (m < a.m ? m : 0) * a.k + ks;
            const u32x4 p = keep16(live, *reinterpret_cast<const u32x4 *>(xs + xo));
            const u32x4 q = keep16(live, *reinterpret_cast<const u32x4 *>(xs + xo + 8));
            const uint32_t v[8] = {p.x, p.y, p.z, p.w, q.x, q.y, q.z, q.w};
#pragma unroll
            for (int j = 0; j < 8; ++j)
                xv[m][j] = v[j];
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            uint32_t w[8];
            words16<MODE, ENC>(keep16(hk[slot][r], hb[slot][r]), keep16(lk[slot][r], lb[slot][r]),
                               w);
#pragma unroll
            for (int m = 0; m < M; ++m)
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    acc[r][m] = __builtin_amdgcn_fdot2(__builtin_bit_cast(half2v, w[j]),
                                                       __builtin_bit_cast(half2v, xv[m][j]),
                                                       acc[r][m], false);
        }
    };

    // the first chunks' weight loads go out before X is staged, so the two
    // latencies overlap
    if (has_rows) {
#pragma unroll
        for (int d = 0; d < kGemvDepth - 1; ++d)
            load(d, d);
    }
    const int64_t nvec = (int64_t)a.m * a.k / 8;  // 16-byte vectors of X
    for (int64_t v = tid; v < nvec; v += W * 64)
        reinterpret_cast<u32x4 *>(xs)[v] = load16(a.x + v * 8);
    __syncthreads();  // the only barrier: waves without rows may leave below
    if (!has_rows)
        return;

    for (int64_t c = 0; c < nchunks; c += kGemvDepth) {
#pragma unroll
        for (int d = 0; d < kGemvDepth; ++d) {
            load((d + kGemvDepth - 1) % kGemvDepth, c + d + kGemvDepth - 1);
            compute(d, c + d);
        }
    }

    // butterfly over the wave: every lane ends with the full sums, in one
    // fixed order
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int m = 0; m < M; ++m)
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1)
                acc[r][m] += __shfl_xor(acc[r][m], off, 64);
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int m = 0; m < M; ++m)
            if (lane == r * M + m && rok[r] && m < a.m)
                a.y[m * a.n + r0 + r] = __builtin_bit_cast(uint16_t, (_Float16)acc[r][m]);
}

template <int MODE, int ENC, int M, int R, int W>
hipError_t launch_mr(const GemvArgs &a, const LinearPlan &plan, hipStream_t stream)
{
    const dim3 grid((unsigned)((a.n + W * R - 1) / (W * R)));
    const size_t lds = (size_t)a.m * (size_t)a.k * 2;
    if (MODE == MODE_FULL && plan.range_addr)
        hipLaunchKernelGGL((gemv_kernel<MODE, ENC, M, R, W, true>), grid, dim3(W * 64), lds,
                           stream, a);
    else
        hipLaunchKernelGGL((gemv_kernel<MODE, ENC, M, R, W, false>), grid, dim3(W * 64), lds,
                           stream, a);
    return hipGetLastError();
}

// Blocks grow with the token count so that staging X stays small against
// the weight rows it serves (MI355X, four tokens on the hidden-4096 QKV and
// O layers: 8-wave blocks 0.75-0.99x the time of 4-wave ones).  One row
// per wave up to 8192 rows (more waves in flight), two beyond.
template <int MODE, int ENC, int M>
hipError_t launch_m(const GemvArgs &a, const LinearPlan &plan, hipStream_t stream)
{
    constexpr int W = M <= 2 ? 4 : 8;
    return a.n <= 8192 ? launch_mr<MODE, ENC, M, 1, W>(a, plan, stream)
                       : launch_mr<MODE, ENC, M, 2, W>(a, plan, stream);
}

template <int MODE, int ENC>
hipError_t launch_mode(const GemvArgs &a, const LinearPlan &plan, int64_t m, hipStream_t stream)
{
    if (m <= 1)
        return launch_m<MODE, ENC, 1>(a, plan, stream);
    if (m <= 2)
        return launch_m<MODE, ENC, 2>(a, plan, stream);
    if (m <= 4)
        return launch_m<MODE, ENC, 4>(a, plan, stream);
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_gemv(const LinearProblem &p, const LinearPlan &plan, hipStream_t stream)
{
    GemvArgs a;
    a.x = p.x;
    a.m = (int)p.rows;
    a.hi = p.hi;
    a.res = p.res;
    a.n = p.n;
    a.k = p.k;
    a.y = p.y;
    if (p.enc == ENC_E4M3)
        return p.mode == MODE_FULL ? launch_mode<MODE_FULL, ENC_E4M3>(a, plan, p.rows, stream)
                                   : launch_mode<MODE_FAST, ENC_E4M3>(a, plan, p.rows, stream);
    return p.mode == MODE_FULL ? launch_mode<MODE_FULL, ENC_E5M2>(a, plan, p.rows, stream)
                               : launch_mode<MODE_FAST, ENC_E5M2>(a, plan, p.rows, stream);
}

}  // namespace dps
