// dps_gemm.hip -- prefill-shaped nested linear on the matrix cores (gfx950).
//
// gemm_f16_kernel: Y = X . W^T with W's upper-byte tile (and, in full mode,
// its residual-byte tile) staged in LDS as bytes -- half the LDS bytes of an
// FP16 tile each -- and merged into FP16 operands in registers right before
// v_mfma_f32_16x16x32_f16 (Sec. IV-C: reconstruction during computation).
// gemm_fp8_kernel: fast mode with FP8 activations; the E5M2 upper bytes are
// used as-is as the A operand of v_mfma_f32_16x16x128_f8f6f4 against E4M3
// activations, and the row scale is applied to the fp32 accumulator.
//
// Block tile 128 (weight rows) x 128 (tokens), 4 waves in a 2 x 2 grid, each
// wave 64 x 64 = 4 x 4 MFMA tiles.  Global -> register -> LDS double
// buffering: tile t+1 is fetched while tile t is multiplied, one barrier per
// K tile.  The weight rows are the MFMA A operand, so a lane ends up holding
// four consecutive output features of one token (8-byte FP16 stores).
// Grouped (MoE) calls map grid.y onto (expert, token tile) by scanning the
// device offsets, so only `experts` blocks at most find no work.
#include "dps_internal.h"

namespace dps {

namespace {

constexpr int BM = 128;  // tokens per block
constexpr int BN = 128;  // weight rows per block

struct GemmArgs {
    const void *x;  // FP16 [rows][k] or E4M3 [rows][k]
    const int32_t *offsets;
    int64_t rows;
    int64_t experts;
    const uint8_t *hi;
    ResidualView res;
    int64_t n, k, ksplit;
    int splits;
    uint16_t *y;
    float *partial;
    const float *scale;
};

// Token range of this block: dense calls use grid.y as the token tile;
// grouped calls walk the experts' tile counts.  Returns false if no work.
__device__ __forceinline__ bool block_rows(const GemmArgs &a, int64_t &e, int64_t &m0,
                                           int64_t &m1, int bm = BM)
{
    const int64_t t = blockIdx.y;
    if (!a.offsets) {
        e = 0;
        m0 = t * bm;
        m1 = m0 + bm < a.rows ? m0 + bm : a.rows;
        return m0 < m1;
    }
    int64_t cum = 0;
    int64_t prev = 0;
    for (int64_t ex = 0; ex < a.experts; ++ex) {
        int64_t o1 = a.offsets[ex + 1];
        o1 = o1 < prev ? prev : (o1 > a.rows ? a.rows : o1);
        const int64_t tiles = (o1 - prev + bm - 1) / bm;
        if (t < cum + tiles) {
            e = ex;
            m0 = prev + (t - cum) * bm;
            m1 = m0 + bm < o1 ? m0 + bm : o1;
            return true;
        }
        cum += tiles;
        prev = o1;
    }
    return false;
}

__device__ __forceinline__ void store_tile_out(const GemmArgs &a, int s, int64_t m, int64_t n0,
                                               f32x4 v, int64_t m1)
{
    if (m >= m1 || n0 >= a.n)
        return;
    if (a.splits == 1) {
        uint16_t *yp = a.y + m * a.n + n0;
        if (n0 + 3 < a.n && (a.n & 3) == 0) {
            typedef _Float16 half4 __attribute__((ext_vector_type(4)));
            half4 hv = {(_Float16)v.x, (_Float16)v.y, (_Float16)v.z, (_Float16)v.w};
            *reinterpret_cast<half4 *>(yp) = hv;
        } else {
            const float vv[4] = {v.x, v.y, v.z, v.w};
            for (int r = 0; r < 4 && n0 + r < a.n; ++r)
                yp[r] = __builtin_bit_cast(uint16_t, (_Float16)vv[r]);
        }
    } else {
        float *pp = a.partial + ((int64_t)s * a.rows + m) * a.n + n0;
        if (n0 + 3 < a.n && (a.n & 3) == 0) {
            *reinterpret_cast<f32x4 *>(pp) = v;
        } else {
            const float vv[4] = {v.x, v.y, v.z, v.w};
            for (int r = 0; r < 4 && n0 + r < a.n; ++r)
                pp[r] = vv[r];
        }
    }
}

// ------------------------------------------------------------------------------
// FP16 matrix cores, weights merged in registers
// ------------------------------------------------------------------------------
constexpr int BK16 = 64;          // K elements per tile
constexpr int XP16 = BK16 + 8;    // X tile pitch, halfs (144 B)
constexpr int WP16 = BK16 + 16;   // weight byte tile pitch (80 B)

template <int MODE, bool RANGE>
__global__ __launch_bounds__(256) void gemm_f16_kernel(GemmArgs a)
{
    __shared__ __attribute__((aligned(16))) uint16_t xs[2][BM * XP16];
    __shared__ __attribute__((aligned(16))) uint8_t hs[2][BN * WP16];
    __shared__ __attribute__((aligned(16))) uint8_t ls[MODE == MODE_FULL ? 2 : 1][BN * WP16];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 15;
    const int lg = lane >> 4;

    int64_t e, mrow0, mrow1;
    if (!block_rows(a, e, mrow0, mrow1))
        return;
    const int ntile = blockIdx.x / a.splits;
    const int s = blockIdx.x % a.splits;
    const int64_t n0 = (int64_t)ntile * BN;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const uint16_t *x = static_cast<const uint16_t *>(a.x);

    // global load assignment (fixed rows per thread)
    const int64_t xr0 = tid >> 3;                // + 32 * j, j < 4
    const int xc = (tid & 7) * 8;                // halfs
    const int64_t wr0 = tid >> 2;                // + 64 * j, j < 2
    const int wc = (tid & 3) * 16;               // bytes
    int64_t lrow[2];
    bool wok[2];
    RangeResidual rr[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int64_t nr = n0 + wr0 + 64 * j;
        wok[j] = nr < a.n;
        lrow[j] = (e * a.n + nr) * a.k;
        if (MODE == MODE_FULL && RANGE) {
            rr[j].ok0 = rr[j].ok1 = false;
            rr[j].delta0 = rr[j].delta1 = 0;
            rr[j].bnd = 0;
            if (wok[j] && ke > kb0)
                rr[j] = range_residual(a.res, lrow[j] + kb0, lrow[j] + ke);
        }
    }

    u32x4 xreg[4], hreg[2], lreg[2];
    auto gload = [&](int64_t kt) {
        const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t m = mrow0 + xr0 + 32 * j;
            xreg[j] = z;
            if (m < mrow1 && kt + xc < ke)
                xreg[j] = load16(x + m * a.k + kt + xc);
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            hreg[j] = z;
            lreg[j] = z;
            if (wok[j] && kt + wc < ke) {
                hreg[j] = load16(a.hi + lrow[j] + kt + wc);
                if (MODE == MODE_FULL)
                    lreg[j] = RANGE ? load_lo_range(a.res, rr[j], lrow[j] + kt + wc)
                                    : load_lo_lookup(a.res, lrow[j] + kt + wc);
            }
        }
    };
    auto sstore = [&](int b) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            *reinterpret_cast<u32x4 *>(&xs[b][(xr0 + 32 * j) * XP16 + xc]) = xreg[j];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            *reinterpret_cast<u32x4 *>(&hs[b][(wr0 + 64 * j) * WP16 + wc]) = hreg[j];
            if (MODE == MODE_FULL)
                *reinterpret_cast<u32x4 *>(&ls[b][(wr0 + 64 * j) * WP16 + wc]) = lreg[j];
        }
    };

    const int wn = wave & 1;
    const int wm = wave >> 1;
    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t ntk = ke > kb0 ? (ke - kb0 + BK16 - 1) / BK16 : 0;
    if (ntk > 0) {
        gload(kb0);
        sstore(0);
    }
    __syncthreads();
    for (int64_t t = 0; t < ntk; ++t) {
        const int b = (int)(t & 1);
        if (t + 1 < ntk)
            gload(kb0 + (t + 1) * BK16);
        half8 a0[4], a1[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int row = wn * 64 + nt * 16 + li;
            const u32x4 h = *reinterpret_cast<const u32x4 *>(&hs[b][row * WP16 + lg * 16]);
            u32x4 l = {0u, 0u, 0u, 0u};
            if (MODE == MODE_FULL)
                l = *reinterpret_cast<const u32x4 *>(&ls[b][row * WP16 + lg * 16]);
            a0[nt] = merge8(h.x, h.y, l.x, l.y);
            a1[nt] = merge8(h.z, h.w, l.z, l.w);
        }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const int row = wm * 64 + mt * 16 + li;
            const half8 b0 = as_half8(*reinterpret_cast<const u32x4 *>(&xs[b][row * XP16 + lg * 16]));
            const half8 b1 =
                as_half8(*reinterpret_cast<const u32x4 *>(&xs[b][row * XP16 + lg * 16 + 8]));
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                acc[nt][mt] = mfma16x16x32(a0[nt], b0, acc[nt][mt]);
                acc[nt][mt] = mfma16x16x32(a1[nt], b1, acc[nt][mt]);
            }
        }
        if (t + 1 < ntk)
            sstore(b ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
            store_tile_out(a, s, mrow0 + wm * 64 + mt * 16 + li, n0 + wn * 64 + nt * 16 + lg * 4,
                           acc[nt][mt], mrow1);
}

// ------------------------------------------------------------------------------
// FP16 matrix cores, LDS-DMA pipeline (gfx950 global_load_lds_dwordx4)
// ------------------------------------------------------------------------------
// Tiles stream global -> LDS with direct-to-LDS loads (no registers in flight)
// through a ring of DMA_STAGES stages; each stage holds, for 64 K elements,
// the 128-row upper-byte tile, the residual-byte tile (full mode) and the
// BM-token X tile.  A DMA instruction writes 64 lanes x 16 bytes contiguously,
// so each lane is pointed at the global chunk that belongs at its LDS slot;
// the slot order is XOR-swizzled per row so that the MFMA-layout reads below
// are free of bank conflicts.  Lanes whose chunk is past the K range, or whose
// residual chunk has no valid slot, load from a zero vector instead (a DMA
// cannot zero-fill).  One barrier per stage.
constexpr int DMA_BK = 64;
constexpr int DMA_STAGES = 3;
constexpr int DMA_W_BYTES = BN * DMA_BK;  // one byte plane, 8 KiB

__device__ __attribute__((aligned(16))) const uint8_t g_zero16[16] = {0};

#define DPS_LDS(p) ((__attribute__((address_space(3))) void *)(p))

__device__ __forceinline__ void dma16(const void *src, void *lds_wave_base)
{
    __builtin_amdgcn_global_load_lds(src, DPS_LDS(lds_wave_base), 16, 0, 0);
}

// s_waitcnt vmcnt(n) leaving the other counters alone (gfx9 encoding).
#define DPS_WAIT_VMCNT(n) \
    __builtin_amdgcn_s_waitcnt(((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8))

// Block barrier between pipeline stages.  __syncthreads() carries a
// workgroup-scope fence, which the compiler satisfies by waiting for every
// outstanding vector-memory operation (direct-to-LDS loads count as LDS
// writes): the whole DMA ring would drain at every stage.  The loops instead
// wait for exactly what they need -- their own DMA of the stage about to be
// read (vmcnt, before this call) and their own LDS reads of the slot about to
// be refilled (lgkmcnt(0), here) -- and then meet at a bare s_barrier.  The
// empty asm statements keep the compiler from moving memory accesses across.
__device__ __forceinline__ void stage_barrier()
{
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt at their maxima
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

template <int MODE, int BM>
struct DmaCfg {
    static constexpr int X_BYTES = BM * DMA_BK * 2;
    static constexpr int PLANES = MODE == MODE_FULL ? 2 : 1;
    static constexpr int STAGE = DMA_W_BYTES * PLANES + X_BYTES;
    static constexpr int LDS = STAGE * DMA_STAGES;
    static constexpr int X_INSTR = X_BYTES / 1024 / 4;          // per wave per stage
    static constexpr int W_INSTR = DMA_W_BYTES / 1024 / 4;      // per wave per plane per stage
    static constexpr int NI = W_INSTR * PLANES + X_INSTR;       // DMA instructions per wave per stage
    static constexpr int MT = BM / 32;                          // 16-token tiles per wave
};

template <int MODE, int BM, bool RANGE>
__global__ __launch_bounds__(256) void gemm_f16_dma_kernel(GemmArgs a)
{
    using C = DmaCfg<MODE, BM>;
    __shared__ __attribute__((aligned(16))) uint8_t smem[C::LDS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 15;
    const int lg = lane >> 4;

    int64_t e, mrow0, mrow1;
    if (!block_rows(a, e, mrow0, mrow1, BM))
        return;
    const int ntile = blockIdx.x / a.splits;
    const int s = blockIdx.x % a.splits;
    const int64_t n0 = (int64_t)ntile * BN;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const int64_t ntk = ke > kb0 ? (ke - kb0 + DMA_BK - 1) / DMA_BK : 0;
    const uint16_t *x = static_cast<const uint16_t *>(a.x);

    // ---- per-lane DMA sources that do not change with the K stage ---------------
    // weight rows: instruction j (= wave * W_INSTR + jj) covers rows 16j .. 16j+15,
    // lane l -> row 16j + l/4, LDS chunk slot l%4 holding logical chunk
    // (l%4) ^ ((row >> 2) & 3)
    const uint8_t *wsrc[C::W_INSTR];
    int64_t wl[C::W_INSTR];
    int wchunk[C::W_INSTR];
    RangeResidual rr[C::W_INSTR];
#pragma unroll
    for (int jj = 0; jj < C::W_INSTR; ++jj) {
        const int j = wave * C::W_INSTR + jj;
        const int r = 16 * j + (lane >> 2);
        int64_t nr = n0 + r;
        nr = nr < a.n ? nr : a.n - 1;
        wl[jj] = (e * a.n + nr) * a.k;
        wsrc[jj] = a.hi + wl[jj];
        wchunk[jj] = (lane & 3) ^ ((r >> 2) & 3);
        rr[jj].ok0 = rr[jj].ok1 = false;
        rr[jj].delta0 = rr[jj].delta1 = 0;
        rr[jj].bnd = 0;
        if (MODE == MODE_FULL && RANGE && ke > kb0)
            rr[jj] = range_residual(a.res, wl[jj] + kb0, wl[jj] + ke);
    }
    // X rows: instruction j covers rows 8j .. 8j+7, lane l -> row 8j + l/8,
    // slot l%8 holding logical chunk (l%8) ^ (row & 7) (8 halfs per chunk)
    const uint16_t *xsrc[C::X_INSTR];
    int xchunk[C::X_INSTR];
#pragma unroll
    for (int jj = 0; jj < C::X_INSTR; ++jj) {
        const int j = wave * C::X_INSTR + jj;
        const int r = 8 * j + (lane >> 3);
        int64_t m = mrow0 + r;
        m = m < mrow1 ? m : mrow1 - 1;
        xsrc[jj] = x + m * a.k;
        xchunk[jj] = (lane & 7) ^ (r & 7);
    }

    auto issue = [&](int64_t t) {
        uint8_t *st = smem + (int)(t % DMA_STAGES) * C::STAGE;
        const bool live = t < ntk;
        const int64_t kt = kb0 + t * DMA_BK;
#pragma unroll
        for (int jj = 0; jj < C::W_INSTR; ++jj) {
            const int j = wave * C::W_INSTR + jj;
            const int64_t kk = kt + wchunk[jj] * 16;
            const bool ok = live && kk < ke;
            dma16(ok ? (const void *)(wsrc[jj] + kk) : (const void *)g_zero16, st + j * 1024);
            if (MODE == MODE_FULL) {
                const int64_t li2 = wl[jj] + (ok ? kk : kb0);
                const void *src = g_zero16;
                if (RANGE) {
                    const bool second = li2 >= rr[jj].bnd;
                    const bool cok = second ? rr[jj].ok1 : rr[jj].ok0;
                    const int64_t d = second ? rr[jj].delta1 : rr[jj].delta0;
                    if (ok && cok)
                        src = a.res.pool + (d + li2);
                } else {
                    const int64_t off = residual_offset(a.res, li2);
                    if (ok && off >= 0)
                        src = a.res.pool + off;
                }
                dma16(src, st + DMA_W_BYTES + j * 1024);
            }
        }
#pragma unroll
        for (int jj = 0; jj < C::X_INSTR; ++jj) {
            const int j = wave * C::X_INSTR + jj;
            const int64_t kk = kt + xchunk[jj] * 8;
            const bool ok = live && kk < ke;
            dma16(ok ? (const void *)(xsrc[jj] + kk) : (const void *)g_zero16,
                  st + DMA_W_BYTES * C::PLANES + j * 1024);
        }
    };

    const int wn = wave & 1;
    const int wm = wave >> 1;
    f32x4 acc[4][C::MT];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < C::MT; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int t = 0; t < DMA_STAGES - 1; ++t)
        issue(t);
    for (int64_t t = 0; t < ntk; ++t) {
        DPS_WAIT_VMCNT(C::NI * (DMA_STAGES - 2));
        stage_barrier();
        issue(t + DMA_STAGES - 1);
        const uint8_t *st = smem + (int)(t % DMA_STAGES) * C::STAGE;
        const uint8_t *xs = st + DMA_W_BYTES * C::PLANES;
        half8 a0[4], a1[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int r = wn * 64 + nt * 16 + li;
            const int off = r * DMA_BK + ((lg ^ ((r >> 2) & 3)) << 4);
            const u32x4 h = *reinterpret_cast<const u32x4 *>(st + off);
            u32x4 l = {0u, 0u, 0u, 0u};
            if (MODE == MODE_FULL)
                l = *reinterpret_cast<const u32x4 *>(st + DMA_W_BYTES + off);
            a0[nt] = merge8(h.x, h.y, l.x, l.y);
            a1[nt] = merge8(h.z, h.w, l.z, l.w);
        }
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) {
            const int r = wm * (BM / 2) + mt * 16 + li;
            const uint8_t *row = xs + r * (DMA_BK * 2);
            const half8 b0 = as_half8(*reinterpret_cast<const u32x4 *>(row + (((2 * lg) ^ (r & 7)) << 4)));
            const half8 b1 =
                as_half8(*reinterpret_cast<const u32x4 *>(row + (((2 * lg + 1) ^ (r & 7)) << 4)));
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                acc[nt][mt] = mfma16x16x32(a0[nt], b0, acc[nt][mt]);
                acc[nt][mt] = mfma16x16x32(a1[nt], b1, acc[nt][mt]);
            }
        }
    }
    DPS_WAIT_VMCNT(0);  // no DMA may still target this block's LDS when it exits

#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
            store_tile_out(a, s, mrow0 + wm * (BM / 2) + mt * 16 + li,
                           n0 + wn * 64 + nt * 16 + lg * 4, acc[nt][mt], mrow1);
}

// ------------------------------------------------------------------------------
// Eight-wave LDS-DMA GEMM (two waves per SIMD), FP16 full/fast and FP8 fast
// ------------------------------------------------------------------------------
// Block tile BN weight rows x BM tokens, waves in a WN x WM grid, each wave
// (BN/WN) x (BM/WM).  A stage covers BK K elements: 64 for FP16 (processed as
// two 32-wide MFMA steps), 128 for FP8 (one 16x16x128 step).  Stages stream
// global -> LDS by direct-to-LDS loads through a ring of NSTAGE slots, one
// barrier per stage.  LDS rows hold 16-byte chunks at slot chunk ^ swz(row),
// swz(row) = (row / rows-per-256-bytes) % chunks-per-row, so the 16 rows a
// fragment read touches land in 16 distinct 16-byte bank groups.
//   FP16 step h, lane (i, g): A = weight row i, K 32h+8g .. +7 (8 bytes per
//   plane, merged into FP16 in registers); B = token row i, same K.
//   FP8, lane (i, g): A and B = bytes 32g .. 32g+31 of the stage.
enum { G3_FULL = 0, G3_FAST = 1, G3_FP8 = 2 };

template <int KIND, int BN_, int BM_, int WN, int WM, int NSTAGE>
struct G3 {
    static constexpr bool FP8 = KIND == G3_FP8;
    static constexpr int PLANES = KIND == G3_FULL ? 2 : 1;
    static constexpr int BK = FP8 ? 128 : 64;
    static constexpr int WROW = BK;                  // bytes per weight row per plane
    static constexpr int XROW = FP8 ? BK : 2 * BK;   // bytes per token row
    static constexpr int W_BYTES = BN_ * WROW;
    static constexpr int X_BYTES = BM_ * XROW;
    static constexpr int STAGE = W_BYTES * PLANES + X_BYTES;
    static constexpr int LDS = STAGE * NSTAGE;
    static constexpr int NWAVES = WN * WM;
    static constexpr int W_INSTR = W_BYTES / 1024 / NWAVES;
    static constexpr int X_INSTR = X_BYTES / 1024 / NWAVES;
    static constexpr int NI = W_INSTR * PLANES + X_INSTR;
    static constexpr int TN = BN_ / WN, TM = BM_ / WM;
    static constexpr int NT = TN / 16, MT = TM / 16;
    static_assert(W_BYTES % (1024 * NWAVES) == 0 && X_BYTES % (1024 * NWAVES) == 0, "tiling");
    static_assert(LDS <= 160 * 1024, "LDS");
};

// slot swizzle for rows of `rowbytes` bytes (64 or 128)
template <int ROWBYTES>
__device__ __forceinline__ int g3_swz(int r)
{
    return (r / (256 / ROWBYTES)) % (ROWBYTES / 16);
}

template <int KIND, int BN_, int BM_, int WN, int WM, int NSTAGE, bool RANGE>
__global__ __launch_bounds__(WN * WM * 64) void gemm3_kernel(GemmArgs a)
{
    using C = G3<KIND, BN_, BM_, WN, WM, NSTAGE>;
    __shared__ __attribute__((aligned(16))) uint8_t smem[C::LDS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 15;
    const int lg = lane >> 4;

    int64_t e, mrow0, mrow1;
    int ntile, s;
    if (a.offsets) {
        if (!block_rows(a, e, mrow0, mrow1, BM_))
            return;
        ntile = blockIdx.x / a.splits;
        s = blockIdx.x % a.splits;
    } else {
        // Dense calls use a 1-D grid remapped for the 8 XCDs: block L runs on
        // XCD L % 8, so XCD x is given the contiguous tile range
        // [x * per_xcd, (x+1) * per_xcd), walked with the token tile fastest.
        // Blocks sharing a weight tile then run together on one XCD and fetch
        // it into that XCD's L2 once.
        const int64_t mtiles = (a.rows + BM_ - 1) / BM_;
        const int64_t ntiles = (a.n + BN_ - 1) / BN_;
        const int64_t total = mtiles * ntiles * a.splits;
        const int64_t per_xcd = (total + 7) / 8;
        const int64_t lin = blockIdx.x;
        const int64_t t = (lin % 8) * per_xcd + lin / 8;
        if (t >= total)
            return;
        const int64_t mt = t % mtiles;
        ntile = (int)((t / mtiles) % ntiles);
        s = (int)(t / (mtiles * ntiles));
        e = 0;
        mrow0 = mt * BM_;
        mrow1 = mrow0 + BM_ < a.rows ? mrow0 + BM_ : a.rows;
    }
    const int64_t n0 = (int64_t)ntile * BN_;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const int64_t ntk = ke > kb0 ? (ke - kb0 + C::BK - 1) / C::BK : 0;

    // ---- per-lane DMA descriptors (fixed across stages) ---------------------------
    // weight instruction j: LDS bytes j*1024 .. +1023 of the plane tile
    const uint8_t *wsrc[C::W_INSTR];
    int64_t wl[C::W_INSTR];
    int wel[C::W_INSTR];  // element offset of this lane's chunk within the stage
    RangeResidual rr[C::W_INSTR];
#pragma unroll
    for (int jj = 0; jj < C::W_INSTR; ++jj) {
        const int j = wave * C::W_INSTR + jj;
        const int pos = j * 1024 + lane * 16;
        const int r = pos / C::WROW;
        const int slot = (pos % C::WROW) / 16;
        const int chunk = slot ^ g3_swz<C::WROW>(r);
        int64_t nr = n0 + r;
        nr = nr < a.n ? nr : a.n - 1;
        wl[jj] = (e * a.n + nr) * a.k;
        wsrc[jj] = a.hi + wl[jj];
        wel[jj] = chunk * 16;
        rr[jj].ok0 = rr[jj].ok1 = false;
        rr[jj].delta0 = rr[jj].delta1 = 0;
        rr[jj].bnd = 0;
        if (KIND == G3_FULL && RANGE && ke > kb0)
            rr[jj] = range_residual(a.res, wl[jj] + kb0, wl[jj] + ke);
    }
    const uint8_t *xsrc[C::X_INSTR];
    int xel[C::X_INSTR];
    constexpr int XELEM = C::FP8 ? 1 : 2;  // bytes per X element
#pragma unroll
    for (int jj = 0; jj < C::X_INSTR; ++jj) {
        const int j = wave * C::X_INSTR + jj;
        const int pos = j * 1024 + lane * 16;
        const int r = pos / C::XROW;
        const int slot = (pos % C::XROW) / 16;
        const int chunk = slot ^ g3_swz<C::XROW>(r);
        int64_t m = mrow0 + r;
        m = m < mrow1 ? m : mrow1 - 1;
        xsrc[jj] = static_cast<const uint8_t *>(a.x) + m * a.k * XELEM;
        xel[jj] = chunk * (16 / XELEM);
    }

    auto issue = [&](int64_t t) {
        uint8_t *st = smem + (int)(t % NSTAGE) * C::STAGE;
        const bool live = t < ntk;
        const int64_t kt = kb0 + t * C::BK;
#pragma unroll
        for (int jj = 0; jj < C::W_INSTR; ++jj) {
            const int j = wave * C::W_INSTR + jj;
            const int64_t kk = kt + wel[jj];
            const bool ok = live && kk < ke;
            dma16(ok ? (const void *)(wsrc[jj] + kk) : (const void *)g_zero16, st + j * 1024);
            if (KIND == G3_FULL) {
                const int64_t lo = wl[jj] + (ok ? kk : kb0);
                const void *src = g_zero16;
                if (RANGE) {
                    const bool second = lo >= rr[jj].bnd;
                    const bool cok = second ? rr[jj].ok1 : rr[jj].ok0;
                    const int64_t d = second ? rr[jj].delta1 : rr[jj].delta0;
                    if (ok && cok)
                        src = a.res.pool + (d + lo);
                } else {
                    const int64_t off = residual_offset(a.res, lo);
                    if (ok && off >= 0)
                        src = a.res.pool + off;
                }
                dma16(src, st + C::W_BYTES + j * 1024);
            }
        }
#pragma unroll
        for (int jj = 0; jj < C::X_INSTR; ++jj) {
            const int j = wave * C::X_INSTR + jj;
            const int64_t kk = kt + xel[jj];
            const bool ok = live && kk < ke;
            dma16(ok ? (const void *)(xsrc[jj] + kk * XELEM) : (const void *)g_zero16,
                  st + C::W_BYTES * C::PLANES + j * 1024);
        }
    };

    const int wn = wave % WN;
    const int wm = wave / WN;
    f32x4 acc[C::NT][C::MT];
#pragma unroll
    for (int i = 0; i < C::NT; ++i)
#pragma unroll
        for (int j = 0; j < C::MT; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int t = 0; t < NSTAGE - 1; ++t)
        issue(t);
    for (int64_t t = 0; t < ntk; ++t) {
        DPS_WAIT_VMCNT(C::NI * (NSTAGE - 2));
        stage_barrier();
        issue(t + NSTAGE - 1);
        const uint8_t *st = smem + (int)(t % NSTAGE) * C::STAGE;
        const uint8_t *xs = st + C::W_BYTES * C::PLANES;
        if (C::FP8) {
            i32x8 av[C::NT];
#pragma unroll
            for (int nt = 0; nt < C::NT; ++nt) {
                const int r = wn * C::TN + nt * 16 + li;
                const uint8_t *row = st + r * C::WROW;
                const int sw = g3_swz<C::WROW>(r);
                const u32x4 p = *reinterpret_cast<const u32x4 *>(row + (((2 * lg) ^ sw) << 4));
                const u32x4 q = *reinterpret_cast<const u32x4 *>(row + (((2 * lg + 1) ^ sw) << 4));
                av[nt] = i32x8{(int)p.x, (int)p.y, (int)p.z, (int)p.w,
                               (int)q.x, (int)q.y, (int)q.z, (int)q.w};
            }
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt) {
                const int r = wm * C::TM + mt * 16 + li;
                const uint8_t *row = xs + r * C::XROW;
                const int sw = g3_swz<C::XROW>(r);
                const u32x4 p = *reinterpret_cast<const u32x4 *>(row + (((2 * lg) ^ sw) << 4));
                const u32x4 q = *reinterpret_cast<const u32x4 *>(row + (((2 * lg + 1) ^ sw) << 4));
                const i32x8 bv = {(int)p.x, (int)p.y, (int)p.z, (int)p.w,
                                  (int)q.x, (int)q.y, (int)q.z, (int)q.w};
#pragma unroll
                for (int nt = 0; nt < C::NT; ++nt)
                    acc[nt][mt] = mfma16x16x128_bf8_fp8(av[nt], bv, acc[nt][mt]);
            }
        } else {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                half8 av[C::NT];
#pragma unroll
                for (int nt = 0; nt < C::NT; ++nt) {
                    const int r = wn * C::TN + nt * 16 + li;
                    const int off = r * C::WROW +
                                    (((2 * h + (lg >> 1)) ^ g3_swz<C::WROW>(r)) << 4) + ((lg & 1) << 3);
                    const u32x2 hv = *reinterpret_cast<const u32x2 *>(st + off);
                    u32x2 lv = {0u, 0u};
                    if (KIND == G3_FULL)
                        lv = *reinterpret_cast<const u32x2 *>(st + C::W_BYTES + off);
                    av[nt] = merge8(hv.x, hv.y, lv.x, lv.y);
                }
#pragma unroll
                for (int mt = 0; mt < C::MT; ++mt) {
                    const int r = wm * C::TM + mt * 16 + li;
                    const half8 bv = as_half8(*reinterpret_cast<const u32x4 *>(
                        xs + r * C::XROW + (((4 * h + lg) ^ g3_swz<C::XROW>(r)) << 4)));
#pragma unroll
                    for (int nt = 0; nt < C::NT; ++nt)
                        acc[nt][mt] = mfma16x16x32(av[nt], bv, acc[nt][mt]);
                }
            }
        }
    }
    DPS_WAIT_VMCNT(0);  // no DMA may still target this block's LDS when it exits

#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) {
        const int64_t m = mrow0 + wm * C::TM + mt * 16 + li;
        float sc = 1.f;
        if (C::FP8)
            sc = m < mrow1 ? a.scale[m] : 0.f;
#pragma unroll
        for (int nt = 0; nt < C::NT; ++nt)
            store_tile_out(a, s, m, n0 + wn * C::TN + nt * 16 + lg * 4,
                           C::FP8 ? acc[nt][mt] * sc : acc[nt][mt], mrow1);
    }
}

// ------------------------------------------------------------------------------
// Wide-row LDS-DMA GEMM, FP16 full/fast: 128 x 128 tiles, 128-element stages
// ------------------------------------------------------------------------------
// On gfx950 an LDS-DMA (or plain) load instruction runs at about half speed
// when each row it touches gets 64 contiguous bytes instead of >= 128 (MI355X,
// L2-resident data: 26 vs 50 B/clk per CU; from HBM 4.4 vs 5.2-7.2 TB/s), so
// a stage here spans 128 K elements: weight planes arrive as 8 rows x 128 B
// per instruction and tokens as 4 rows x 256 B.  LDS keeps the rows, 16-byte
// chunks placed at slot chunk ^ swz(row), and fragment reads are single
// ds_read_b128 in patterns measured conflict-free:
//   weight plane, 128-byte rows, swz8(r) = (r >> 1) & 7: lane (i, g) of
//     K-half q reads chunk 4q + g of row i, K 64q+16g .. +15, which feeds two
//     MFMA steps s (bytes 8s .. 8s+7, merged into FP16 in registers);
//   tokens, 256-byte rows, swz16(r) = r & 15: step (q, s) of lane (i, g)
//     reads chunk 8q + 2g + s of token i, K 64q+16g+8s .. +7.
// Both operands of every MFMA pair the same K elements.  Eight waves: waves
// 0-3 take K-half 0 of every stage and waves 4-7 K-half 1, each over a
// 64 x BM/2 quarter of the tile (two waves per SIMD); the halves are summed
// through LDS at the end, in a fixed order.  The token tile BM (32, 64 or
// 128) follows the call's token count, so short calls stage no padding rows.
//
// SPEC adds four DMA waves (one per SIMD) that do nothing but issue the
// direct-to-LDS loads and wait for them; the eight compute waves then never
// stall on address-unit slots and keep the matrix cores fed, and a stage costs
// about max(DMA, MFMA) instead of their sum.  Both kinds of wave meet at the
// one barrier per stage.
//
// Weights and tokens stream through separate LDS rings of WS and XS slots
// (XS <= WS).  Iteration t issues tokens of stage t+XS-1, then weights of
// stage t+WS-1.  The vector-memory counter retires in issue order, so waiting
// until only the instructions issued after the later of tokens t and weights
// t are outstanding (G4::OUTSTANDING) retires exactly those two, and the later
// stages stay in flight across the barrier.
template <int MODE, int BM, int WS, int XS, int NISS>
struct G4 {
    static constexpr int PLANES = MODE == MODE_FULL ? 2 : 1;
    static constexpr int BK = 128;
    static constexpr int MT = BM / 32;              // 16-token tiles per wave
    static constexpr int W_BYTES = 128 * BK;        // one plane, 128 rows
    static constexpr int W_SLOT = W_BYTES * PLANES;
    static constexpr int X_SLOT = BM * BK * 2;      // BM tokens, FP16
    static constexpr int X_BASE = W_SLOT * WS;
    static constexpr int LDS = X_BASE + XS * X_SLOT;
    static constexpr int W_INSTR = W_BYTES / 1024 / NISS;  // per issuing wave per plane
    static constexpr int X_INSTR = X_SLOT / 1024 / NISS;
    static constexpr int NW = W_INSTR * PLANES;  // weight instructions per issuing wave per stage
    static constexpr int NX = X_INSTR;
    // Instructions that may stay outstanding at the wait for stage t: those
    // issued after the later of tokens t and weights t.  With XS < WS that is
    // tokens t, followed in its iteration by one weight group; with XS == WS
    // both go out in the same iteration and weights t come last.
    static constexpr int OUTSTANDING = (XS < WS ? NW : 0) + (XS - 2) * (NX + NW);
    static_assert(WS >= 3 && XS >= 2 && XS <= WS, "ring depths of the counter scheme");
    static_assert(OUTSTANDING <= 63, "vmcnt range");
    static_assert(BM == 32 || BM == 64 || BM == 128, "token tile");
    static_assert(X_INSTR >= 1 && W_INSTR >= 1, "DMA split over the issuing waves");
    static_assert(LDS <= 160 * 1024 && LDS >= 4 * 16384, "LDS (the K-half reduction needs 64 KiB)");
};

__device__ __forceinline__ int swz8(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int swz16(int r) { return r & 15; }

template <int MODE, int BM, int WS, int XS, bool RANGE, bool SPEC>
__global__ __launch_bounds__(SPEC ? 768 : 512) void gemm4_kernel(GemmArgs a)
{
    using C = G4<MODE, BM, WS, XS, SPEC ? 4 : 8>;
    __shared__ __attribute__((aligned(16))) uint8_t smem[C::LDS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 15;
    const int lg = lane >> 4;
    const bool dma_wave = SPEC && wave >= 8;
    const int issuer = SPEC ? wave - 8 : wave;  // index among the waves that issue DMA
    const int kh = (wave >> 2) & 1;  // K-half of every stage (compute waves)
    const int wn = (wave >> 1) & 1;  // 64-row quarter
    const int wm = wave & 1;         // BM/2-token half

    int64_t e, mrow0, mrow1;
    int ntile, s;
    if (a.offsets) {
        if (!block_rows(a, e, mrow0, mrow1, BM))
            return;
        ntile = blockIdx.x / a.splits;
        s = blockIdx.x % a.splits;
    } else {
        // 1-D grid remapped for the 8 XCDs (block L runs on XCD L % 8): XCD x
        // takes the tile range [x * per_xcd, (x+1) * per_xcd).  Tiles are
        // walked in groups of four weight tiles: token tile, then weight tile
        // within the group, so the ~32 blocks resident on an XCD cover about
        // 4 weight tiles x 8 token tiles and both operands are re-read from
        // that XCD's L2 rather than from HBM.
        const int64_t mtiles = (a.rows + BM - 1) / BM;
        const int64_t ntiles = (a.n + 127) / 128;
        const int64_t total = mtiles * ntiles * a.splits;
        const int64_t per_xcd = (total + 7) / 8;
        const int64_t lin = blockIdx.x;
        const int64_t t = (lin % 8) * per_xcd + lin / 8;
        if (t >= total)
            return;
        constexpr int64_t G = 4;
        s = (int)(t / (mtiles * ntiles));
        const int64_t r = t % (mtiles * ntiles);
        const int64_t chunk = r / (G * mtiles);
        const int64_t within = r % (G * mtiles);
        const int64_t gc = ntiles - chunk * G < G ? ntiles - chunk * G : G;
        const int64_t mt = within / gc;
        ntile = (int)(chunk * G + within % gc);
        e = 0;
        mrow0 = mt * BM;
        mrow1 = mrow0 + BM < a.rows ? mrow0 + BM : a.rows;
    }
    const int64_t n0 = (int64_t)ntile * 128;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const int64_t ntk = ke > kb0 ? (ke - kb0 + C::BK - 1) / C::BK : 0;

    // ---- per-lane DMA state (fixed across stages) ------------------------------
    // Stage t of a lane's weight piece starts at wp + 128 t (upper bytes) and,
    // in full mode, at rp0/rp1 + 128 t (residual bytes in the first / second
    // chunk the row's K range touches; the second serves stages >= tsw).  A
    // piece lies inside [kb0, ke) while 128 t < wlim.  Token pieces likewise:
    // xp + 128 t elements, inside while 128 t < xlim.
    // weight instruction j: rows 8j .. 8j+7, lane -> row 8j + lane/8, slot lane%8
    const uint8_t *wp[C::W_INSTR];
    const uint8_t *rp0[C::W_INSTR], *rp1[C::W_INSTR];
    int64_t wlog[C::W_INSTR];  // logical residual index of the piece at stage 0
    int wlim[C::W_INSTR], tsw[C::W_INSTR];
    bool rok0[C::W_INSTR], rok1[C::W_INSTR];
    const bool issues = !SPEC || dma_wave;  // compute waves of a SPEC block keep no DMA state
#pragma unroll
    for (int jj = 0; jj < C::W_INSTR && issues; ++jj) {
        const int j = issuer * C::W_INSTR + jj;
        const int r = 8 * j + (lane >> 3);
        int64_t nr = n0 + r;
        nr = nr < a.n ? nr : a.n - 1;
        const int wel = ((lane & 7) ^ swz8(r)) * 16;
        const int64_t wl = (e * a.n + nr) * a.k;
        wp[jj] = a.hi + wl + kb0 + wel;
        wlim[jj] = (int)(ke - kb0 - wel);
        wlog[jj] = wl + kb0 + wel;
        rp0[jj] = rp1[jj] = a.res.pool;
        tsw[jj] = 0;
        rok0[jj] = rok1[jj] = false;
        if (MODE == MODE_FULL && RANGE && ke > kb0) {
            const RangeResidual rr = range_residual(a.res, wl + kb0, wl + ke);
            rp0[jj] = a.res.pool + rr.delta0 + wlog[jj];
            rp1[jj] = a.res.pool + rr.delta1 + wlog[jj];
            rok0[jj] = rr.ok0;
            rok1[jj] = rr.ok1;
            const int64_t d = rr.bnd - wlog[jj];  // first stage at or past the chunk boundary
            tsw[jj] = d <= 0 ? 0 : (int)((d + C::BK - 1) / C::BK);
        }
    }
    // token instruction j: rows 4j .. 4j+3, lane -> row 4j + lane/16, slot lane%16
    const uint16_t *xp[C::X_INSTR];
    int xlim[C::X_INSTR];
#pragma unroll
    for (int jj = 0; jj < C::X_INSTR && issues; ++jj) {
        const int j = issuer * C::X_INSTR + jj;
        const int r = 4 * j + (lane >> 4);
        int64_t m = mrow0 + r;
        m = m < mrow1 ? m : mrow1 - 1;
        const int xel = ((lane & 15) ^ swz16(r)) * 8;
        xp[jj] = static_cast<const uint16_t *>(a.x) + m * a.k + kb0 + xel;
        xlim[jj] = (int)(ke - kb0 - xel);
    }
    // stages entirely inside the K range need no masks
    const int64_t t_full = (ke - kb0) / C::BK;

    // One DMA "unit": token instruction jj of stage t, or weight instruction jj
    // of stage t (upper bytes and, in full mode, residual bytes).
    auto issue_w1 = [&](int jj, int64_t t) {
        uint8_t *st = smem + (int)(t % WS) * C::W_SLOT;
        const bool masked = t >= t_full;
        const int64_t off = t * C::BK;
        const int j = issuer * C::W_INSTR + jj;
        const bool ok = !masked || off < wlim[jj];
        dma16(ok ? (const void *)(wp[jj] + off) : (const void *)g_zero16, st + j * 1024);
        if (MODE == MODE_FULL) {
            const void *src = g_zero16;
            if (RANGE) {
                const bool second = t >= tsw[jj];
                const bool cok = second ? rok1[jj] : rok0[jj];
                const uint8_t *base = second ? rp1[jj] : rp0[jj];
                if (ok && cok)
                    src = base + off;
            } else {
                const int64_t o = residual_offset(a.res, wlog[jj] + (ok ? off : 0));
                if (ok && o >= 0)
                    src = a.res.pool + o;
            }
            dma16(src, st + C::W_BYTES + j * 1024);
        }
    };
    auto issue_x1 = [&](int jj, int64_t t) {
        uint8_t *st = smem + C::X_BASE + (int)(t % XS) * C::X_SLOT;
        const bool masked = t >= t_full;
        const int64_t off = t * C::BK;
        const int j = issuer * C::X_INSTR + jj;
        const bool ok = !masked || off < xlim[jj];
        dma16(ok ? (const void *)(xp[jj] + off) : (const void *)g_zero16, st + j * 1024);
    };
    auto issue_w = [&](int64_t t) {
#pragma unroll
        for (int jj = 0; jj < C::W_INSTR; ++jj)
            issue_w1(jj, t);
    };
    auto issue_x = [&](int64_t t) {
#pragma unroll
        for (int jj = 0; jj < C::X_INSTR; ++jj)
            issue_x1(jj, t);
    };
    f32x4 acc[4][C::MT];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < C::MT; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // fragment read offsets (fixed across stages)
    int aoff[4], boff[C::MT][2];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
        const int r = wn * 64 + nt * 16 + li;
        aoff[nt] = r * 128 + (((4 * kh + lg) ^ swz8(r)) << 4);
    }
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) {
        const int r = wm * (BM / 2) + mt * 16 + li;
#pragma unroll
        for (int sidx = 0; sidx < 2; ++sidx)
            boff[mt][sidx] = r * 256 + (((8 * kh + 2 * lg + sidx) ^ swz16(r)) << 4);
    }

    // one stage of matrix work on the slots of stage t
    auto compute = [&](int64_t t) {
        const uint8_t *st = smem + (int)(t % WS) * C::W_SLOT;
        const uint8_t *xs = smem + C::X_BASE + (int)(t % XS) * C::X_SLOT;
        u32x4 hv[4], lv[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            hv[nt] = *reinterpret_cast<const u32x4 *>(st + aoff[nt]);
            lv[nt] = u32x4{0u, 0u, 0u, 0u};
            if (MODE == MODE_FULL)
                lv[nt] = *reinterpret_cast<const u32x4 *>(st + C::W_BYTES + aoff[nt]);
        }
        // without DMA waves, this wave issues its share of the next stages'
        // DMA here, after its fragment reads (their latency overlaps the issue)
        if (!SPEC) {
            issue_x(t + XS - 1);
            issue_w(t + WS - 1);
        }
        half8 a0[4], a1[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            a0[nt] = merge8(hv[nt].x, hv[nt].y, lv[nt].x, lv[nt].y);
            a1[nt] = merge8(hv[nt].z, hv[nt].w, lv[nt].z, lv[nt].w);
        }
#pragma unroll
        for (int sidx = 0; sidx < 2; ++sidx) {
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt) {
                const half8 bv = as_half8(*reinterpret_cast<const u32x4 *>(xs + boff[mt][sidx]));
#pragma unroll
                for (int nt = 0; nt < 4; ++nt)
                    acc[nt][mt] = mfma16x16x32(sidx ? a1[nt] : a0[nt], bv, acc[nt][mt]);
            }
        }
    };

    if (!SPEC || dma_wave) {
        // prologue: the steady-state issue of iterations -(WS-1) .. -1, keeping
        // only stages >= 0, so the counter arithmetic holds from iteration 0
#pragma unroll
        for (int u = -(WS - 1); u < 0; ++u) {
            if (u + XS - 1 >= 0)
                issue_x(u + XS - 1);
            if (u + WS - 1 >= 0)
                issue_w(u + WS - 1);
        }
    }
    if (!SPEC) {
        for (int64_t t = 0; t < ntk; ++t) {
            DPS_WAIT_VMCNT(C::OUTSTANDING);  // tokens t and weights t have landed
            stage_barrier();
            compute(t);
        }
    } else if (dma_wave) {
        // separate loops per role keep the DMA state out of the compute waves'
        // registers and the accumulators out of the DMA waves'
        for (int64_t t = 0; t < ntk; ++t) {
            DPS_WAIT_VMCNT(C::OUTSTANDING);
            stage_barrier();
            issue_x(t + XS - 1);
            issue_w(t + WS - 1);
        }
        DPS_WAIT_VMCNT(0);  // no DMA may still target this block's LDS
        __syncthreads();    // matches the compute waves' two barriers below
        __syncthreads();
        return;
    } else {
        for (int64_t t = 0; t < ntk; ++t) {
            stage_barrier();
            compute(t);
        }
    }
    DPS_WAIT_VMCNT(0);  // no DMA may still target this block's LDS
    __syncthreads();    // every wave is done reading the stages

    // K-half 1 hands its partial sums to K-half 0 through LDS (4 KB per tile)
    f32x4 *red = reinterpret_cast<f32x4 *>(smem) + (wave & 3) * (4 * C::MT * 64);
    if (kh == 1) {
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt)
                red[(nt * C::MT + mt) * 64 + lane] = acc[nt][mt];
    }
    __syncthreads();
    if (kh == 1)
        return;
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) {
        const int64_t m = mrow0 + wm * (BM / 2) + mt * 16 + li;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
            store_tile_out(a, s, m, n0 + wn * 64 + nt * 16 + lg * 4,
                           acc[nt][mt] + red[(nt * C::MT + mt) * 64 + lane], mrow1);
    }
}

// ------------------------------------------------------------------------------
// FP8 matrix cores: E5M2 weights x E4M3 activations
// ------------------------------------------------------------------------------
constexpr int BK8 = 128;        // K elements (= bytes) per tile
constexpr int P8 = BK8 + 16;    // tile pitch, bytes

__global__ __launch_bounds__(256) void gemm_fp8_kernel(GemmArgs a)
{
    __shared__ __attribute__((aligned(16))) uint8_t xs[2][BM * P8];
    __shared__ __attribute__((aligned(16))) uint8_t hs[2][BN * P8];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 15;
    const int lg = lane >> 4;

    int64_t e, mrow0, mrow1;
    if (!block_rows(a, e, mrow0, mrow1))
        return;
    const int ntile = blockIdx.x / a.splits;
    const int s = blockIdx.x % a.splits;
    const int64_t n0 = (int64_t)ntile * BN;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const uint8_t *xq = static_cast<const uint8_t *>(a.x);

    const int64_t r0 = tid >> 3;      // + 32 * j, j < 4 (both tiles)
    const int c0 = (tid & 7) * 16;    // bytes
    u32x4 xreg[4], hreg[4];
    auto gload = [&](int64_t kt) {
        const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t m = mrow0 + r0 + 32 * j;
            const int64_t nr = n0 + r0 + 32 * j;
            xreg[j] = z;
            hreg[j] = z;
            if (kt + c0 < ke) {
                if (m < mrow1)
                    xreg[j] = load16(xq + m * a.k + kt + c0);
                if (nr < a.n)
                    hreg[j] = load16(a.hi + (e * a.n + nr) * a.k + kt + c0);
            }
        }
    };
    auto sstore = [&](int b) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            *reinterpret_cast<u32x4 *>(&xs[b][(r0 + 32 * j) * P8 + c0]) = xreg[j];
            *reinterpret_cast<u32x4 *>(&hs[b][(r0 + 32 * j) * P8 + c0]) = hreg[j];
        }
    };

    const int wn = wave & 1;
    const int wm = wave >> 1;
    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int64_t ntk = ke > kb0 ? (ke - kb0 + BK8 - 1) / BK8 : 0;
    if (ntk > 0) {
        gload(kb0);
        sstore(0);
    }
    __syncthreads();
    for (int64_t t = 0; t < ntk; ++t) {
        const int b = (int)(t & 1);
        if (t + 1 < ntk)
            gload(kb0 + (t + 1) * BK8);
        i32x8 av[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int row = wn * 64 + nt * 16 + li;
            const u32x4 p = *reinterpret_cast<const u32x4 *>(&hs[b][row * P8 + lg * 32]);
            const u32x4 q = *reinterpret_cast<const u32x4 *>(&hs[b][row * P8 + lg * 32 + 16]);
            av[nt] = i32x8{(int)p.x, (int)p.y, (int)p.z, (int)p.w,
                           (int)q.x, (int)q.y, (int)q.z, (int)q.w};
        }
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
            const int row = wm * 64 + mt * 16 + li;
            const u32x4 p = *reinterpret_cast<const u32x4 *>(&xs[b][row * P8 + lg * 32]);
            const u32x4 q = *reinterpret_cast<const u32x4 *>(&xs[b][row * P8 + lg * 32 + 16]);
            const i32x8 bv = {(int)p.x, (int)p.y, (int)p.z, (int)p.w,
                              (int)q.x, (int)q.y, (int)q.z, (int)q.w};
#pragma unroll
            for (int nt = 0; nt < 4; ++nt)
                acc[nt][mt] = mfma16x16x128_bf8_fp8(av[nt], bv, acc[nt][mt]);
        }
        if (t + 1 < ntk)
            sstore(b ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
        const int64_t m = mrow0 + wm * 64 + mt * 16 + li;
        const float sc = m < mrow1 ? a.scale[m] : 0.f;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
            store_tile_out(a, s, m, n0 + wn * 64 + nt * 16 + lg * 4, acc[nt][mt] * sc, mrow1);
    }
}

int64_t token_tiles(int64_t rows, int64_t experts, bool grouped, int bm = BM)
{
    return grouped ? (rows + bm - 1) / bm + experts : (rows + bm - 1) / bm;
}

template <int MODE, int BMT>
void launch_dma(const GemmArgs &a, const LinearPlan &plan, dim3 grid, hipStream_t stream)
{
    if (MODE == MODE_FULL && plan.range_addr)
        hipLaunchKernelGGL((gemm_f16_dma_kernel<MODE, BMT, true>), grid, dim3(256), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm_f16_dma_kernel<MODE, BMT, false>), grid, dim3(256), 0, stream, a);
}

}  // namespace

int gemm_rows_per_block(int variant)
{
    return (variant == GEMM_G3_256x256 || variant == GEMM_G3_256x128 ||
            variant == GEMM_G3_256x256_W16)
               ? 256
               : BN;  // GEMM_G4_128x128 included
}
int gemm_tokens_per_block(int variant)
{
    if (variant == GEMM_G4_128x64 || variant == GEMM_G4S_128x64)
        return 64;
    if (variant == GEMM_G4_128x32 || variant == GEMM_G4S_128x32)
        return 32;
    return (variant == GEMM_DMA_256 || variant == GEMM_G3_256x256 || variant == GEMM_G3_128x256 ||
            variant == GEMM_G3_256x256_W16)
               ? 256
               : BM;
}

namespace {

template <int KIND, int BN_, int BM_, int WN, int WM, int NS>
hipError_t launch_g3(const GemmArgs &a, const LinearPlan &plan, bool grouped, hipStream_t stream)
{
    const int64_t nt = (a.n + BN_ - 1) / BN_;
    dim3 grid((unsigned)(nt * plan.splits),
              (unsigned)token_tiles(a.rows, a.experts, grouped, BM_), 1);
    if (!grouped) {
        const int64_t total = nt * plan.splits * ((a.rows + BM_ - 1) / BM_);
        grid = dim3((unsigned)((total + 7) / 8 * 8), 1, 1);
    }
    if (KIND == G3_FULL && plan.range_addr)
        hipLaunchKernelGGL((gemm3_kernel<KIND, BN_, BM_, WN, WM, NS, true>), grid,
                           dim3(WN * WM * 64), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm3_kernel<KIND, BN_, BM_, WN, WM, NS, false>), grid,
                           dim3(WN * WM * 64), 0, stream, a);
    return hipGetLastError();
}

template <int MODE, int BM, int WS, int XS, bool SPEC>
hipError_t launch_g4(const GemmArgs &a, const LinearPlan &plan, bool grouped, hipStream_t stream)
{
    const int64_t nt = (a.n + 127) / 128;
    dim3 grid((unsigned)(nt * plan.splits), (unsigned)token_tiles(a.rows, a.experts, grouped, BM),
              1);
    if (!grouped) {
        const int64_t total = nt * plan.splits * ((a.rows + BM - 1) / BM);
        grid = dim3((unsigned)((total + 7) / 8 * 8), 1, 1);
    }
    const dim3 block(SPEC ? 768 : 512);
    if (MODE == MODE_FULL && plan.range_addr)
        hipLaunchKernelGGL((gemm4_kernel<MODE, BM, WS, XS, true, SPEC>), grid, block, 0, stream, a);
    else
        hipLaunchKernelGGL((gemm4_kernel<MODE, BM, WS, XS, false, SPEC>), grid, block, 0, stream, a);
    return hipGetLastError();
}

// ring depths per (mode, token tile), within 160 KiB: weights want depth (HBM),
// tokens at least a second slot ahead where it fits
template <int MODE>
hipError_t launch_g4_variant(const GemmArgs &a, const LinearPlan &plan, bool grouped,
                             hipStream_t stream)
{
    // (token tile, weight slots, token slots) per mode, each within 160 KiB
    if constexpr (MODE == MODE_FULL) {
        switch (plan.variant) {
        case GEMM_G4_128x128: return launch_g4<MODE, 128, 3, 2, false>(a, plan, grouped, stream);
        case GEMM_G4_128x64: return launch_g4<MODE, 64, 4, 2, false>(a, plan, grouped, stream);
        case GEMM_G4_128x32: return launch_g4<MODE, 32, 4, 4, false>(a, plan, grouped, stream);
        case GEMM_G4S_128x128: return launch_g4<MODE, 128, 3, 2, true>(a, plan, grouped, stream);
        case GEMM_G4S_128x64: return launch_g4<MODE, 64, 4, 2, true>(a, plan, grouped, stream);
        case GEMM_G4S_128x32: return launch_g4<MODE, 32, 4, 4, true>(a, plan, grouped, stream);
        default: return hipErrorInvalidValue;
        }
    } else {
        switch (plan.variant) {
        case GEMM_G4_128x128: return launch_g4<MODE, 128, 4, 3, false>(a, plan, grouped, stream);
        case GEMM_G4_128x64: return launch_g4<MODE, 64, 6, 4, false>(a, plan, grouped, stream);
        case GEMM_G4_128x32: return launch_g4<MODE, 32, 8, 4, false>(a, plan, grouped, stream);
        case GEMM_G4S_128x128: return launch_g4<MODE, 128, 4, 3, true>(a, plan, grouped, stream);
        case GEMM_G4S_128x64: return launch_g4<MODE, 64, 6, 4, true>(a, plan, grouped, stream);
        case GEMM_G4S_128x32: return launch_g4<MODE, 32, 8, 4, true>(a, plan, grouped, stream);
        default: return hipErrorInvalidValue;
        }
    }
}

template <int KIND>
hipError_t launch_g3_variant(const GemmArgs &a, const LinearPlan &plan, bool grouped,
                             hipStream_t stream)
{
    constexpr bool TWO = KIND == G3_FULL;  // two byte planes: shallower rings
    switch (plan.variant) {
    case GEMM_G3_256x256: return launch_g3<KIND, 256, 256, 2, 4, TWO ? 2 : (KIND == G3_FP8 ? 2 : 3)>(a, plan, grouped, stream);
    case GEMM_G3_128x256: return launch_g3<KIND, 128, 256, 2, 4, 3>(a, plan, grouped, stream);
    case GEMM_G3_256x128: return launch_g3<KIND, 256, 128, 4, 2, 3>(a, plan, grouped, stream);
    case GEMM_G3_128x128: return launch_g3<KIND, 128, 128, 2, 4, 3>(a, plan, grouped, stream);
    case GEMM_G3_256x256_W16: return launch_g3<KIND, 256, 256, 4, 4, TWO ? 2 : (KIND == G3_FP8 ? 2 : 3)>(a, plan, grouped, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_gemm_f16(const LinearProblem &p, const LinearPlan &plan, float *partial,
                           hipStream_t stream)
{
    GemmArgs a;
    a.x = p.x;
    a.offsets = p.offsets;
    a.rows = p.rows;
    a.experts = p.experts;
    a.hi = p.hi;
    a.res = p.res;
    a.n = p.n;
    a.k = p.k;
    a.ksplit = plan.ksplit;
    a.splits = plan.splits;
    a.y = p.y;
    a.partial = partial;
    a.scale = nullptr;
    const int64_t nt = (p.n + BN - 1) / BN;
    if (plan.variant >= GEMM_G4_128x128)
        return p.mode == MODE_FULL ? launch_g4_variant<MODE_FULL>(a, plan, p.offsets != nullptr, stream)
                                   : launch_g4_variant<MODE_FAST>(a, plan, p.offsets != nullptr, stream);
    if (plan.variant >= GEMM_G3_256x256)
        return p.mode == MODE_FULL ? launch_g3_variant<G3_FULL>(a, plan, p.offsets != nullptr, stream)
                                   : launch_g3_variant<G3_FAST>(a, plan, p.offsets != nullptr, stream);
    if (plan.variant == GEMM_DMA_128 || plan.variant == GEMM_DMA_256) {
        const int bm = plan.variant == GEMM_DMA_256 ? 256 : 128;
        dim3 grid((unsigned)(nt * plan.splits),
                  (unsigned)token_tiles(p.rows, p.experts, p.offsets != nullptr, bm), 1);
        if (p.mode == MODE_FULL) {
            if (bm == 256)
                launch_dma<MODE_FULL, 256>(a, plan, grid, stream);
            else
                launch_dma<MODE_FULL, 128>(a, plan, grid, stream);
        } else {
            if (bm == 256)
                launch_dma<MODE_FAST, 256>(a, plan, grid, stream);
            else
                launch_dma<MODE_FAST, 128>(a, plan, grid, stream);
        }
        return hipGetLastError();
    }
    dim3 grid((unsigned)(nt * plan.splits),
              (unsigned)token_tiles(p.rows, p.experts, p.offsets != nullptr), 1);
    if (p.mode == MODE_FULL) {
        if (plan.range_addr)
            hipLaunchKernelGGL((gemm_f16_kernel<MODE_FULL, true>), grid, dim3(256), 0, stream, a);
        else
            hipLaunchKernelGGL((gemm_f16_kernel<MODE_FULL, false>), grid, dim3(256), 0, stream, a);
    } else {
        hipLaunchKernelGGL((gemm_f16_kernel<MODE_FAST, false>), grid, dim3(256), 0, stream, a);
    }
    return hipGetLastError();
}

hipError_t launch_gemm_fp8(const uint8_t *xq, const float *scale, int64_t m, int64_t n,
                           int64_t k, const uint8_t *hi, uint16_t *y, const LinearPlan &plan,
                           float *partial, hipStream_t stream)
{
    GemmArgs a;
    a.x = xq;
    a.offsets = nullptr;
    a.rows = m;
    a.experts = 1;
    a.hi = hi;
    a.res = ResidualView{nullptr, nullptr, 0, 0, 0};
    a.n = n;
    a.k = k;
    a.ksplit = plan.ksplit;
    a.splits = plan.splits;
    a.y = y;
    a.partial = partial;
    a.scale = scale;
    if (plan.variant >= GEMM_G3_256x256)
        return launch_g3_variant<G3_FP8>(a, plan, false, stream);
    const int64_t nt = (n + BN - 1) / BN;
    dim3 grid((unsigned)(nt * plan.splits), (unsigned)token_tiles(m, 1, false), 1);
    hipLaunchKernelGGL(gemm_fp8_kernel, grid, dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace dps
