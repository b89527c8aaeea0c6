// dps_gemm.hip -- prefill-shaped nested linear on the matrix cores (gfx950).
//
// gemm4_kernel: FP16 activations, full and fast mode.  The weight tile's
// upper-byte plane (and, in full mode, its residual plane) is staged in LDS
// as bytes and merged into FP16 operands in registers right before
// v_mfma_f32_16x16x32_f16 (Sec. IV-C: reconstruction during computation);
// fast mode feeds zero residual bytes through the same merge.
// gemm3_kernel: fast mode with FP8 activations.  The upper bytes go to
// v_mfma_f32_16x16x128_f8f6f4 as they are stored -- E5M2, or E4M3 whose
// fast-mode value is E4M3 * 2^-8 -- against E4M3 activations, and the row
// scale (times 2^-8 for E4M3 weights) is applied to the fp32 accumulator.
//
// Both stream their tiles global -> LDS with direct-to-LDS loads through
// rings of stages, one barrier per stage.  Dense calls walk a 1-D grid
// remapped for the 8 XCDs; grouped (MoE) calls map grid.y onto (expert,
// token tile) by scanning the device offsets, so only `experts` blocks at
// most find no work.
#include <type_traits>

#include "dps_internal.h"

namespace dps {

namespace {

constexpr int BM = 128;  // default token tile of block_rows

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
    int rotate;  // wide-row GEMM: start each block's K walk by weight tile (see gemm4)
};

// Token range of this block: dense calls use grid.y as the token tile;
// grouped calls walk the experts' tile counts.  Returns false if no work.
// With tail > 0 (grouped calls) an expert's last tile also takes up to `tail`
// rows beyond bm, so an expert of bm + 1 .. bm + tail rows is one tile, not
// two: its weights are read once.  Such a range [m0, m1) spans more than bm
// rows; the kernel treats rows m0 + bm .. m1 - 1 as its tail.  The tile
// count per expert never grows, so the host's grid bound still holds.
__device__ __forceinline__ bool block_rows(const GemmArgs &a, int64_t &e, int64_t &m0,
                                           int64_t &m1, int bm = BM, int tail = 0)
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
        const int64_t r = o1 - prev;
        const int64_t tiles =
            r <= 0 ? 0 : (r <= bm + tail ? 1 : (r - tail + bm - 1) / bm);
        if (t < cum + tiles) {
            e = ex;
            m0 = prev + (t - cum) * bm;
            m1 = t == cum + tiles - 1 ? o1 : m0 + bm;  // the last tile takes the tail
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


// ------------------------------------------------------------------------------
// Eight-wave LDS-DMA GEMM (two waves per SIMD), fast mode with FP8 activations
// ------------------------------------------------------------------------------
// Block tile BN weight rows x BM tokens, waves in a WN x WM grid, each wave
// (BN/WN) x (BM/WM).  A stage covers 128 K elements (one 16x16x128 MFMA
// step).  Stages stream global -> LDS by direct-to-LDS loads, weights and
// tokens through separate rings of WS and XS slots (the 256 x 256 tile keeps
// two weight stages in flight within 160 KiB), one barrier per stage.  LDS
// rows hold 16-byte chunks at
// slot chunk ^ swz(row), swz(row) = (row / 2) % 8 for the 128-byte rows, so
// the 16 rows a fragment read touches land in 16 distinct 16-byte bank
// groups.  Lane (i, g): A = weight row i and B = token row i, bytes
// 16g .. 16g+15 and 64+16g .. 64+16g+15 of the stage (the MFMA's 32-byte K
// slice of lane group g, permuted alike in both operands).  Reading chunks
// 2g and 2g+1 instead cost ~4 LDS bank-conflict cycles per read (rocprofv3
// SQ_LDS_BANK_CONFLICT) and 3-5% of the prefill time on MI355X.
template <int BN_, int BM_, int WN, int WM, int WS, int XS, bool DW>
struct G3 {
    static constexpr int BK = 128;
    static constexpr int ROW = BK;                   // bytes per row, both operands
    static constexpr int W_BYTES = BN_ * ROW;
    static constexpr int X_BYTES = BM_ * ROW;
    static constexpr int X_BASE = W_BYTES * WS;      // weight ring, then token ring
    static constexpr int LDS = X_BASE + X_BYTES * XS;
    static constexpr int NWAVES = WN * WM;                  // compute waves
    static constexpr int NISS = DW ? 4 : NWAVES;            // waves that issue the DMA
    static constexpr int W_INSTR = W_BYTES / 1024 / NISS;
    static constexpr int X_INSTR = X_BYTES / 1024 / NISS;
    // Iteration t issues tokens of stage t+XS-1, then weights of stage
    // t+WS-1 (XS <= WS).  At the wait for stage t the instructions issued
    // after the later of tokens t and weights t may stay outstanding.
    static constexpr int OUTSTANDING =
        (XS < WS ? W_INSTR : 0) + (XS - 2) * (W_INSTR + X_INSTR);
    static_assert(WS >= 2 && XS >= 2 && XS <= WS, "ring depths");
    static constexpr int TN = BN_ / WN, TM = BM_ / WM;
    static constexpr int NT = TN / 16, MT = TM / 16;
    static_assert(W_BYTES % (1024 * NISS) == 0 && X_BYTES % (1024 * NISS) == 0, "tiling");
    static_assert(LDS <= 160 * 1024, "LDS");
};

__device__ __forceinline__ int g3_swz(int r) { return (r >> 1) & 7; }

// TAIL (grouped calls on the 256 x 128 tile): as in the FP16 wide-row GEMM,
// an expert's last token tile may run up to TAIL rows past 128 (block_rows);
// each compute wave loads the 32-byte K slices of the 16 tail tokens for
// every stage straight from memory into registers and runs them against
// two of its four weight fragments (token half 0 the first two, half 1 the
// last two): 18 MFMAs per stage instead of 16.
template <int ENC, int BN_, int BM_, int WN, int WM, int WS, int XS, bool DW, int TAIL = 0>
__global__ __launch_bounds__(WN * WM * 64 + (DW ? 256 : 0)) void gemm3_kernel(GemmArgs a)
{
    using C = G3<BN_, BM_, WN, WM, WS, XS, DW>;
    static_assert(TAIL == 0 || (TAIL == 16 && DW && BM_ == 128 && WM == 2 && C::NT == 4),
                  "tail rows: the 256 x 128 tile with DMA waves");
    __shared__ __attribute__((aligned(16))) uint8_t smem[C::LDS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 15;
    const int lg = lane >> 4;
    // DW: four more waves (one per SIMD) only issue the direct-to-LDS loads
    // and wait for them; a wave that issues vector-memory instructions stalls
    // on them, and the compute waves then keep the matrix cores busy instead
    const bool dma_wave = DW && wave >= C::NWAVES;
    const int iss = DW ? wave - C::NWAVES : wave;  // index among the issuing waves
    const bool issues = !DW || dma_wave;

    int64_t e, mrow0, mrow1;
    int64_t mtail1 = 0;  // end of the tail rows (TAIL blocks whose range passes BM_)
    int ntile, s;
    if (a.offsets) {
        // grouped: grid.y walks the experts' token tiles, grid.x the weight
        // tiles times the K ranges
        if (!block_rows(a, e, mrow0, mtail1, BM_, TAIL))
            return;
        mrow1 = mrow0 + BM_ < mtail1 ? mrow0 + BM_ : mtail1;
        ntile = blockIdx.x / a.splits;
        s = blockIdx.x % a.splits;
    } else {
        // 1-D grid remapped for the 8 XCDs: block L runs on XCD L % 8, so XCD
        // x is given the contiguous tile range [x * per_xcd, (x+1) * per_xcd),
        // walked with the token tile fastest.  Blocks sharing a weight tile
        // then run together on one XCD and fetch it into that XCD's L2 once.
        const int64_t mtiles = (a.rows + BM_ - 1) / BM_;
        const int64_t ntiles = (a.n + BN_ - 1) / BN_;
        const int64_t total = mtiles * ntiles * a.splits;
        const int64_t per_xcd = (total + 7) / 8;
        const int64_t lin = blockIdx.x;
        const int64_t t0 = (lin % 8) * per_xcd + lin / 8;
        if (t0 >= total)
            return;
        ntile = (int)((t0 / mtiles) % ntiles);
        s = (int)(t0 / (mtiles * ntiles));
        e = 0;
        mrow0 = (t0 % mtiles) * BM_;
        mrow1 = mrow0 + BM_ < a.rows ? mrow0 + BM_ : a.rows;
        mtail1 = mrow1;
    }
    const int64_t n0 = (int64_t)ntile * BN_;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const int64_t ntk = ke > kb0 ? (ke - kb0 + C::BK - 1) / C::BK : 0;

    // Tail rows: lane (i, g) of a compute wave reads bytes 16g .. 16g+15 and
    // 64+16g .. 64+16g+15 of each stage of token mrow0 + BM_ + i (the slice
    // its MFMA operand takes).  K being a multiple of 16, a piece is inside
    // [kb0, ke) whenever it starts there; otherwise the lane reads the row's
    // first 16 bytes of the range and zeroes them.  Lanes past the tail read
    // its last row, whose sums they do not store.
    const bool has_tail = TAIL > 0 && mtail1 > mrow0 + BM_;
    const uint8_t *xt = static_cast<const uint8_t *>(a.x);
    if (has_tail) {
        int64_t m = mrow0 + BM_ + li;
        m = m < mtail1 ? m : mtail1 - 1;
        xt += m * a.k + kb0;
    }

    // ---- per-lane DMA sources (fixed across stages) ------------------------------
    // instruction j covers LDS bytes j*1024 .. +1023 of its operand tile:
    // rows 8j .. 8j+7, lane -> row 8j + lane/8, slot lane%8
    const uint8_t *wsrc[C::W_INSTR];
    int wel[C::W_INSTR];  // K offset of this lane's chunk within the stage
#pragma unroll
    for (int jj = 0; jj < C::W_INSTR && issues; ++jj) {
        const int j = iss * C::W_INSTR + jj;
        const int r = 8 * j + (lane >> 3);
        int64_t nr = n0 + r;
        nr = nr < a.n ? nr : a.n - 1;
        wsrc[jj] = a.hi + (e * a.n + nr) * a.k;
        wel[jj] = ((lane & 7) ^ g3_swz(r)) * 16;
    }
    const uint8_t *xsrc[C::X_INSTR];
    int xel[C::X_INSTR];
#pragma unroll
    for (int jj = 0; jj < C::X_INSTR && issues; ++jj) {
        const int j = iss * C::X_INSTR + jj;
        const int r = 8 * j + (lane >> 3);
        int64_t m = mrow0 + r;
        m = m < mrow1 ? m : mrow1 - 1;
        xsrc[jj] = static_cast<const uint8_t *>(a.x) + m * a.k;
        xel[jj] = ((lane & 7) ^ g3_swz(r)) * 16;
    }

    auto issue_w = [&](int64_t t) {
        uint8_t *st = smem + (int)(t % WS) * C::W_BYTES;
        const bool live = t < ntk;
        const int64_t kt = kb0 + t * C::BK;
#pragma unroll
        for (int jj = 0; jj < C::W_INSTR; ++jj) {
            const int j = iss * C::W_INSTR + jj;
            const int64_t kk = kt + wel[jj];
            const bool ok = live && kk < ke;
            dma16(ok ? (const void *)(wsrc[jj] + kk) : (const void *)g_zero16, st + j * 1024);
        }
    };
    auto issue_x = [&](int64_t t) {
        uint8_t *st = smem + C::X_BASE + (int)(t % XS) * C::X_BYTES;
        const bool live = t < ntk;
        const int64_t kt = kb0 + t * C::BK;
#pragma unroll
        for (int jj = 0; jj < C::X_INSTR; ++jj) {
            const int j = iss * C::X_INSTR + jj;
            const int64_t kk = kt + xel[jj];
            const bool ok = live && kk < ke;
            dma16(ok ? (const void *)(xsrc[jj] + kk) : (const void *)g_zero16, st + j * 1024);
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

    // prologue: the steady-state issue of iterations -(WS-1) .. -1, keeping
    // only stages >= 0
#pragma unroll
    for (int u = -(WS - 1); u < 0 && issues; ++u) {
        if (u + XS - 1 >= 0)
            issue_x(u + XS - 1);
        if (u + WS - 1 >= 0)
            issue_w(u + WS - 1);
    }
    if (DW && dma_wave) {
        // the DMA waves' own loop keeps their source pointers out of the
        // compute waves' registers (and the accumulators out of theirs)
        for (int64_t t = 0; t < ntk; ++t) {
            DPS_WAIT_VMCNT(C::OUTSTANDING);  // tokens t and weights t have landed
            stage_barrier();
            issue_x(t + XS - 1);
            issue_w(t + WS - 1);
        }
        DPS_WAIT_VMCNT(0);  // no DMA may still target this block's LDS when it exits
        return;
    }
    f32x4 tacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
    const int wmu = __builtin_amdgcn_readfirstlane(wm);  // token half, wave-uniform
    // one stage of a compute wave, which without DW also issues its share of
    // the DMA (tail_c: std::true_type in blocks with tail rows)
    auto stage = [&](int64_t t, auto tail_c) {
        constexpr bool TL = decltype(tail_c)::value;
        if (!DW)
            DPS_WAIT_VMCNT(C::OUTSTANDING);  // tokens t and weights t have landed
        stage_barrier();
        if (!DW) {
            issue_x(t + XS - 1);
            issue_w(t + WS - 1);
        }
        u32x4 tp = {0u, 0u, 0u, 0u}, tq = {0u, 0u, 0u, 0u};
        if constexpr (TL) {
            const int64_t off = t * C::BK + 16 * lg;
            const bool ok = kb0 + off < ke;
            const uint32_t msk = 0u - (uint32_t)ok;
            const uint8_t *pp = xt + (ok ? off : 0);
            tp = load16(pp) & u32x4{msk, msk, msk, msk};
            tq = load16(pp + (ok ? 64 : 0)) & u32x4{msk, msk, msk, msk};
        }
        const uint8_t *st = smem + (int)(t % WS) * C::W_BYTES;
        const uint8_t *xs = smem + C::X_BASE + (int)(t % XS) * C::X_BYTES;
        i32x8 av[C::NT];
#pragma unroll
        for (int nt = 0; nt < C::NT; ++nt) {
            const int r = wn * C::TN + nt * 16 + li;
            const uint8_t *row = st + r * C::ROW;
            const int sw = g3_swz(r);
            const u32x4 p = *reinterpret_cast<const u32x4 *>(row + ((lg ^ sw) << 4));
            const u32x4 q = *reinterpret_cast<const u32x4 *>(row + (((4 + lg) ^ sw) << 4));
            av[nt] = i32x8{(int)p.x, (int)p.y, (int)p.z, (int)p.w,
                           (int)q.x, (int)q.y, (int)q.z, (int)q.w};
        }
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) {
            const int r = wm * C::TM + mt * 16 + li;
            const uint8_t *row = xs + r * C::ROW;
            const int sw = g3_swz(r);
            const u32x4 p = *reinterpret_cast<const u32x4 *>(row + ((lg ^ sw) << 4));
            const u32x4 q = *reinterpret_cast<const u32x4 *>(row + (((4 + lg) ^ sw) << 4));
            const i32x8 bv = {(int)p.x, (int)p.y, (int)p.z, (int)p.w,
                              (int)q.x, (int)q.y, (int)q.z, (int)q.w};
#pragma unroll
            for (int nt = 0; nt < C::NT; ++nt)
                acc[nt][mt] = mfma16x16x128_fp8<ENC>(av[nt], bv, acc[nt][mt]);
        }
        if constexpr (TL) {
            const i32x8 tb = {(int)tp.x, (int)tp.y, (int)tp.z, (int)tp.w,
                              (int)tq.x, (int)tq.y, (int)tq.z, (int)tq.w};
            if (wmu == 0) {
                tacc[0] = mfma16x16x128_fp8<ENC>(av[0], tb, tacc[0]);
                tacc[1] = mfma16x16x128_fp8<ENC>(av[1], tb, tacc[1]);
            } else {
                tacc[0] = mfma16x16x128_fp8<ENC>(av[2], tb, tacc[0]);
                tacc[1] = mfma16x16x128_fp8<ENC>(av[3], tb, tacc[1]);
            }
        }
    };
    if (has_tail) {
        for (int64_t t = 0; t < ntk; ++t)
            stage(t, std::integral_constant<bool, (TAIL > 0)>{});
    } else {
        for (int64_t t = 0; t < ntk; ++t)
            stage(t, std::false_type{});
    }
    DPS_WAIT_VMCNT(0);  // no DMA may still target this block's LDS when it exits

    // E4M3 weights carry the fast-mode factor 2^-8 (exact in fp32)
    constexpr float wscale = ENC == ENC_E4M3 ? 0.00390625f : 1.f;
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) {
        const int64_t m = mrow0 + wm * C::TM + mt * 16 + li;
        const float sc = m < mrow1 ? a.scale[m] * wscale : 0.f;
#pragma unroll
        for (int nt = 0; nt < C::NT; ++nt)
            store_tile_out(a, s, m, n0 + wn * C::TN + nt * 16 + lg * 4, acc[nt][mt] * sc,
                           mrow1);
    }
    if (TAIL > 0 && has_tail) {
        const int64_t m = mrow0 + BM_ + li;
        const float sc = m < mtail1 ? a.scale[m] * wscale : 0.f;
#pragma unroll
        for (int j = 0; j < 2; ++j)
            store_tile_out(a, s, m, n0 + wn * C::TN + (2 * wmu + j) * 16 + lg * 4,
                           tacc[j] * sc, mtail1);
    }
}

// ------------------------------------------------------------------------------
// Wide-row LDS-DMA GEMM, FP16 full/fast: 128 weight rows, 128-element stages
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

// TAIL (grouped calls, 128-token tiles with DMA waves): the block's token
// range may run up to TAIL rows past its 128-token tile (block_rows).  Those
// rows take no LDS: each compute wave loads its K-half of their 16-token
// fragment straight from memory into registers after the stage barrier (the
// tokens of a call are a few MiB and sit in L2) and runs it against the
// weight fragments it already holds, waves of token half 0 on the first two
// 16-row weight sub-tiles of their quarter and waves of half 1 on the other
// two, so every compute wave does 36 MFMAs per stage instead of 32.  The
// tail's K-half sums go through LDS with the others.
template <int MODE, int ENC, int BM, int WS, int XS, bool RANGE, bool SPEC, int TAIL = 0>
__global__ __launch_bounds__(SPEC ? 768 : 512) void gemm4_kernel(GemmArgs a)
{
    using C = G4<MODE, BM, WS, XS, SPEC ? 4 : 8>;
    static_assert(TAIL == 0 || (TAIL == 16 && SPEC && BM == 128), "tail rows: 128-token DMA-wave tile");
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
    int64_t mtail1 = 0;  // end of the tail rows (TAIL blocks whose range passes BM)
    int ntile, s;
    if (a.offsets) {
        if (!block_rows(a, e, mrow0, mtail1, BM, TAIL))
            return;
        mrow1 = mrow0 + BM < mtail1 ? mrow0 + BM : mtail1;
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
        mtail1 = mrow1;
    }
    const int64_t n0 = (int64_t)ntile * 128;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const int64_t ntk = ke > kb0 ? (ke - kb0 + C::BK - 1) / C::BK : 0;

    // Tail rows: lane (i, g) of a compute wave loads 32 bytes of token
    // mrow0 + BM + i per stage, K 64 kh + 16 g .. +15 (its two MFMA steps).
    // K being a multiple of 16, such a piece lies inside [kb0, ke) whenever
    // it starts there (stage offset below xtlim); otherwise the lane reads the
    // row's first 16 elements of the range and zeroes them.  Lanes past the
    // tail read its last row, whose sums they do not store.
    const bool has_tail = TAIL > 0 && mtail1 > mrow0 + BM;
    const uint16_t *xt = static_cast<const uint16_t *>(a.x);
    const int xtk = 64 * kh + 16 * lg;
    int xtlim = 0;
    if (has_tail) {
        int64_t m = mrow0 + BM + li;
        m = m < mtail1 ? m : mtail1 - 1;
        xt += m * a.k + kb0;
        xtlim = (int)(ke - kb0 - xtk);
    }
    const int wmu = __builtin_amdgcn_readfirstlane(wm);  // token half, wave-uniform

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
    // Iteration t stages K range tk(t).  With rows a multiple of 4 KiB apart,
    // blocks walking their K ranges in step would all touch the same 128-byte
    // column (address bits 7-11) at once; each group of four weight tiles
    // starts at another stage instead.  Token tiles of one weight tile keep
    // the same order, so they still meet in L2.  (MI355X, gate+up 28672 x
    // 4096 in full mode: 0.78x the time at 32 tokens, 0.83x at 128, 0.91x at
    // 256; the other hidden-4096 layers within 3%.)
    const int64_t grot = a.rotate && ntk > 0 ? (int64_t)(ntile >> 2) % ntk : 0;
    auto tk = [&](int64_t t) {
        return t < ntk ? (t + grot < ntk ? t + grot : t + grot - ntk) : t;
    };

    // One DMA "unit": token instruction jj of stage t, or weight instruction jj
    // of stage t (upper bytes and, in full mode, residual bytes).
    auto issue_w1 = [&](int jj, int64_t t) {
        uint8_t *st = smem + (int)(t % WS) * C::W_SLOT;
        const int64_t tr = tk(t);
        const bool masked = tr >= t_full;
        const int64_t off = tr * C::BK;
        const int j = issuer * C::W_INSTR + jj;
        const bool ok = !masked || off < wlim[jj];
        dma16(ok ? (const void *)(wp[jj] + off) : (const void *)g_zero16, st + j * 1024);
        if (MODE == MODE_FULL) {
            const void *src = g_zero16;
            if (RANGE) {
                const bool second = tr >= tsw[jj];
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
        const int64_t tr = tk(t);
        const bool masked = tr >= t_full;
        const int64_t off = tr * C::BK;
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

    f32x4 tacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};

    // one stage of matrix work on the slots of stage t (tail_c: std::true_type
    // in blocks with tail rows)
    auto compute = [&](int64_t t, auto tail_c) {
        constexpr bool TL = decltype(tail_c)::value;
        const uint8_t *st = smem + (int)(t % WS) * C::W_SLOT;
        const uint8_t *xs = smem + C::X_BASE + (int)(t % XS) * C::X_SLOT;
        u32x4 tx0 = {0u, 0u, 0u, 0u}, tx1 = {0u, 0u, 0u, 0u};
        if constexpr (TL) {
            const int64_t off = tk(t) * C::BK;
            const bool ok = off < xtlim;
            const uint32_t msk = 0u - (uint32_t)ok;
            const uint16_t *p = xt + (ok ? off + xtk : 0);
            tx0 = load16(p) & u32x4{msk, msk, msk, msk};
            tx1 = load16(p + 8) & u32x4{msk, msk, msk, msk};
        }
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
            a0[nt] = weight8<MODE, ENC>(hv[nt].x, hv[nt].y, lv[nt].x, lv[nt].y);
            a1[nt] = weight8<MODE, ENC>(hv[nt].z, hv[nt].w, lv[nt].z, lv[nt].w);
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
        if constexpr (TL) {
            const half8 b0 = as_half8(tx0), b1 = as_half8(tx1);
            if (wmu == 0) {
                tacc[0] = mfma16x16x32(a0[0], b0, tacc[0]);
                tacc[1] = mfma16x16x32(a0[1], b0, tacc[1]);
                tacc[0] = mfma16x16x32(a1[0], b1, tacc[0]);
                tacc[1] = mfma16x16x32(a1[1], b1, tacc[1]);
            } else {
                tacc[0] = mfma16x16x32(a0[2], b0, tacc[0]);
                tacc[1] = mfma16x16x32(a0[3], b0, tacc[1]);
                tacc[0] = mfma16x16x32(a1[2], b1, tacc[0]);
                tacc[1] = mfma16x16x32(a1[3], b1, tacc[1]);
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
            compute(t, std::false_type{});
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
    } else if (has_tail) {
        for (int64_t t = 0; t < ntk; ++t) {
            stage_barrier();
            compute(t, std::integral_constant<bool, (TAIL > 0)>{});
        }
    } else {
        for (int64_t t = 0; t < ntk; ++t) {
            stage_barrier();
            compute(t, std::false_type{});
        }
    }
    DPS_WAIT_VMCNT(0);  // no DMA may still target this block's LDS
    __syncthreads();    // every wave is done reading the stages

    // K-half 1 hands its partial sums to K-half 0 through LDS (4 KB per tile)
    constexpr int RED = 4 * C::MT + (TAIL > 0 ? 2 : 0);  // 16 x 16 tiles per wave
    static_assert(4 * RED * 64 * 16 <= C::LDS, "K-half reduction area");
    f32x4 *red = reinterpret_cast<f32x4 *>(smem) + (wave & 3) * (RED * 64);
    if (kh == 1) {
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
            for (int mt = 0; mt < C::MT; ++mt)
                red[(nt * C::MT + mt) * 64 + lane] = acc[nt][mt];
        if (TAIL > 0 && has_tail) {
            red[(4 * C::MT) * 64 + lane] = tacc[0];
            red[(4 * C::MT + 1) * 64 + lane] = tacc[1];
        }
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
    if (TAIL > 0 && has_tail) {
        const int64_t m = mrow0 + BM + li;
#pragma unroll
        for (int j = 0; j < 2; ++j)
            store_tile_out(a, s, m, n0 + wn * 64 + (2 * wmu + j) * 16 + lg * 4,
                           tacc[j] + red[(4 * C::MT + j) * 64 + lane], mtail1);
    }
}

// ------------------------------------------------------------------------------
// Large-tile LDS-DMA GEMM, FP16 full/fast: 256 weight rows, 64-element stages
// ------------------------------------------------------------------------------
// The wide-row GEMM above is bound by its LDS traffic: a 128 x 128 tile
// fills 64 KiB of LDS per 128-element stage for 1024 MFMA cycles per SIMD,
// and its 64 x 64 wave tiles read 16 KiB of fragments per wave per stage.
// This kernel takes 256 weight rows x BM tokens per block (dense calls; the
// planner launches BM = 256) with eight waves in a 4 x 2 grid, each over a
// 64 x BM/2 wave tile on the whole K range of every stage: per FP16 flop it
// fills half the LDS bytes (256 x 256) and reads 0.75x the fragment bytes
// (12 of 16 per 32 MFMAs at BM = 256) of the 128 x 128 tile, and it does
// twice the matrix work between two barriers.  Each wave merges its 64
// weight rows once per stage (two waves share them), keeps them in registers
// and streams the token fragments past them.
//
// A stage is 64 K elements.  A DMA instruction fills 1 KiB of LDS: 8 weight
// lines of 128 bytes (full mode: 8 rows x (64 upper + 64 residual bytes);
// fast mode: 16 rows x 64 upper bytes) or 8 token rows of 128 bytes.  The
// 16-byte chunks sit at swizzled slots (see the weight-line and token-row
// notes below) so that the 16 rows of every fragment read land in distinct
// bank groups.  Lane (i, g) reads the 16-byte chunk holding K 16g .. 16g+15
// of weight row i (both MFMA steps s, bytes 8s .. 8s+7 merged into FP16) and
// the chunk holding K 16g+8s .. +7 of token i: both operands of every MFMA
// pair the same K elements.  All eight waves issue their share of the
// direct-to-LDS loads after the stage barrier; the counter scheme is the
// wide-row GEMM's (weights and tokens in separate rings of WS and XS slots,
// XS <= WS, exact vmcnt waits).
template <int MODE, int BM, int WS, int XS>
struct G5 {
    static constexpr int PLANES = MODE == MODE_FULL ? 2 : 1;
    static constexpr int BN = 256;
    static constexpr int BK = 64;
    static constexpr int W_SLOT = BN * BK * PLANES;     // 128-byte weight lines
    static constexpr int X_SLOT = BM * BK * 2;          // BM rows x 128 bytes
    static constexpr int X_BASE = W_SLOT * WS;
    static constexpr int LDS = X_BASE + XS * X_SLOT;
    static constexpr int NW = W_SLOT / 1024 / 8;        // weight instructions per wave per stage
    static constexpr int NX = X_SLOT / 1024 / 8;
    static constexpr int OUTSTANDING = (XS < WS ? NW : 0) + (XS - 2) * (NX + NW);
    static constexpr int TM = BM / 2;                   // tokens per wave
    static constexpr int MT = TM / 16;
    static_assert(WS >= 2 && XS >= 2 && XS <= WS, "ring depths of the counter scheme");
    static_assert(OUTSTANDING <= 63, "vmcnt range");
    static_assert(BM == 256 || BM == 128, "token tile");
    static_assert(NW >= 1 && NX >= 1, "DMA split over the waves");
    static_assert(LDS <= 160 * 1024, "LDS");
};

// Weight lines: 128 bytes, 16-byte slots at slot chunk ^ swz8(line).  Full
// mode: line r holds weight row r, its upper bytes in chunks 0-3 and its
// residual bytes in chunks 4-7 (16 K elements each).  Fast mode: line
// 16t + i holds row 32t + i in chunks 0-3 and row 32t + 16 + i in chunks 4-7.
// Either way a fragment read -- lane (i, g) of 16 lines reading chunk 4q + g
// -- is the pattern measured conflict-free on MI355X (ds_read_b128 at ~210
// B/clk per CU), where 64-byte rows read whole lose half the rate to bank
// conflicts.
// Token rows: K chunk c (8 elements) of a 128-byte row sits at slot
// sigma(c) ^ swz8(row), sigma(c) = (c >> 1) | (c & 1) << 2, so the chunks
// 2g + s that lane group g reads in MFMA step s are slots (g + 4s) ^ swz8:
// four consecutive slots per step.  Reading chunks 2g + s through the plain
// swizzle costs LDS bank conflicts on MI355X (rocprofv3 SQ_LDS_BANK_CONFLICT
// about half of the LDS active cycles); tok_chunk is sigma's inverse, the K
// chunk the DMA writes into a slot.
__device__ __forceinline__ int tok_chunk(int slot) { return ((slot & 3) << 1) | (slot >> 2); }

template <int MODE, int ENC, int BM, int WS, int XS, bool RANGE>
__global__ __launch_bounds__(512) void gemm5_kernel(GemmArgs a)
{
    using C = G5<MODE, BM, WS, XS>;
    __shared__ __attribute__((aligned(16))) uint8_t smem[C::LDS];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 15;
    const int lg = lane >> 4;
    const int wn = wave & 3;   // 64-row quarter of the weight tile
    const int wm = wave >> 2;  // BM/2-token half of the token tile

    // 1-D grid remapped for the 8 XCDs (block L runs on XCD L % 8): XCD x
    // takes the tile range [x * per_xcd, (x+1) * per_xcd), walked in groups
    // of four weight tiles with the weight tile fastest, so the ~32 blocks
    // resident on an XCD share 4 weight tiles and 8 token tiles through its L2.
    const int64_t mtiles = (a.rows + BM - 1) / BM;
    const int64_t ntiles = (a.n + C::BN - 1) / C::BN;
    const int64_t total = mtiles * ntiles * a.splits;
    const int64_t per_xcd = (total + 7) / 8;
    const int64_t lin = blockIdx.x;
    const int64_t tl = (lin % 8) * per_xcd + lin / 8;
    if (tl >= total)
        return;
    constexpr int64_t G = 4;
    const int s = (int)(tl / (mtiles * ntiles));
    const int64_t rr = tl % (mtiles * ntiles);
    const int64_t chunk = rr / (G * mtiles);
    const int64_t within = rr % (G * mtiles);
    const int64_t gc = ntiles - chunk * G < G ? ntiles - chunk * G : G;
    const int ntile = (int)(chunk * G + within % gc);
    const int64_t e = 0;
    const int64_t mrow0 = (within / gc) * BM;
    const int64_t mrow1 = mrow0 + BM < a.rows ? mrow0 + BM : a.rows;
    const int64_t n0 = (int64_t)ntile * C::BN;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const int64_t ntk = ke > kb0 ? (ke - kb0 + C::BK - 1) / C::BK : 0;

    // ---- per-lane DMA state (fixed across stages) ------------------------------
    // weight instruction j: lines 8j .. 8j+7, lane -> line 8j + lane/8, slot
    // lane%8 = chunk c ^ swz8(line): K chunk c & 3 of the upper bytes (full
    // mode c < 4, fast mode any c) or of the residual (full mode c >= 4).
    // Stage t of the lane's piece starts at p0 + 64 t, or for a residual piece
    // past the row range's chunk boundary (stages >= tsw) at p1 + 64 t.
    const uint8_t *p0[C::NW], *p1[C::NW];
    int64_t wlog[C::NW];
    int wlim[C::NW], tsw[C::NW];
    bool lo[C::NW], ok0[C::NW], ok1[C::NW];
#pragma unroll
    for (int jj = 0; jj < C::NW; ++jj) {
        const int j = wave * C::NW + jj;
        const int line = 8 * j + (lane >> 3);
        const int c = (lane & 7) ^ swz8(line);
        const int r = MODE == MODE_FULL ? line : (2 * (line >> 4) + (c >> 2)) * 16 + (line & 15);
        int64_t nr = n0 + r;
        nr = nr < a.n ? nr : a.n - 1;
        const int wel = (c & 3) * 16;
        const int64_t wl = (e * a.n + nr) * a.k;
        lo[jj] = MODE == MODE_FULL && c >= 4;
        p0[jj] = p1[jj] = a.hi + wl + kb0 + wel;
        wlim[jj] = (int)(ke - kb0 - wel);
        wlog[jj] = wl + kb0 + wel;
        tsw[jj] = 0;
        ok0[jj] = ok1[jj] = true;
        if (lo[jj]) {
            p0[jj] = p1[jj] = a.res.pool;
            ok0[jj] = ok1[jj] = false;
            if (RANGE && ke > kb0) {
                const RangeResidual rr = range_residual(a.res, wl + kb0, wl + ke);
                p0[jj] = a.res.pool + rr.delta0 + wlog[jj];
                p1[jj] = a.res.pool + rr.delta1 + wlog[jj];
                ok0[jj] = rr.ok0;
                ok1[jj] = rr.ok1;
                const int64_t d = rr.bnd - wlog[jj];  // first stage at or past the chunk boundary
                tsw[jj] = d <= 0 ? 0 : (int)((d + C::BK - 1) / C::BK);
            }
        }
    }
    // token instruction j: rows 8j .. 8j+7, lane -> row 8j + lane/8, slot
    // lane%8.  The wave's rows are 8 apart from one instruction to the next,
    // so one row pointer serves them all (rows past the tile's last token
    // load zeros); the swizzled K offset alternates with the instruction's
    // parity.
    const int xr0 = 8 * wave * C::NX + (lane >> 3);
    const uint16_t *xp0 = static_cast<const uint16_t *>(a.x) + (mrow0 + xr0) * a.k + kb0;
    int xel[2];
#pragma unroll
    for (int par = 0; par < 2; ++par)
        xel[par] = tok_chunk((lane & 7) ^ swz8(xr0 + 8 * par)) * 8;
    const int64_t t_full = (ke - kb0) / C::BK;  // stages entirely inside the K range
    // Serpentine K walk: odd groups of four weight tiles walk K backwards.
    // An XCD runs its groups one after another over the same token tiles, so
    // a group then starts on the token stages the previous one read last,
    // still in that XCD's L2 (MI355X, against the per-group rotation the
    // wide-row GEMM uses: gate+up at 2048 tokens 0.94x the time in fast
    // mode, 0.99x in full mode, 0.98x at 8192 tokens).
    const bool rev = (ntile >> 2) & 1;
    auto tk = [&](int64_t t) {
        return t < ntk ? (rev ? ntk - 1 - t : t) : t;
    };

    auto issue_w = [&](int64_t t) {
        uint8_t *st = smem + (int)(t % WS) * C::W_SLOT;
        const int64_t tr = tk(t);
        const bool masked = tr >= t_full;
        const int64_t off = tr * C::BK;
#pragma unroll
        for (int jj = 0; jj < C::NW; ++jj) {
            const int j = wave * C::NW + jj;
            const bool ok = !masked || off < wlim[jj];
            const void *src = g_zero16;
            if (!lo[jj] || RANGE) {
                const bool second = tr >= tsw[jj];
                if (ok && (second ? ok1[jj] : ok0[jj]))
                    src = (second ? p1[jj] : p0[jj]) + off;
            } else {
                const int64_t o = residual_offset(a.res, wlog[jj] + (ok ? off : 0));
                if (ok && o >= 0)
                    src = a.res.pool + o;
            }
            dma16(src, st + j * 1024);
        }
    };
    auto issue_x = [&](int64_t t) {
        uint8_t *st = smem + C::X_BASE + (int)(t % XS) * C::X_SLOT;
        const int64_t tr = tk(t);
        const bool masked = tr >= t_full;
        const int64_t off = tr * C::BK;
#pragma unroll
        for (int jj = 0; jj < C::NX; ++jj) {
            const int j = wave * C::NX + jj;
            const int xe = xel[jj & 1];
            const bool ok = (mrow0 + xr0 + 8 * jj < mrow1) &&
                            (!masked || off + xe < ke - kb0);
            dma16(ok ? (const void *)(xp0 + (int64_t)(8 * jj) * a.k + off + xe)
                     : (const void *)g_zero16,
                  st + j * 1024);
        }
    };

    f32x4 acc[4][C::MT];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < C::MT; ++j)
            acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // fragment offsets: the swizzles depend on the low bits of the line or
    // row only, which every 16-line tile shares with the lane's li.  Row
    // tile nt (0-3) of the wave: full mode upper bytes at aoff + 2048 nt,
    // residual 64 bytes further in the swizzled line (aoff_lo); fast mode at
    // aoff_f[nt & 1] + 2048 (nt >> 1).  Token tile mt at boff[s] + 2048 mt.
    const int aoff = (wn * 64 + li) * 128 + ((lg ^ swz8(li)) << 4);
    const int aoff_lo = (wn * 64 + li) * 128 + (((4 + lg) ^ swz8(li)) << 4);
    int aoff_f[2];
#pragma unroll
    for (int q = 0; q < 2; ++q)
        aoff_f[q] = (wn * 32 + li) * 128 + (((4 * q + lg) ^ swz8(li)) << 4);
    int boff[2];
#pragma unroll
    for (int sidx = 0; sidx < 2; ++sidx)
        boff[sidx] = (wm * C::TM + li) * 128 + (((lg + 4 * sidx) ^ swz8(li)) << 4);

#pragma unroll
    for (int u = -(WS - 1); u < 0; ++u) {
        if (u + XS - 1 >= 0)
            issue_x(u + XS - 1);
        if (u + WS - 1 >= 0)
            issue_w(u + WS - 1);
    }
    for (int64_t t = 0; t < ntk; ++t) {
        DPS_WAIT_VMCNT(C::OUTSTANDING);  // tokens t and weights t have landed
        stage_barrier();
        const uint8_t *st = smem + (int)(t % WS) * C::W_SLOT;
        const uint8_t *xs = smem + C::X_BASE + (int)(t % XS) * C::X_SLOT;
        // the wave's four weight row tiles are read and merged once per
        // stage and stay in registers (both MFMA steps); the token fragments
        // stream one 16-token tile at a time, the next read while this one's
        // MFMAs run
        half8 av[2][4];
        {
            u32x4 hv[4], lv[4];
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                lv[nt] = u32x4{0u, 0u, 0u, 0u};
                if (MODE == MODE_FULL) {
                    hv[nt] = *reinterpret_cast<const u32x4 *>(st + aoff + nt * 2048);
                    lv[nt] = *reinterpret_cast<const u32x4 *>(st + aoff_lo + nt * 2048);
                } else {
                    hv[nt] = *reinterpret_cast<const u32x4 *>(st + aoff_f[nt & 1] + (nt >> 1) * 2048);
                }
            }
            // the next stages' DMA goes out while the fragment reads are in flight
            issue_x(t + XS - 1);
            issue_w(t + WS - 1);
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                av[0][nt] = weight8<MODE, ENC>(hv[nt].x, hv[nt].y, lv[nt].x, lv[nt].y);
                av[1][nt] = weight8<MODE, ENC>(hv[nt].z, hv[nt].w, lv[nt].z, lv[nt].w);
            }
        }
        half8 bv[2][2];
        auto read_b = [&](int buf, int mt) {
#pragma unroll
            for (int sidx = 0; sidx < 2; ++sidx)
                bv[buf][sidx] =
                    as_half8(*reinterpret_cast<const u32x4 *>(xs + boff[sidx] + mt * 2048));
        };
        read_b(0, 0);
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) {
            __builtin_amdgcn_sched_barrier(0);
            if (mt + 1 < C::MT)
                read_b((mt + 1) & 1, mt + 1);
#pragma unroll
            for (int sidx = 0; sidx < 2; ++sidx)
#pragma unroll
                for (int nt = 0; nt < 4; ++nt)
                    acc[nt][mt] = mfma16x16x32(av[sidx][nt], bv[mt & 1][sidx], acc[nt][mt]);
        }
    }
    DPS_WAIT_VMCNT(0);  // no DMA may still target this block's LDS when it exits

#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) {
        const int64_t m = mrow0 + wm * C::TM + mt * 16 + li;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
            store_tile_out(a, s, m, n0 + wn * 64 + nt * 16 + lg * 4, acc[nt][mt], mrow1);
    }
}

int64_t token_tiles(int64_t rows, int64_t experts, bool grouped, int bm = BM)
{
    return grouped ? (rows + bm - 1) / bm + experts : (rows + bm - 1) / bm;
}

}  // namespace

int gemm_rows_per_block(int variant)
{
    return (variant == GEMM_G3_256x256 || variant == GEMM_G3_256x128 ||
            variant == GEMM_G5_256x256)
               ? 256
               : 128;
}
int gemm_tokens_per_block(int variant)
{
    switch (variant) {
    case GEMM_G3_256x256: return 256;
    case GEMM_G5_256x256: return 256;
    case GEMM_G4S_128x64: return 64;
    case GEMM_G4_128x32: return 32;
    default: return 128;
    }
}

namespace {

// dense calls: a 1-D grid, padded to a multiple of the 8 XCDs
dim3 dense_grid(int64_t tiles)
{
    return dim3((unsigned)((tiles + 7) / 8 * 8), 1, 1);
}

template <int ENC, int BN_, int BM_, int WN, int WM, int WS, int XS, bool DW>
hipError_t launch_g3(const GemmArgs &a, const LinearPlan &plan, hipStream_t stream)
{
    const int64_t nt = (a.n + BN_ - 1) / BN_;
    const dim3 grid = a.offsets ? dim3((unsigned)(nt * plan.splits),
                                       (unsigned)token_tiles(a.rows, a.experts, true, BM_), 1)
                                : dense_grid(nt * plan.splits * ((a.rows + BM_ - 1) / BM_));
    // grouped calls on the 256 x 128 tile take up to 16 tail rows per expert
    constexpr int TL = DW && BM_ == 128 ? 16 : 0;
    if (TL > 0 && a.offsets)
        hipLaunchKernelGGL((gemm3_kernel<ENC, BN_, BM_, WN, WM, WS, XS, DW, TL>), grid,
                           dim3(WN * WM * 64 + (DW ? 256 : 0)), 0, stream, a);
    else
        hipLaunchKernelGGL((gemm3_kernel<ENC, BN_, BM_, WN, WM, WS, XS, DW>), grid,
                           dim3(WN * WM * 64 + (DW ? 256 : 0)), 0, stream, a);
    return hipGetLastError();
}

template <int ENC>
hipError_t launch_g3_variant(const GemmArgs &a, const LinearPlan &plan, hipStream_t stream)
{
    switch (plan.variant) {
    case GEMM_G3_256x256: return launch_g3<ENC, 256, 256, 2, 4, 3, 2, false>(a, plan, stream);
    case GEMM_G3_256x128: return launch_g3<ENC, 256, 128, 4, 2, 3, 3, true>(a, plan, stream);
    default: return hipErrorInvalidValue;
    }
}

// Grouped calls on the 128-token tile with DMA waves take up to 16 tail rows
// per expert into its last tile (gemm4_kernel, block_rows): an expert of
// 129-144 rows reads its weights once, not twice.
template <int MODE, int ENC, int BM, int WS, int XS, bool SPEC>
hipError_t launch_g4(const GemmArgs &a, const LinearPlan &plan, bool grouped, hipStream_t stream)
{
    const int64_t nt = (a.n + 127) / 128;
    const dim3 grid = grouped ? dim3((unsigned)(nt * plan.splits),
                                     (unsigned)token_tiles(a.rows, a.experts, true, BM), 1)
                              : dense_grid(nt * plan.splits * ((a.rows + BM - 1) / BM));
    const dim3 block(SPEC ? 768 : 512);
    // every mode and encoding fits the tail's 16 registers within the 168
    // that three waves per SIMD allow (E4M3 full mode since its conversion-
    // based merge; the bit-move merge spilled)
    constexpr int TL = SPEC && BM == 128 ? 16 : 0;
    if (MODE == MODE_FULL && plan.range_addr) {
        if (TL > 0 && grouped)
            hipLaunchKernelGGL((gemm4_kernel<MODE, ENC, BM, WS, XS, true, SPEC, TL>), grid, block,
                               0, stream, a);
        else
            hipLaunchKernelGGL((gemm4_kernel<MODE, ENC, BM, WS, XS, true, SPEC>), grid, block, 0,
                               stream, a);
    } else {
        if (TL > 0 && grouped)
            hipLaunchKernelGGL((gemm4_kernel<MODE, ENC, BM, WS, XS, false, SPEC, TL>), grid,
                               block, 0, stream, a);
        else
            hipLaunchKernelGGL((gemm4_kernel<MODE, ENC, BM, WS, XS, false, SPEC>), grid, block,
                               0, stream, a);
    }
    return hipGetLastError();
}

template <int MODE, int ENC, int BM, int WS, int XS>
hipError_t launch_g5(const GemmArgs &a, const LinearPlan &plan, bool grouped, hipStream_t stream)
{
    if (grouped)  // dense calls only
        return hipErrorInvalidValue;
    const dim3 grid = dense_grid((a.n + 255) / 256 * plan.splits * ((a.rows + BM - 1) / BM));
    if (MODE == MODE_FULL && plan.range_addr)
        hipLaunchKernelGGL((gemm5_kernel<MODE, ENC, BM, WS, XS, true>), grid, dim3(512), 0,
                           stream, a);
    else
        hipLaunchKernelGGL((gemm5_kernel<MODE, ENC, BM, WS, XS, false>), grid, dim3(512), 0,
                           stream, a);
    return hipGetLastError();
}

// (token tile, weight slots, token slots) per mode, each within 160 KiB:
// weights want depth (HBM), tokens at least a second slot ahead where it fits
template <int MODE, int ENC>
hipError_t launch_g4_variant(const GemmArgs &a, const LinearPlan &plan, bool grouped,
                             hipStream_t stream)
{
    if constexpr (MODE == MODE_FULL) {
        switch (plan.variant) {
        case GEMM_G4_128x32: return launch_g4<MODE, ENC, 32, 4, 4, false>(a, plan, grouped, stream);
        case GEMM_G4S_128x128: return launch_g4<MODE, ENC, 128, 3, 2, true>(a, plan, grouped, stream);
        case GEMM_G4S_128x64: return launch_g4<MODE, ENC, 64, 4, 2, true>(a, plan, grouped, stream);
        case GEMM_G5_256x256: return launch_g5<MODE, ENC, 256, 3, 2>(a, plan, grouped, stream);
        default: return hipErrorInvalidValue;
        }
    } else {
        switch (plan.variant) {
        case GEMM_G4_128x32: return launch_g4<MODE, ENC, 32, 8, 4, false>(a, plan, grouped, stream);
        case GEMM_G4S_128x128: return launch_g4<MODE, ENC, 128, 4, 3, true>(a, plan, grouped, stream);
        case GEMM_G4S_128x64: return launch_g4<MODE, ENC, 64, 6, 4, true>(a, plan, grouped, stream);
        case GEMM_G5_256x256: return launch_g5<MODE, ENC, 256, 4, 3>(a, plan, grouped, stream);
        default: return hipErrorInvalidValue;
        }
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
    a.rotate = p.k % 4096 == 0;
    const bool grouped = p.offsets != nullptr;
    if (p.enc == ENC_E4M3)
        return p.mode == MODE_FULL ? launch_g4_variant<MODE_FULL, ENC_E4M3>(a, plan, grouped, stream)
                                   : launch_g4_variant<MODE_FAST, ENC_E4M3>(a, plan, grouped, stream);
    return p.mode == MODE_FULL ? launch_g4_variant<MODE_FULL, ENC_E5M2>(a, plan, grouped, stream)
                               : launch_g4_variant<MODE_FAST, ENC_E5M2>(a, plan, grouped, stream);
}

hipError_t launch_gemm_fp8(int enc, const uint8_t *xq, const float *scale, const int32_t *offsets,
                           int64_t m, int64_t experts, int64_t n, int64_t k, const uint8_t *hi,
                           uint16_t *y, const LinearPlan &plan, float *partial, hipStream_t stream)
{
    GemmArgs a;
    a.x = xq;
    a.offsets = offsets;
    a.rows = m;
    a.experts = experts;
    a.hi = hi;
    a.res = ResidualView{nullptr, nullptr, 0, 0, 0};
    a.n = n;
    a.k = k;
    a.ksplit = plan.ksplit;
    a.splits = plan.splits;
    a.y = y;
    a.partial = partial;
    a.scale = scale;
    a.rotate = 0;
    return enc == ENC_E4M3 ? launch_g3_variant<ENC_E4M3>(a, plan, stream)
                           : launch_g3_variant<ENC_E5M2>(a, plan, stream);
}

}  // namespace dps
