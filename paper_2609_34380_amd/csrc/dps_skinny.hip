// dps_skinny.hip -- decode-shaped nested linear (up to 64 activation rows per
// pass), gfx950.
//
// Y = X . W^T with W streamed from HBM straight into registers with
// nontemporal 16-byte loads, merged there (full mode) or zero-extended (fast
// mode) into FP16 operands and fed to v_mfma_f32_16x16x32_f16 with the weights
// as the A operand (16 weight rows per tile) and the activations as the B
// operand (16 tokens per tile).  The op is bound by the weight stream:
//   - every weight byte is loaded once, by one lane, in a 16-byte vector; a
//     wave covers 16 rows x 64 bytes per load instruction;
//   - weight batches are ping-ponged: the loads of batch b+1 are in flight
//     while batch b is multiplied;
//   - the block's slice of X ([rows][K range], FP16) is staged once in LDS
//     and read back as B operands, so activations cost no global traffic in
//     the loop and no registers across it;
//   - K is cut into `splits` ranges (grid.y) so that enough waves stream at
//     once; each range writes fp32 partials that a second kernel sums in a
//     fixed order (deterministic, no atomics);
//   - a lane's residual bytes for one row and one K range fall into at most
//     two chunks, resolved once before the loop (RANGE), or the chunk table
//     is read per vector when a range is longer than a chunk.
// Within one 64-element K block, lane group g = lane/16 holds elements
// 16g .. 16g+15 of its row; the first MFMA takes the low 8, the second the
// high 8.  A and B use the same assignment, so the contraction is complete.
#include "dps_internal.h"

namespace dps {

namespace {

constexpr int kWaves = 4;  // waves per block; each owns 16 * RT weight rows

struct SkinnyArgs {
    const uint16_t *x;
    const int32_t *offsets;
    int64_t rows;
    const uint8_t *hi;
    ResidualView res;
    int64_t n, k, ksplit;
    uint16_t *y;
    float *partial;
    int splits;
    int x_rows;    // X rows staged in LDS per pass (<= 16 * MT)
};

__device__ __forceinline__ u32x4 load_nt(const void *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

// v if keep, else zero -- as a bitwise mask, so the compiler keeps the load
// unconditional instead of turning a select of a load into a branch.
__device__ __forceinline__ u32x4 select16(bool keep, u32x4 v)
{
    const uint32_t m = 0u - (uint32_t)keep;
    return v & u32x4{m, m, m, m};
}

// Per-lane row state for the weight stream.  Every load below is issued
// unconditionally: lanes whose row, K position or residual chunk is out of
// range read an always-valid address instead (safe_*) and zero the value
// with a select.  Branch-free loads let the compiler wait only for the batch
// it is about to multiply while the next batch stays in flight.
template <int RT>
struct RowState {
    const uint8_t *hrow[RT];   // upper-byte row base (clamped to row 0 if beyond n)
    int64_t lrow[RT];          // logical residual offset of the row
    bool rok[RT];
    RangeResidual rr[RT];
};

template <int MODE, int RT, int U, bool RANGE>
struct WBatch {
    u32x4 h[U][RT];
    u32x4 l[MODE == MODE_FULL ? U : 1][RT];

    // Loads the batch starting at K position kb; `live` false loads a dummy
    // (cached) vector per lane and yields zeros.
    __device__ __forceinline__ void load(const RowState<RT> &st, const ResidualView &res,
                                         int64_t kb, int64_t ke, int64_t klast, bool live, int lg)
    {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t kk = kb + u * 64 + lg * 16;
            const bool kin = live && kk < ke;
            const int64_t ks = kin ? kk : klast;
#pragma unroll
            for (int rt = 0; rt < RT; ++rt) {
                const bool ok = kin && st.rok[rt];
                h[u][rt] = select16(ok, load_nt(st.hrow[rt] + ks));
                if (MODE == MODE_FULL) {
                    const int64_t li = st.lrow[rt] + ks;
                    if (RANGE) {
                        const RangeResidual &r = st.rr[rt];
                        const bool second = li >= r.bnd;
                        const bool cok = second ? r.ok1 : r.ok0;
                        const int64_t d = second ? r.delta1 : r.delta0;
                        const int64_t off = cok ? d + li : 0;
                        l[u][rt] = select16(ok && cok, load_nt(res.pool + off));
                    } else {
                        const int64_t off = residual_offset(res, li);
                        l[u][rt] = select16(ok && off >= 0, load_nt(res.pool + (off >= 0 ? off : 0)));
                    }
                }
            }
        }
    }
};

template <int MODE, int ENC, int RT, int MT, int U, bool RANGE>
__device__ __forceinline__ void compute_batch(const WBatch<MODE, RT, U, RANGE> &w,
                                              const uint16_t *xs, int xpitch, int xrow_last,
                                              int64_t kb, int64_t kb0, int64_t ke,
                                              const bool *xok, int li, int lg,
                                              f32x4 (&acc)[RT][MT])
{
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t kk = kb + u * 64 + lg * 16;
        const bool kin = kk < ke;
        const int64_t kc = (kin ? kk : kb0) - kb0;
        half8 b0[MT], b1[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const bool ok = xok[mt] && kin;
            const int r = ok ? mt * 16 + li : xrow_last;
            const uint16_t *src = xs + r * xpitch + kc;
            b0[mt] = as_half8(select16(ok, *reinterpret_cast<const u32x4 *>(src)));
            b1[mt] = as_half8(select16(ok, *reinterpret_cast<const u32x4 *>(src + 8)));
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const u32x4 h = w.h[u][rt];
            const u32x4 l = MODE == MODE_FULL ? w.l[u][rt] : u32x4{0u, 0u, 0u, 0u};
            const half8 a0 = weight8<MODE, ENC>(h.x, h.y, l.x, l.y);
            const half8 a1 = weight8<MODE, ENC>(h.z, h.w, l.z, l.w);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                acc[rt][mt] = mfma16x16x32(a0, b0[mt], acc[rt][mt]);
                acc[rt][mt] = mfma16x16x32(a1, b1[mt], acc[rt][mt]);
            }
        }
    }
}

template <int MODE, int ENC, int RT, int MT, int U, bool RANGE>
__global__ __launch_bounds__(kWaves * 64) void skinny_kernel(SkinnyArgs a)
{
    extern __shared__ __attribute__((aligned(16))) uint16_t xs[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 15;
    const int lg = lane >> 4;
    const int e = blockIdx.z;

    int64_t row0 = 0, row1 = a.rows;
    if (a.offsets) {
        const int64_t o0 = a.offsets[e], o1 = a.offsets[e + 1];
        row0 = o0 < 0 ? 0 : (o0 > a.rows ? a.rows : o0);
        row1 = o1 < row0 ? row0 : (o1 > a.rows ? a.rows : o1);
    }
    if (row0 >= row1)
        return;  // uniform across the block
    const int64_t nb = ((int64_t)blockIdx.x * kWaves + wave) * (16 * RT);
    const bool active = nb < a.n;  // whole wave has rows (no early return: barriers below)
    const int s = blockIdx.y;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const int64_t klen = ke > kb0 ? ke - kb0 : 0;
    const int xpitch = (int)a.ksplit + 8;

    RowState<RT> st;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int64_t nr = nb + rt * 16 + li;
        st.rok[rt] = nr < a.n;
        st.lrow[rt] = ((int64_t)e * a.n + (st.rok[rt] ? nr : 0)) * a.k;
        st.hrow[rt] = a.hi + st.lrow[rt];
        st.rr[rt].ok0 = st.rr[rt].ok1 = false;
        st.rr[rt].delta0 = st.rr[rt].delta1 = 0;
        st.rr[rt].bnd = 0;
        if (MODE == MODE_FULL && RANGE && klen > 0)
            st.rr[rt] = range_residual(a.res, st.lrow[rt] + kb0, st.lrow[rt] + ke);
    }
    const int64_t klast = klen > 0 ? ke - 16 : 0;  // an in-range K position for dummy loads

    for (int64_t mg = row0; mg < row1; mg += a.x_rows) {
        const int64_t mrows = row1 - mg < a.x_rows ? row1 - mg : a.x_rows;
        // ---- stage X[mg .. mg+mrows)[kb0 .. ke) into LDS --------------------------
        __syncthreads();
        {
            const int64_t vpr = klen >> 3;  // 16-byte vectors per row
            const int64_t total = mrows * vpr;
            for (int64_t v = tid; v < total; v += kWaves * 64) {
                const int64_t r = v / vpr;
                const int64_t c = v - r * vpr;
                *reinterpret_cast<u32x4 *>(xs + r * xpitch + c * 8) =
                    load16(a.x + (mg + r) * a.k + kb0 + c * 8);
            }
        }
        __syncthreads();
        if (!active)
            continue;

        f32x4 acc[RT][MT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                acc[rt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
        bool xok[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            xok[mt] = mt * 16 + li < mrows;

        constexpr int KB = 64 * U;
        const int64_t nbatch = (klen + KB - 1) / KB;
        const int xrow_last = (int)mrows - 1;
        WBatch<MODE, RT, U, RANGE> wa, wb;
        wa.load(st, a.res, kb0, ke, klast, nbatch > 0, lg);
        for (int64_t b = 0; b < nbatch; b += 2) {
            wb.load(st, a.res, kb0 + (b + 1) * KB, ke, klast, b + 1 < nbatch, lg);
            compute_batch<MODE, ENC, RT, MT, U, RANGE>(wa, xs, xpitch, xrow_last, kb0 + b * KB, kb0,
                                                  ke, xok, li, lg, acc);
            wa.load(st, a.res, kb0 + (b + 2) * KB, ke, klast, b + 2 < nbatch, lg);
            if (b + 1 < nbatch)
                compute_batch<MODE, ENC, RT, MT, U, RANGE>(wb, xs, xpitch, xrow_last,
                                                      kb0 + (b + 1) * KB, kb0, ke, xok, li, lg,
                                                      acc);
        }

        // lane holds D[4*lg + r][li]: weight rows n0..n0+3 of token m
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const int64_t n0 = nb + rt * 16 + lg * 4;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int64_t m = mg + mt * 16 + li;
                if (mt * 16 + li >= mrows || n0 >= a.n)
                    continue;
                const f32x4 v = acc[rt][mt];
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
        }
    }
}

// ------------------------------------------------------------------------------
// Ring variant: the weight stream goes global -> LDS with direct-to-LDS loads
// (gfx950 global_load_lds_dwordx4) through a private ring of RING stages per
// wave, so many stages are in flight without holding registers.  A stage is
// 16 weight rows x 256 K bytes per plane; each of its DMA instructions reads 4
// rows x 256 contiguous bytes.  Within a row the 16-byte chunk for K offset
// 16c sits at slot c ^ (row % 16), which makes the MFMA-layout reads (16 rows
// at one K offset) hit distinct banks.  X is the only other global traffic and
// is staged before the stream starts, so the wait for stage t is a plain
// vmcnt on this wave's own DMA queue -- no barriers inside the loop.
// ------------------------------------------------------------------------------
constexpr int RING_SK = 256;                    // K bytes per stage and plane
constexpr int RING_STAGE_PLANE = 16 * RING_SK;  // 4 KiB

__device__ __attribute__((aligned(16))) const uint8_t g_zero16_s[16] = {0};

#define DPS_LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))
#define DPS_WAIT_VM(n) \
    __builtin_amdgcn_s_waitcnt(((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8))

template <int MODE, int ENC, int MT, int RING, bool RANGE>
__global__ __launch_bounds__(kWaves * 64) void ring_kernel(SkinnyArgs a)
{
    constexpr int PLANES = MODE == MODE_FULL ? 2 : 1;
    constexpr int STAGE = RING_STAGE_PLANE * PLANES;
    constexpr int NI = 4 * PLANES;  // DMA instructions per stage and wave
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int li = lane & 15;
    const int lg = lane >> 4;
    const int e = blockIdx.z;

    int64_t row0 = 0, row1 = a.rows;
    if (a.offsets) {
        const int64_t o0 = a.offsets[e], o1 = a.offsets[e + 1];
        row0 = o0 < 0 ? 0 : (o0 > a.rows ? a.rows : o0);
        row1 = o1 < row0 ? row0 : (o1 > a.rows ? a.rows : o1);
    }
    if (row0 >= row1)
        return;  // uniform across the block
    const int64_t nb = ((int64_t)blockIdx.x * kWaves + wave) * 16;
    const bool active = nb < a.n;
    const int s = blockIdx.y;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;
    const int64_t klen = ke > kb0 ? ke - kb0 : 0;
    const int xpitch = (int)a.ksplit + 8;  // halfs
    uint16_t *xs = reinterpret_cast<uint16_t *>(lds);
    uint8_t *ring = lds + (((size_t)a.x_rows * xpitch * 2 + 255) & ~(size_t)255) +
                    (size_t)wave * RING * STAGE;

    // DMA sources: instruction j of a stage covers rows 4j .. 4j+3; lane l ->
    // row 4j + l/16, slot l%16, logical 16-byte chunk (l%16) ^ row
    const uint8_t *wsrc[4];
    int64_t wl[4];
    int wchunk[4];
    RangeResidual rr[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int r = 4 * j + (lane >> 4);
        int64_t nr = nb + r;
        nr = nr < a.n ? nr : a.n - 1;
        wl[j] = ((int64_t)e * a.n + nr) * a.k;
        wsrc[j] = a.hi + wl[j];
        wchunk[j] = (lane & 15) ^ r;
        rr[j].ok0 = rr[j].ok1 = false;
        rr[j].delta0 = rr[j].delta1 = 0;
        rr[j].bnd = 0;
        if (MODE == MODE_FULL && RANGE && klen > 0)
            rr[j] = range_residual(a.res, wl[j] + kb0, wl[j] + ke);
    }
    const int64_t nstage = (klen + RING_SK - 1) / RING_SK;

    auto issue = [&](int64_t t) {
        uint8_t *st = ring + (int)(t % RING) * STAGE;
        const bool live = t < nstage;
        const int64_t kt = kb0 + t * RING_SK;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t kk = kt + wchunk[j] * 16;
            const bool ok = live && kk < ke;
            __builtin_amdgcn_global_load_lds(ok ? (const void *)(wsrc[j] + kk)
                                                : (const void *)g_zero16_s,
                                             DPS_LDS_PTR(st + j * 1024), 16, 0, 0);
            if (MODE == MODE_FULL) {
                const int64_t lo = wl[j] + (ok ? kk : kb0);
                const void *src = g_zero16_s;
                if (RANGE) {
                    const bool second = lo >= rr[j].bnd;
                    const bool cok = second ? rr[j].ok1 : rr[j].ok0;
                    const int64_t d = second ? rr[j].delta1 : rr[j].delta0;
                    if (ok && cok)
                        src = a.res.pool + (d + lo);
                } else {
                    const int64_t off = residual_offset(a.res, lo);
                    if (ok && off >= 0)
                        src = a.res.pool + off;
                }
                __builtin_amdgcn_global_load_lds(src, DPS_LDS_PTR(st + RING_STAGE_PLANE + j * 1024),
                                                 16, 0, 0);
            }
        }
    };

    for (int64_t mg = row0; mg < row1; mg += a.x_rows) {
        const int64_t mrows = row1 - mg < a.x_rows ? row1 - mg : a.x_rows;
        // ---- stage X[mg .. mg+mrows)[kb0 .. ke) into LDS (plain loads) -------------
        __syncthreads();
        {
            const int64_t vpr = klen >> 3;
            const int64_t total = mrows * vpr;
            for (int64_t v = tid; v < total; v += kWaves * 64) {
                const int64_t r = v / vpr;
                const int64_t c = v - r * vpr;
                *reinterpret_cast<u32x4 *>(xs + r * xpitch + c * 8) =
                    load16(a.x + (mg + r) * a.k + kb0 + c * 8);
            }
        }
        __syncthreads();
        if (!active)
            continue;

        f32x4 acc[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
        bool xok[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            xok[mt] = mt * 16 + li < mrows;
        const int xrow_last = (int)mrows - 1;

#pragma unroll
        for (int t = 0; t < RING - 1; ++t)
            issue(t);
        for (int64_t t = 0; t < nstage; ++t) {
            DPS_WAIT_VM(NI * (RING - 2));
            const uint8_t *st = ring + (int)(t % RING) * STAGE;
            const int64_t kt = kb0 + t * RING_SK;
#pragma unroll
            for (int q = 0; q < RING_SK / 64; ++q) {
                // lane (li, lg): row li, K chunk 4q + lg of this stage
                const int slot = ((4 * q + lg) ^ li) << 4;
                const u32x4 h = *reinterpret_cast<const u32x4 *>(st + li * RING_SK + slot);
                u32x4 l = {0u, 0u, 0u, 0u};
                if (MODE == MODE_FULL)
                    l = *reinterpret_cast<const u32x4 *>(st + RING_STAGE_PLANE + li * RING_SK + slot);
                const half8 a0 = weight8<MODE, ENC>(h.x, h.y, l.x, l.y);
                const half8 a1 = weight8<MODE, ENC>(h.z, h.w, l.z, l.w);
                const int64_t kk = kt + q * 64 + lg * 16;
                const bool kin = kk < ke;
                const int64_t kc = (kin ? kk : kb0) - kb0;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const bool ok = xok[mt] && kin;
                    const int r = ok ? mt * 16 + li : xrow_last;
                    const uint16_t *src = xs + r * xpitch + kc;
                    const half8 b0 = as_half8(select16(ok, *reinterpret_cast<const u32x4 *>(src)));
                    const half8 b1 =
                        as_half8(select16(ok, *reinterpret_cast<const u32x4 *>(src + 8)));
                    acc[mt] = mfma16x16x32(a0, b0, acc[mt]);
                    acc[mt] = mfma16x16x32(a1, b1, acc[mt]);
                }
            }
            issue(t + RING - 1);
        }
        DPS_WAIT_VM(0);

        // lane holds D[4*lg + r][li]: weight rows n0..n0+3 of token m
        const int64_t n0 = nb + lg * 4;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int64_t m = mg + mt * 16 + li;
            if (mt * 16 + li >= mrows || n0 >= a.n)
                continue;
            const f32x4 v = acc[mt];
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
    }
}

// Register-stream tile variants (rows per wave = 16 * RT, K elements per
// batch = 64 * U); SKINNY_RING streams through the LDS rings instead.
struct SkinnyVariant {
    int rt, u;
};
constexpr SkinnyVariant kVariants[] = {{1, 4}, {2, 2}};

template <int MODE, int ENC, int RT, int MT, int U>
hipError_t launch_t(const SkinnyArgs &args, const LinearPlan &plan, int64_t experts,
                    hipStream_t stream)
{
    const int64_t rows_per_block = (int64_t)kWaves * RT * 16;
    dim3 grid((unsigned)((args.n + rows_per_block - 1) / rows_per_block), (unsigned)plan.splits,
              (unsigned)experts);
    const size_t lds = (size_t)args.x_rows * (size_t)(args.ksplit + 8) * 2;
    if (plan.range_addr)
        hipLaunchKernelGGL((skinny_kernel<MODE, ENC, RT, MT, U, true>), grid, dim3(kWaves * 64),
                           lds, stream, args);
    else
        hipLaunchKernelGGL((skinny_kernel<MODE, ENC, RT, MT, U, false>), grid, dim3(kWaves * 64),
                           lds, stream, args);
    return hipGetLastError();
}

// The rings take half of a gfx950 CU's 160 KiB LDS, so two blocks share a CU.
constexpr int kRingLds = 80 * 1024;

template <int MODE>
constexpr int ring_depth() { return MODE == MODE_FULL ? 2 : 3; }

template <int MODE>
constexpr int ring_bytes()
{
    return kWaves * ring_depth<MODE>() * RING_STAGE_PLANE * (MODE == MODE_FULL ? 2 : 1);
}

template <int MODE, int ENC, int MT>
hipError_t launch_ring(const SkinnyArgs &args, const LinearPlan &plan, int64_t experts,
                       hipStream_t stream)
{
    constexpr int RING = ring_depth<MODE>();
    const size_t xbytes = ((size_t)args.x_rows * (size_t)(args.ksplit + 8) * 2 + 255) & ~(size_t)255;
    const size_t lds = xbytes + ring_bytes<MODE>();
    if (lds > (size_t)kRingLds)
        return hipErrorInvalidValue;
    dim3 grid((unsigned)((args.n + kWaves * 16 - 1) / (kWaves * 16)), (unsigned)plan.splits,
              (unsigned)experts);
    // more than 64 KiB of dynamic LDS needs the per-kernel limit raised once
    if (plan.range_addr) {
        static const hipError_t attr =
            hipFuncSetAttribute((const void *)ring_kernel<MODE, ENC, MT, RING, true>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, kRingLds);
        if (attr != hipSuccess)
            return attr;
        hipLaunchKernelGGL((ring_kernel<MODE, ENC, MT, RING, true>), grid, dim3(kWaves * 64), lds,
                           stream, args);
    } else {
        static const hipError_t attr =
            hipFuncSetAttribute((const void *)ring_kernel<MODE, ENC, MT, RING, false>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, kRingLds);
        if (attr != hipSuccess)
            return attr;
        hipLaunchKernelGGL((ring_kernel<MODE, ENC, MT, RING, false>), grid, dim3(kWaves * 64),
                           lds, stream, args);
    }
    return hipGetLastError();
}

template <int MODE, int ENC, int MT>
hipError_t launch_mt(const SkinnyArgs &args, const LinearPlan &plan, int64_t experts,
                     hipStream_t stream)
{
    switch (plan.variant) {
    case SKINNY_RING: return launch_ring<MODE, ENC, MT>(args, plan, experts, stream);
    case 0: return launch_t<MODE, ENC, 1, MT, 4>(args, plan, experts, stream);
    case 1: return launch_t<MODE, ENC, 2, MT, 2>(args, plan, experts, stream);
    default: return hipErrorInvalidValue;
    }
}

template <int MODE, int ENC>
hipError_t launch_mode(const SkinnyArgs &args, const LinearPlan &plan, int mt, int64_t experts,
                       hipStream_t stream)
{
    switch (mt) {
    case 1: return launch_mt<MODE, ENC, 1>(args, plan, experts, stream);
    case 2: return launch_mt<MODE, ENC, 2>(args, plan, experts, stream);
    default: return launch_mt<MODE, ENC, 4>(args, plan, experts, stream);
    }
}

}  // namespace

int skinny_rows_per_block(int variant)
{
    return variant == SKINNY_RING ? kWaves * 16 : kWaves * kVariants[variant].rt * 16;
}
int skinny_k_per_batch(int variant)
{
    return variant == SKINNY_RING ? RING_SK : kVariants[variant].u * 64;
}
// Largest K range (multiple of the batch) whose X slice fits the block's LDS.
int64_t skinny_max_ksplit(int variant, int mode, int64_t pass_rows)
{
    const int64_t kpb = skinny_k_per_batch(variant);
    int64_t budget = 65536;
    if (variant == SKINNY_RING)
        budget = kRingLds - 256 -
                 (mode == MODE_FULL ? ring_bytes<MODE_FULL>() : ring_bytes<MODE_FAST>());
    const int64_t kmax = (budget / 2 / pass_rows - 8) / kpb * kpb;
    return kmax < kpb ? 0 : kmax;  // 0: this variant cannot hold the X slice
}

// Tokens per pass for a call with `rows` rows in total (dense) or grouped.
int skinny_pass_rows(int64_t rows, bool grouped)
{
    if (grouped)
        return 64;
    return rows <= 16 ? (int)rows : (rows <= 32 ? (int)rows : (int)(rows < 64 ? rows : 64));
}

hipError_t launch_skinny(const LinearProblem &p, const LinearPlan &plan, float *partial,
                         hipStream_t stream)
{
    SkinnyArgs args;
    args.x = p.x;
    args.offsets = p.offsets;
    args.rows = p.rows;
    args.hi = p.hi;
    args.res = p.res;
    args.n = p.n;
    args.k = p.k;
    args.ksplit = plan.ksplit;
    args.y = p.y;
    args.partial = partial;
    args.splits = plan.splits;
    args.x_rows = skinny_pass_rows(p.rows, p.offsets != nullptr);
    const int mt = (args.x_rows + 15) / 16;
    if (p.enc == ENC_E4M3)
        return p.mode == MODE_FULL
                   ? launch_mode<MODE_FULL, ENC_E4M3>(args, plan, mt, p.experts, stream)
                   : launch_mode<MODE_FAST, ENC_E4M3>(args, plan, mt, p.experts, stream);
    return p.mode == MODE_FULL ? launch_mode<MODE_FULL, ENC_E5M2>(args, plan, mt, p.experts, stream)
                               : launch_mode<MODE_FAST, ENC_E5M2>(args, plan, mt, p.experts, stream);
}

}  // namespace dps
