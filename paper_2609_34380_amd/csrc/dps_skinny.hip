// dps_skinny.hip -- decode-shaped nested linear (few activation rows), gfx950.
//
// Y = X . W^T with W read straight from HBM into registers, merged there
// (full mode) or zero-extended (fast mode) into FP16 operands, and fed to
// v_mfma_f32_16x16x32_f16 with the weights as the A operand (16 weight rows
// per tile) and the activations as the B operand (16 tokens per tile, rows
// past the end read as zero).  The op is bound by the weight stream, so:
//   - every weight byte is loaded exactly once, in 16-byte vectors, by one
//     lane; a wave covers 16 rows x 64 bytes per load instruction;
//   - the K dimension is cut into `splits` ranges (grid.y) so that enough
//     waves stream concurrently; each range writes fp32 partials that a
//     second kernel sums in a fixed order (deterministic, no atomics);
//   - each lane's residual bytes for one row and one K range fall into at
//     most two chunks, resolved once before the loop (RANGE), or the chunk
//     table is read per vector when a range is longer than a chunk.
// Within one 64-element K block the lane group g = lane/16 holds elements
// 16g .. 16g+15 of its row; the first MFMA takes the low 8, the second the
// high 8.  A and B use the same assignment, so the contraction is complete.
#include "dps_internal.h"

namespace dps {

namespace {

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
};

template <int MODE, int RT, int MT, int U, int WPG, bool RANGE>
__global__ __launch_bounds__(WPG * 64) void skinny_kernel(SkinnyArgs a)
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
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
        return;
    const int64_t nb = ((int64_t)blockIdx.x * WPG + wave) * (16 * RT);
    if (nb >= a.n)
        return;
    const int s = blockIdx.y;
    const int64_t kb0 = (int64_t)s * a.ksplit;
    const int64_t ke = kb0 + a.ksplit < a.k ? kb0 + a.ksplit : a.k;

    const uint8_t *hrow[RT];
    int64_t lrow[RT];
    bool rok[RT];
    RangeResidual rr[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const int64_t nr = nb + rt * 16 + li;
        rok[rt] = nr < a.n;
        lrow[rt] = ((int64_t)e * a.n + nr) * a.k;
        hrow[rt] = a.hi + lrow[rt];
        if (MODE == MODE_FULL && RANGE) {
            rr[rt].ok0 = rr[rt].ok1 = false;
            rr[rt].delta0 = rr[rt].delta1 = 0;
            rr[rt].bnd = 0;
            if (rok[rt] && ke > kb0)
                rr[rt] = range_residual(a.res, lrow[rt] + kb0, lrow[rt] + ke);
        }
    }

    for (int64_t mg = row0; mg < row1; mg += 16 * MT) {
        f32x4 acc[RT][MT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                acc[rt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

        const uint16_t *xrow[MT];
        bool xok[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int64_t m = mg + mt * 16 + li;
            xok[mt] = m < row1;
            xrow[mt] = a.x + m * a.k;
        }

        for (int64_t kb = kb0; kb < ke; kb += 64 * U) {
            u32x4 wh[U][RT], wl[U][RT], xv[U][MT][2];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t kk = kb + u * 64 + lg * 16;
                const bool kin = kk < ke;
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    const u32x4 z = {0u, 0u, 0u, 0u};
                    wh[u][rt] = z;
                    wl[u][rt] = z;
                    if (rok[rt] && kin) {
                        wh[u][rt] = load16(hrow[rt] + kk);
                        if (MODE == MODE_FULL)
                            wl[u][rt] = RANGE ? load_lo_range(a.res, rr[rt], lrow[rt] + kk)
                                              : load_lo_lookup(a.res, lrow[rt] + kk);
                    }
                }
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const u32x4 z = {0u, 0u, 0u, 0u};
                    xv[u][mt][0] = z;
                    xv[u][mt][1] = z;
                    if (xok[mt] && kin) {
                        xv[u][mt][0] = load16(xrow[mt] + kk);
                        xv[u][mt][1] = load16(xrow[mt] + kk + 8);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    const u32x4 h = wh[u][rt];
                    const u32x4 l = MODE == MODE_FULL ? wl[u][rt] : u32x4{0u, 0u, 0u, 0u};
                    const half8 a0 = merge8(h.x, h.y, l.x, l.y);
                    const half8 a1 = merge8(h.z, h.w, l.z, l.w);
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        acc[rt][mt] = mfma16x16x32(a0, as_half8(xv[u][mt][0]), acc[rt][mt]);
                        acc[rt][mt] = mfma16x16x32(a1, as_half8(xv[u][mt][1]), acc[rt][mt]);
                    }
                }
            }
        }

        // lane holds D[4*lg + r][li]: weight rows n0..n0+3 of token m
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const int64_t n0 = nb + rt * 16 + lg * 4;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const int64_t m = mg + mt * 16 + li;
                if (m >= row1 || n0 >= a.n)
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

// Tile variants: rows per wave = 16 * RT, K elements per batch = 64 * U.
struct SkinnyVariant {
    int rt, u, wpg;
};
constexpr SkinnyVariant kVariants[] = {{2, 4, 4}, {1, 4, 4}, {2, 2, 4}, {1, 8, 4}};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);

template <int MODE, int RT, int MT, int U, int WPG>
hipError_t launch_t(const SkinnyArgs &args, const LinearPlan &plan, int64_t experts,
                    hipStream_t stream)
{
    const int64_t rows_per_block = (int64_t)WPG * RT * 16;
    dim3 grid((unsigned)((args.n + rows_per_block - 1) / rows_per_block), (unsigned)plan.splits,
              (unsigned)experts);
    if (plan.range_addr)
        hipLaunchKernelGGL((skinny_kernel<MODE, RT, MT, U, WPG, true>), grid, dim3(WPG * 64), 0,
                           stream, args);
    else
        hipLaunchKernelGGL((skinny_kernel<MODE, RT, MT, U, WPG, false>), grid, dim3(WPG * 64), 0,
                           stream, args);
    return hipGetLastError();
}

template <int MODE, int MT>
hipError_t launch_mt(const SkinnyArgs &args, const LinearPlan &plan, int64_t experts,
                     hipStream_t stream)
{
    switch (plan.variant) {
    case 0: return launch_t<MODE, 2, MT, 4, 4>(args, plan, experts, stream);
    case 1: return launch_t<MODE, 1, MT, 4, 4>(args, plan, experts, stream);
    case 2: return launch_t<MODE, 2, MT, 2, 4>(args, plan, experts, stream);
    case 3: return launch_t<MODE, 1, MT, 8, 4>(args, plan, experts, stream);
    default: return hipErrorInvalidValue;
    }
}

template <int MODE>
hipError_t launch_mode(const SkinnyArgs &args, const LinearPlan &plan, int mt, int64_t experts,
                       hipStream_t stream)
{
    switch (mt) {
    case 1: return launch_mt<MODE, 1>(args, plan, experts, stream);
    case 2: return launch_mt<MODE, 2>(args, plan, experts, stream);
    default: return launch_mt<MODE, 4>(args, plan, experts, stream);
    }
}

}  // namespace

int skinny_variant_count() { return kNumVariants; }
int skinny_rows_per_block(int variant)
{
    return kVariants[variant].wpg * kVariants[variant].rt * 16;
}
int skinny_k_per_batch(int variant) { return kVariants[variant].u * 64; }

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
    // tokens per pass: 16 * mt; grouped calls loop over passes per expert
    int mt = 4;
    if (!p.offsets)
        mt = p.rows <= 16 ? 1 : (p.rows <= 32 ? 2 : 4);
    return p.mode == MODE_FULL ? launch_mode<MODE_FULL>(args, plan, mt, p.experts, stream)
                               : launch_mode<MODE_FAST>(args, plan, mt, p.experts, stream);
}

}  // namespace dps
