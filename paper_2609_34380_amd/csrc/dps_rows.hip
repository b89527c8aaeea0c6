// dps_rows.hip -- dense nested linear for up to 16 tokens on the matrix cores
// (gfx950).
//
// A call of a few tokens is bound by the weight stream, so this kernel is
// built around the load shape that streams fastest from HBM and around
// whole weight rows per block:
//   - a pipeline stage is 16 weight rows x 1024 K elements: per plane one
//     wave instruction moves 1 KiB of one row (64 lanes x 16 contiguous
//     bytes, measured at 7.2 TB/s from HBM against 5.2 TB/s for 8 rows x
//     128 B), straight into LDS (direct-to-LDS loads) through a ring of
//     stages;
//   - a block owns G groups of 16 rows over the whole K range, so K is never
//     split across blocks: one launch, no partial sums in memory, and G is
//     chosen so that the grid about fills the chip once;
//   - the eight waves split each stage's K range: wave w multiplies the
//     128-element slice [128w, 128w+128) of every stage, its activations
//     held in registers for the whole 1024-element chunk, and keeps one fp32
//     accumulator tile per row group and 16-token tile.  The activation
//     slice of the next chunk streams into a 4 KiB LDS area of the wave with
//     direct-to-LDS loads, like the weights, so every load the kernel issues
//     is counted by the same vector-memory counter and the ring's waits
//     retire exactly what the stage about to be read needs;
//   - at the end the eight slices are summed through LDS in wave order, so
//     the result does not depend on timing, and written as FP16.
// Weights are merged (full mode) or converted (fast mode) into FP16 words in
// registers exactly as in the other matrix-core kernels (Sec. IV-C:
// reconstruction during computation), so fast mode equals full mode over a
// zero residual bit for bit.
//
// LDS layout of a stage slot: plane p (upper bytes, then residual bytes),
// row i (0..15), 1 KiB per row; lane l of the instruction that fills row i
// writes 16-byte position l and loads K chunk l ^ swz(i), so K chunk q of
// row i sits at position q ^ swz(i).  The fragment read of lane (i, g) in
// step pair s2 is chunk 8w + 4 s2 + g of row i (a ds_read_b128 per plane);
// its two 8-byte halves feed two MFMA steps, and the activations are loaded
// with the same K permutation.
#include "dps_internal.h"

namespace dps {

namespace {

constexpr int kRowsKC = 1024;  // K elements per stage

struct RowsArgs {
    const uint16_t *x;  // FP16 [m][k]
    int64_t m;
    const uint8_t *hi;
    ResidualView res;
    uint64_t slots_const;  // res.slots, read through the scalar cache
    int64_t n, k;
    uint16_t *y;  // FP16 [m][n]
    int rotate;   // walk the K chunks starting at (block / 4) mod chunks
};

__device__ __attribute__((aligned(16))) const uint8_t g_rows_zero16[16] = {0};

#define DPS_ROWS_LDS(p) ((__attribute__((address_space(3))) void *)(p))

// s_waitcnt vmcnt(n), the other counters untouched (gfx9 encoding)
#define DPS_ROWS_WAIT_VMCNT(n) \
    __builtin_amdgcn_s_waitcnt(((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8))

// lgkmcnt(0) (the wave's LDS reads and scalar loads are done), then a bare
// barrier; __syncthreads() would also wait for every direct-to-LDS load in
// flight and drain the ring.
__device__ __forceinline__ void rows_barrier()
{
    __builtin_amdgcn_s_waitcnt(0xC07F);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ int rows_swz(int i) { return (i & 15) << 2; }

typedef const __attribute__((address_space(4))) int32_t *const_i32p;

// Ring depth: WS - 2 <= G keeps the activation load of the next chunk
// (issued at the first stage of a chunk) behind the DMA the counter waits
// for, so the waits retire no DMA a later stage could still have overlapped
// (the counter arithmetic is derived at the main loop).  Deeper rings serve
// blocks with more row groups.  Behind the ring, each wave has XB areas of
// XA bytes for its activation slice of one chunk: two where LDS allows
// (the next chunk's slice then streams in while this one is read), else
// one, refilled right after it has been read.
template <int MODE, int NT, int G>
struct RowsConfig {
    static constexpr int PLANES = MODE == MODE_FULL ? 2 : 1;
    static constexpr int SLOT = 16 * kRowsKC * PLANES;  // one stage
    static constexpr int WSMAX = MODE == MODE_FULL ? 4 : 8;
    static constexpr int WS = G + 2 < WSMAX ? G + 2 : WSMAX;
    static constexpr int NI = 2 * PLANES;  // DMA instructions per wave per stage
    static constexpr int RED = 8 * G * NT * 1024;  // slice sums, reusing the ring
    static constexpr int RING = WS * SLOT > RED ? WS * SLOT : RED;
    static constexpr int XL = 4 * NT;              // activation instructions per wave per chunk
    static constexpr int XA = XL * 1024;           // activation area of one wave
    static constexpr int XB = RING + 2 * 8 * XA <= 160 * 1024 ? 2 : 1;
    static constexpr int LDS = RING + XB * 8 * XA;
    static_assert(WS >= 3 && WS - 2 <= G, "ring depth");
    static_assert(LDS <= 160 * 1024, "LDS");
};

// NT: 16-token tiles (tokens <= 16 NT); G: 16-row groups per block; RANGE:
// residual chunks of >= 1 KiB, so that one row piece spans at most two
// chunks (else a per-vector table lookup).
template <int MODE, int ENC, int NT, int G, bool RANGE>
__global__ __launch_bounds__(512) void rows_kernel(RowsArgs a)
{
    using C = RowsConfig<MODE, NT, G>;
    constexpr int SLOT = C::SLOT;
    constexpr int WS = C::WS;
    constexpr int NI = C::NI;
    __shared__ __attribute__((aligned(16))) uint8_t smem[C::LDS];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane & 15;
    const int lg = lane >> 4;
    const int64_t r0 = (int64_t)blockIdx.x * (16 * G);
    const int64_t nkc = (a.k + kRowsKC - 1) / kRowsKC;
    const int64_t nst = nkc * G;  // stage t: chunk step t / G, row group t % G
    // Chunk step c reads K chunk kc(c).  When rows are a multiple of 4 KiB
    // apart, all blocks reading the same chunk at once would hit the same
    // address bits 10-11; starting each group of four blocks at another chunk
    // spreads the stream (MI355X, hidden-4096 set at 8 tokens: gate+up and O
    // 0.81-0.91x the time, QKV 1.03x in full mode; 14 KiB rows lose with it).
    const int64_t rot = a.rotate ? (int64_t)(blockIdx.x >> 2) % nkc : 0;
    auto kc = [&](int64_t c) { return c + rot < nkc ? c + rot : c + rot - nkc; };

    // ---- DMA: wave w fills rows 2w and 2w+1 of the stage's row group, upper
    // bytes then (full mode) residual bytes: NI = 2 or 4 instructions.  Stages
    // past the end load zeros, so that every iteration issues NI.
    auto issue = [&](int64_t t) {
        uint8_t *slot = smem + (int)(t % WS) * SLOT;
        const bool live = t < nst;
        const int64_t c = live ? kc(t / G) : 0;
        const int g = live ? (int)(t % G) : 0;
        int64_t L0[2];
        int64_t sl0[2] = {-1, -1}, sl1[2] = {-1, -1};
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            int64_t row = r0 + 16 * g + 2 * wave + j;
            row = row < a.n ? row : a.n - 1;
            L0[j] = row * a.k + c * kRowsKC;  // wave-uniform
        }
        if (C::PLANES == 2 && RANGE) {
            // the residual slots of both pieces first (scalar loads, one wait)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int64_t c0 = L0[j] >> a.res.log2c;
                const int64_t nc = a.res.n_chunks;
                const int64_t v0 = ((const_i32p)a.slots_const)[c0 < nc ? c0 : nc - 1];
                const int64_t v1 = ((const_i32p)a.slots_const)[c0 + 1 < nc ? c0 + 1 : nc - 1];
                sl0[j] = (c0 < nc && v0 >= 0 && v0 < a.res.n_pool_slots) ? v0 : -1;
                sl1[j] = (c0 + 1 < nc && v1 >= 0 && v1 < a.res.n_pool_slots) ? v1 : -1;
            }
        }
#pragma unroll
        for (int pl = 0; pl < C::PLANES; ++pl)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int ri = 2 * wave + j;
                const int p = lane ^ rows_swz(ri);
                const bool ok = live && c * kRowsKC + 16 * p < a.k;
                const int64_t li16 = L0[j] + 16 * p;
                const void *src = g_rows_zero16;
                if (pl == 0) {
                    if (ok)
                        src = a.hi + li16;
                } else if (RANGE) {
                    const bool second = (li16 >> a.res.log2c) != (L0[j] >> a.res.log2c);
                    const int64_t sv = second ? sl1[j] : sl0[j];
                    if (ok && sv >= 0)
                        src = a.res.pool + ((sv << a.res.log2c) |
                                            (li16 & ((int64_t(1) << a.res.log2c) - 1)));
                } else {
                    const int64_t off = residual_offset(a.res, ok ? li16 : 0);
                    if (ok && off >= 0)
                        src = a.res.pool + off;
                }
                __builtin_amdgcn_global_load_lds(
                    src, DPS_ROWS_LDS(slot + pl * 16 * kRowsKC + ri * kRowsKC), 16, 0, 0);
            }
    };

    // ---- activations of this wave's K slice for chunk step c: instruction q
    // = (s2, h, nt) of lane (j, g) loads X[16 nt + j][kc(c) KC + 16 (8w + 4 s2
    // + g) + 8 h .. +7] (token rows past m repeat row m-1; past K a valid
    // address, the value is cleared when read) into 16-byte position `lane`
    // of 1 KiB piece q of the wave's area, so each lane later reads back
    // exactly its own 16 bytes.
    constexpr int XL = C::XL;
    constexpr int XB = C::XB;
    // the wave's area for chunk c
    auto xarea = [&](int64_t c) {
        return smem + C::RING + ((XB == 2 ? (int)(c & 1) : 0) * 8 + wave) * C::XA;
    };
    auto issue_x = [&](int64_t c, int64_t cbuf) {
        uint8_t *xa = xarea(cbuf);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            int64_t tok = 16 * nt + li;
            tok = tok < a.m ? tok : a.m - 1;
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                const int64_t kk = kc(c) * kRowsKC + 16 * (8 * wave + 4 * s2 + lg);
                const int64_t kv = kk < a.k ? kk : 0;
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    __builtin_amdgcn_global_load_lds(
                        a.x + tok * a.k + kv + 8 * h,
                        DPS_ROWS_LDS(xa + ((s2 * 2 + h) * NT + nt) * 1024), 16, 0, 0);
            }
        }
    };
    // after the wait that retires chunk c's activation loads: registers from
    // the wave's area, with what lies past K cleared
    u32x4 xr[2][2][NT];
    auto read_x = [&](int64_t c) {
        const uint8_t *xa = xarea(c);
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
            const int64_t kk = kc(c) * kRowsKC + 16 * (8 * wave + 4 * s2 + lg);
            const uint32_t msk = 0u - (uint32_t)(kk < a.k);
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    xr[s2][h][nt] = *reinterpret_cast<const u32x4 *>(
                        xa + ((s2 * 2 + h) * NT + nt) * 1024 + lane * 16);
                    xr[s2][h][nt] &= u32x4{msk, msk, msk, msk};
                }
        }
    };

    f32x4 acc[G][NT];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
            acc[g][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    // fragment offsets within a plane of a slot (fixed)
    int foff[2];
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
        foff[s2] = li * kRowsKC + (((8 * wave + 4 * s2 + lg) ^ rows_swz(li)) << 4);

    // Issue order with one area per wave (XB == 1): X(0); DMA of stages
    // 0 .. WS-2; then per stage t = cG + g: wait, barrier, at g = 0 the read
    // of X(c) from the area followed by the load of X(c+1) into it (the last
    // chunk loads its own again), then the DMA of stage t+WS-1 (always NI
    // instructions).  The counter retires in issue order.  The wait for
    // stage t may leave outstanding what was issued after the later of
    // DMA(t) and, at g = 0, X(c):
    //   - DMA(t+1) .. DMA(t+WS-2), issued in earlier iterations: BASE;
    //   - at g = 0, X(c) went out in iteration (c-1)G, ahead of that
    //     iteration's DMA, which is DMA(t+1) when WS = G+2 and DMA(t) or an
    //     earlier one otherwise (WS - 2 <= G), so BASE retires X(c) too;
    //   - at 1 <= g <= WS-2, X(c+1) (iteration cG) followed DMA(t)
    //     (iteration t-WS+1 < cG): BASE + XL; from g = WS-1 on it precedes.
    // With two areas (XB == 2), X(c+1) goes into the other area at the start
    // of chunk c, before the wait of its first stage: X(c) then precedes
    // DMA(t) at g = 0, and X(c+1) follows DMA(t) for g <= WS-2 (BASE + XL),
    // not after.  (A model of both issue orders on the host shows every wait
    // retires what its stage reads and nothing later, for G = 1..8 and both
    // modes.)
    constexpr int BASE = (WS - 2) * NI;
    static_assert(BASE + XL <= 63, "vmcnt range");

    issue_x(0, 0);
#pragma unroll
    for (int u = 0; u < WS - 1; ++u)
        issue(u);
    for (int64_t c = 0; c < nkc; ++c) {
        if (XB == 2)
            issue_x(c + 1 < nkc ? c + 1 : c, c + 1);
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int64_t t = c * G + g;
            const bool x_pending = XB == 2 ? g <= WS - 2 : (g >= 1 && g <= WS - 2);
            if (x_pending)
                DPS_ROWS_WAIT_VMCNT(BASE + XL);
            else
                DPS_ROWS_WAIT_VMCNT(BASE);
            rows_barrier();
            if (g == 0) {
                read_x(c);
                if (XB == 1) {
                    // the area is refilled only once this wave's reads of it are done
                    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
                    issue_x(c + 1 < nkc ? c + 1 : c, 0);
                }
            }
            issue(t + WS - 1);
            const uint8_t *slot = smem + (int)(t % WS) * SLOT;
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                const u32x4 hv = *reinterpret_cast<const u32x4 *>(slot + foff[s2]);
                u32x4 lv = {0u, 0u, 0u, 0u};
                if (MODE == MODE_FULL)
                    lv = *reinterpret_cast<const u32x4 *>(slot + 16 * kRowsKC + foff[s2]);
                const half8 w0 = weight8<MODE, ENC>(hv.x, hv.y, lv.x, lv.y);
                const half8 w1 = weight8<MODE, ENC>(hv.z, hv.w, lv.z, lv.w);
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    acc[g][nt] = mfma16x16x32(w0, as_half8(xr[s2][0][nt]), acc[g][nt]);
                    acc[g][nt] = mfma16x16x32(w1, as_half8(xr[s2][1][nt]), acc[g][nt]);
                }
            }
        }
    }

    DPS_ROWS_WAIT_VMCNT(0);  // no DMA may still target the ring or the areas
    __syncthreads();         // every wave is done reading the ring

    // ---- slice sums: wave w stores its tiles, then tile (g, nt) is summed
    // over w = 0..7 in order by wave (g NT + nt) % 8.
    f32x4 *red = reinterpret_cast<f32x4 *>(smem);
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
            red[((wave * G + g) * NT + nt) * 64 + lane] = acc[g][nt];
    __syncthreads();
    for (int tile = wave; tile < G * NT; tile += 8) {
        const int g = tile / NT;
        const int nt = tile % NT;
        f32x4 s = red[((0 * G + g) * NT + nt) * 64 + lane];
#pragma unroll
        for (int w = 1; w < 8; ++w)
            s += red[((w * G + g) * NT + nt) * 64 + lane];
        // lane (j, q) holds rows 4q .. 4q+3 of the group for token j
        const int64_t tok = 16 * nt + li;
        const int64_t n0 = r0 + 16 * g + 4 * lg;
        if (tok < a.m && n0 < a.n) {
            uint16_t *yp = a.y + tok * a.n + n0;
            if (n0 + 3 < a.n && (a.n & 3) == 0) {
                typedef _Float16 half4 __attribute__((ext_vector_type(4)));
                const half4 hv = {(_Float16)s.x, (_Float16)s.y, (_Float16)s.z, (_Float16)s.w};
                *reinterpret_cast<half4 *>(yp) = hv;
            } else {
                const float vv[4] = {s.x, s.y, s.z, s.w};
                for (int r = 0; r < 4 && n0 + r < a.n; ++r)
                    yp[r] = __builtin_bit_cast(uint16_t, (_Float16)vv[r]);
            }
        }
    }
}

template <int MODE, int ENC, int NT, int G>
hipError_t launch_g(const RowsArgs &a, bool range, hipStream_t stream)
{
    const dim3 grid((unsigned)((a.n + 16 * G - 1) / (16 * G)));
    if (MODE == MODE_FULL && !range)
        hipLaunchKernelGGL((rows_kernel<MODE, ENC, NT, G, false>), grid, dim3(512), 0, stream, a);
    else
        hipLaunchKernelGGL((rows_kernel<MODE, ENC, NT, G, true>), grid, dim3(512), 0, stream, a);
    return hipGetLastError();
}

template <int MODE, int ENC, int NT>
hipError_t launch_nt(const RowsArgs &a, int groups, bool range, hipStream_t stream)
{
    switch (groups) {
    case 1: return launch_g<MODE, ENC, NT, 1>(a, range, stream);
    case 2: return launch_g<MODE, ENC, NT, 2>(a, range, stream);
    case 3: return launch_g<MODE, ENC, NT, 3>(a, range, stream);
    case 4: return launch_g<MODE, ENC, NT, 4>(a, range, stream);
    case 5: return launch_g<MODE, ENC, NT, 5>(a, range, stream);
    case 6: return launch_g<MODE, ENC, NT, 6>(a, range, stream);
    case 7: return launch_g<MODE, ENC, NT, 7>(a, range, stream);
    case 8: return launch_g<MODE, ENC, NT, 8>(a, range, stream);
    default: return hipErrorInvalidValue;
    }
}

// One 16-token tile: with two (17-32 tokens) every block re-reads twice the
// activations, and on MI355X the hidden-4096 layers ran 5-70% slower than on
// the wide-row GEMM's 32-token tile.
template <int MODE, int ENC>
hipError_t launch_mode(const RowsArgs &a, int groups, bool range, hipStream_t stream)
{
    return launch_nt<MODE, ENC, 1>(a, groups, range, stream);
}

}  // namespace

hipError_t launch_rows(const LinearProblem &p, const LinearPlan &plan, hipStream_t stream)
{
    if (p.rows < 1 || p.rows > 16 || p.experts != 1 || plan.variant < 1 || plan.variant > 8)
        return hipErrorInvalidValue;
    RowsArgs a;
    a.x = p.x;
    a.m = p.rows;
    a.hi = p.hi;
    a.res = p.res;
    a.slots_const = (uint64_t)(uintptr_t)p.res.slots;
    a.n = p.n;
    a.k = p.k;
    a.y = p.y;
    a.rotate = p.k % 4096 == 0;
    const bool range = p.mode == MODE_FULL && p.res.log2c >= 10;
    if (p.enc == ENC_E4M3)
        return p.mode == MODE_FULL
                   ? launch_mode<MODE_FULL, ENC_E4M3>(a, plan.variant, range, stream)
                   : launch_mode<MODE_FAST, ENC_E4M3>(a, plan.variant, range, stream);
    return p.mode == MODE_FULL ? launch_mode<MODE_FULL, ENC_E5M2>(a, plan.variant, range, stream)
                               : launch_mode<MODE_FAST, ENC_E5M2>(a, plan.variant, range, stream);
}

}  // namespace dps
