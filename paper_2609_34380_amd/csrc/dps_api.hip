// dps_api.hip -- the C ABI of libdps: argument validation, kernel planning and
// launches.  Nothing here allocates device memory or synchronizes.
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "dps.h"
#include "dps_internal.h"

#define DPS_EXPORT extern "C" __attribute__((visibility("default")))

namespace dps {
int skinny_rows_per_block(int variant);
int skinny_k_per_batch(int variant);
int skinny_pass_rows(int64_t rows, bool grouped);
int64_t skinny_max_ksplit(int variant, int mode, int64_t pass_rows);
int gemm_rows_per_block(int variant);
int gemm_tokens_per_block(int variant);
}  // namespace dps

namespace {

thread_local char g_err[256] = "";

dps_status fail(dps_status s, const char *fmt, const char *what)
{
    snprintf(g_err, sizeof(g_err), fmt, what);
    return s;
}

#define REQUIRE(cond, status, what)                        \
    do {                                                   \
        if (!(cond))                                       \
            return fail(status, "%s", what);               \
    } while (0)

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t round_up(int64_t a, int64_t b) { return cdiv(a, b) * b; }
size_t align256(int64_t bytes) { return (size_t)round_up(bytes, 256); }

int current_cu_count()
{
    static int cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return 256;
    if (dev < 64 && cache[dev] > 0)
        return cache[dev];
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        cus = 256;
    if (dev < 64)
        cache[dev] = cus;
    return cus;
}

// Pool geometry checks shared by every call that touches a residual.
dps_status check_pool(const dps_residual *r, int64_t numel)
{
    REQUIRE(r != nullptr, DPS_ERR_INVALID_ARG, "residual descriptor is NULL");
    REQUIRE(r->pool != nullptr, DPS_ERR_INVALID_ARG, "residual pool is NULL");
    REQUIRE(aligned(r->pool, 16), DPS_ERR_ALIGNMENT, "residual pool is not 16-byte aligned");
    REQUIRE(r->log2_chunk >= 4 && r->log2_chunk <= 30, DPS_ERR_INVALID_ARG,
            "log2_chunk must be in 4..30");
    const int64_t c = int64_t(1) << r->log2_chunk;
    REQUIRE(r->pool_bytes >= c, DPS_ERR_INVALID_ARG, "pool_bytes is smaller than one chunk");
    REQUIRE(r->n_chunks >= 0, DPS_ERR_INVALID_ARG, "n_chunks is negative");
    REQUIRE(r->n_chunks >= cdiv(numel, c), DPS_ERR_INVALID_ARG,
            "n_chunks does not cover the tensor");
    return DPS_OK;
}

// Residual descriptor checks shared by split, merge and full-mode linears.
dps_status check_residual(const dps_residual *r, int64_t numel)
{
    const dps_status s = check_pool(r, numel);
    if (s != DPS_OK)
        return s;
    REQUIRE(r->slots != nullptr, DPS_ERR_INVALID_ARG, "residual slot table is NULL");
    REQUIRE(aligned(r->slots, 4), DPS_ERR_ALIGNMENT, "residual slot table is not 4-byte aligned");
    return DPS_OK;
}

// Host slot-table entries of chunks [c0, c1) must address whole pool slots.
dps_status check_host_slots(const dps_residual *r, const int32_t *slots_host, int64_t c0,
                            int64_t c1)
{
    REQUIRE(slots_host != nullptr, DPS_ERR_INVALID_ARG, "host slot table is NULL");
    const int64_t n_slots = r->pool_bytes >> r->log2_chunk;
    for (int64_t c = c0; c < c1; ++c)
        REQUIRE(slots_host[c] >= 0 && slots_host[c] < n_slots, DPS_ERR_INVALID_ARG,
                "host slot table entry outside the pool");
    return DPS_OK;
}

dps::ResidualView view_of(const dps_residual *r)
{
    dps::ResidualView v;
    v.pool = r->pool;
    v.slots = r->slots;
    v.log2c = r->log2_chunk;
    v.n_pool_slots = r->pool_bytes >> r->log2_chunk;
    v.n_chunks = r->n_chunks;
    return v;
}

dps_status launched(hipError_t e)
{
    if (e != hipSuccess) {
        snprintf(g_err, sizeof(g_err), "HIP launch failed: %s", hipGetErrorString(e));
        return DPS_ERR_HIP;
    }
    return DPS_OK;
}

dps_status check_weight(const dps_weight *w, int mode)
{
    REQUIRE(w != nullptr, DPS_ERR_INVALID_ARG, "weight descriptor is NULL");
    REQUIRE(w->enc == DPS_ENC_E5M2 || w->enc == DPS_ENC_E4M3, DPS_ERR_INVALID_ARG,
            "unknown nested encoding");
    REQUIRE(w->experts >= 1 && w->experts <= 65535, DPS_ERR_INVALID_ARG,
            "experts must be in 1..65535");
    REQUIRE(w->n > 0 && w->n <= 0x7fffffff, DPS_ERR_INVALID_ARG, "n must be in 1..2^31-1");
    REQUIRE(w->k > 0 && w->k % 16 == 0, DPS_ERR_INVALID_ARG, "k must be a positive multiple of 16");
    // the kernels keep a block's K range in 32-bit lane registers
    REQUIRE(w->k <= (int64_t(1) << 30), DPS_ERR_INVALID_ARG, "k must be at most 2^30");
    REQUIRE(w->hi != nullptr, DPS_ERR_INVALID_ARG, "upper-byte plane is NULL");
    REQUIRE(aligned(w->hi, 16), DPS_ERR_ALIGNMENT, "upper-byte plane is not 16-byte aligned");
    if (mode == DPS_MODE_FULL) {
        dps_status s = check_residual(&w->res, w->experts * w->n * w->k);
        if (s != DPS_OK)
            return s;
    }
    return DPS_OK;
}

}  // namespace

namespace dps {

LinearPlan plan_linear(int mode, uint32_t flags, int64_t rows, int64_t n, int64_t k,
                       int64_t experts, int log2c, int cu_count, bool grouped)
{
    LinearPlan p;
    memset(&p, 0, sizeof(p));
    const int64_t rows_per_expert = grouped ? cdiv(rows, experts) : rows;
    if (flags & DPS_ACT_FP8_ROWSCALE) {
        p.kind = KIND_GEMM_FP8;
        // 256 x 256 tiles once their grid gives every CU a block and its last
        // round of blocks is at least half full, else 256 x 128.  MI355X,
        // hidden-4096 layers: gate+up at 1024 tokens (448 big tiles) 136
        // against 165 us, down and O at 4096 tokens (256) 245 / 78 against
        // 297 / 95; QKV at 2048 tokens (192) 94 against 110 and at 3072
        // (288, a last round of 32) 129 against 139 on the smaller tile.
        // Grouped calls take the 128-token tile: an expert's rows rarely
        // fill 256.
        {
            const int64_t cus = cu_count;
            const int64_t big = cdiv(n, 256) * cdiv(rows, 256);
            const bool fills = big >= cus && (big % cus == 0 || 2 * (big % cus) >= cus);
            p.variant = fills && !grouped ? GEMM_G3_256x256 : GEMM_G3_256x128;
        }
        // K is split only while the tiles alone leave CUs idle: the fp32
        // partials cost more than a half-filled last wave of blocks (MI355X,
        // split to two blocks per CU against one: gate+up at 512 tokens 129
        // against 95 us, O at 2048 tokens 71 against 51, down 167 against
        // 148; QKV at 512 tokens 48 against 50)
        const int64_t tiles =
            cdiv(n, gemm_rows_per_block(p.variant)) * cdiv(rows, gemm_tokens_per_block(p.variant));
        int64_t s = cdiv((int64_t)cu_count, tiles);
        const int64_t smax = k / 1024 > 1 ? k / 1024 : 1;
        s = s < 1 ? 1 : (s > smax ? smax : s);
        p.ksplit = round_up(cdiv(k, s), 128);
        p.splits = (int)cdiv(k, p.ksplit);
        p.ws_quant = align256(rows * k) + align256(rows * 4);
    } else if (!grouped && (rows <= 2 || (rows <= 4 && n * k <= (int64_t(1) << 25))) &&
               rows * k * 2 <= 65536) {
        // Dense calls of 1-2 tokens, and up to 4 on layers of at most 2^25
        // weights, whose activations fit 64 KiB of LDS: whole weight rows per
        // wave in 1 KiB loads on the vector ALUs, no K split.  Measured on
        // MI355X against the decode and wide-row kernels (hidden-4096 set):
        // 0.62-0.76x the time at 1 token, 0.69-0.86x at 2 tokens (down: even
        // over both modes); at 4 tokens on the large layers and at 8 tokens
        // the vector ALUs and activation reads make it slower.
        p.kind = KIND_GEMV;
        p.variant = 0;
        p.ksplit = k;
        p.splits = 1;
    } else if (!grouped && rows <= 16) {
        // Dense calls of 3-16 tokens (and 1-2 whose activations exceed the row
        // GEMV's LDS): 16-row groups over the whole K range per block,
        // streamed in 1 KiB row pieces, no K split, one launch; G groups per
        // block so that the grid about fills the chip once.  Measured on
        // MI355X at 8 tokens (hidden-4096 set) against the wide-row GEMM with
        // its split-K reduction: 0.68-0.83x the time in fast mode and
        // 0.86-0.95x in full mode.
        p.kind = KIND_ROWS;
        const int64_t groups = cdiv(n, 16);
        int64_t g = cdiv(groups, (int64_t)cu_count);
        p.variant = (int)(g < 1 ? 1 : (g > 8 ? 8 : g));
        p.ksplit = k;
        p.splits = 1;
    } else if (rows_per_expert <= 1 || (rows_per_expert <= 4 && n * k <= (int64_t(1) << 25))) {
        // The decode kernel serves one token per expert, and up to four on
        // layers of at most 2^25 weights.  Everywhere else the wide-row GEMM
        // with 32-token tiles is as fast or faster on MI355X (8 tokens,
        // hidden-4096 set, both modes: 182 us against 224 us; the full-mode
        // 28672 x 4096 layer 50 us against 68).
        p.kind = KIND_SKINNY;
        // measured on MI355X: up to 8 tokens, the weight stream through
        // per-wave LDS rings (two blocks per CU); above that (grouped passes
        // of 64 rows), registers with 16 rows per wave up to 16 tokens and 32
        // rows (half batches) beyond
        const int64_t xr = skinny_pass_rows(rows, grouped);
        p.variant = xr <= 16 ? 0 : 1;
        if (xr <= 8 && skinny_max_ksplit(SKINNY_RING, mode, xr) > 0)
            p.variant = SKINNY_RING;
        const int64_t kpb = skinny_k_per_batch(p.variant);
        // the block's X slice [pass rows][ksplit + 8] FP16 must fit its LDS share
        const int64_t kmax = skinny_max_ksplit(p.variant, mode, xr);
        const int64_t blocks = cdiv(n, skinny_rows_per_block(p.variant)) * experts;
        int64_t s = cdiv((int64_t)cu_count, blocks);
        const int64_t smax = k / kpb > 1 ? k / kpb : 1;
        s = s < 1 ? 1 : (s > smax ? smax : s);
        p.ksplit = round_up(cdiv(k, s), kpb);
        if (p.ksplit > kmax)
            p.ksplit = kmax;
        p.splits = (int)cdiv(k, p.ksplit);
    } else {
        p.kind = KIND_GEMM_F16;
        // One plan for both modes, so that fast mode equals full mode over a
        // zero residual bit for bit (same tiles, same K ranges, same order).
        // Every other FP16 shape takes the wide-row GEMM (on MI355X it beat
        // register-staged and eight-wave FP16 kernels at 128 and 256 tokens
        // and matched them at 2048), with a 32-, 64- or 128-token tile so
        // that short calls stage no padding rows.  K is split
        // so that about one block of eight waves per CU is resident (the split
        // count rounds down); each range keeps >= 1024 elements.
        // four dedicated DMA waves pay off from 64-token tiles on (MI355X:
        // 3-10% at 128-2048 tokens; at 32 tokens the plain kernel is 2% ahead)
        // Layers of at most 2^24 weights keep the 32-token tile up to 256
        // tokens: more tiles and shorter split-K chains win there (MI355X,
        // hidden-4096 O layer, both modes: 34.5 against 40.3 us at 128
        // tokens, even at 256; the QKV, gate+up and down layers lose 1-30%
        // with it).  From 512 tokens on the wider tiles read each weight
        // tile for 4x as many tokens and win (O layer, full / fast mode:
        // 33 / 28 against 51 / 39 us at 512 tokens, 94 / 77 against 185 /
        // 150 us at 2048).
        p.variant = (rows_per_expert <= 32 ||
                     (n * k <= (int64_t(1) << 24) && rows_per_expert <= 256))
                        ? GEMM_G4_128x32
                        : (rows_per_expert <= 64 ? GEMM_G4S_128x64 : GEMM_G4S_128x128);
        // Dense prefill-sized calls take the 256 x 256 tile when it fills the
        // chip (at least one block per CU), or fills it with two K ranges and
        // K is long enough (>= 8192) for them to pay for their fp32 partials.
        // MI355X, hidden-4096 set, full mode: gate+up at 1024 / 2048 tokens
        // 318 / 619 against 345 / 669 us, down at 2048 tokens (two ranges)
        // 284 against 302, every layer at 8192 tokens 0.82-0.92x the time
        // (gate+up 1962 against 2340 us).  Slower on it: QKV and O at 2048
        // tokens (192 and 128 tiles, 4-5%), down at 512 / 1024 tokens (8 / 4
        // ranges: 89 / 161 against 80 / 154 us) and every decode call up to
        // 256 tokens (gate+up at 256 tokens 93 against 88 us).
        if (!grouped && rows >= 512) {
            const int64_t t5 = cdiv(n, 256) * cdiv(rows, 256);
            if (t5 >= cu_count || (k >= 8192 && 2 * t5 >= cu_count))
                p.variant = GEMM_G5_256x256;
        }
        const bool g5 = p.variant == GEMM_G5_256x256;
        const int64_t tiles =
            cdiv(n, gemm_rows_per_block(p.variant)) * cdiv(rows, gemm_tokens_per_block(p.variant));
        // the 256-row tiles hold one block per CU (160 KiB of LDS); the
        // wide-row GEMM's eight waves share a CU with others
        int64_t s = (int64_t)cu_count / tiles;
        const int64_t smax = k / 1024 > 1 ? k / 1024 : 1;
        s = s < 1 ? 1 : (s > smax ? smax : s);
        p.ksplit = round_up(cdiv(k, s), g5 ? 64 : 128);
        p.splits = (int)cdiv(k, p.ksplit);
    }
    p.range_addr = mode == MODE_FULL && p.ksplit <= (int64_t(1) << log2c);
    p.ws_partial = p.splits > 1 ? align256((int64_t)p.splits * rows * n * 4) : 0;
    return p;
}

}  // namespace dps

DPS_EXPORT const char *dps_status_str(dps_status s)
{
    switch (s) {
    case DPS_OK: return "ok";
    case DPS_ERR_INVALID_ARG: return "invalid argument";
    case DPS_ERR_ALIGNMENT: return "misaligned pointer";
    case DPS_ERR_UNSUPPORTED: return "unsupported";
    case DPS_ERR_WORKSPACE: return "workspace too small";
    case DPS_ERR_HIP: return "HIP error";
    case DPS_ERR_NO_SPACE: return "no space";
    case DPS_ERR_TIMEOUT: return "timed out";
    }
    return "unknown status";
}

DPS_EXPORT const char *dps_last_error(void) { return g_err; }

DPS_EXPORT dps_status dps_select_enc(const uint16_t *w, int64_t numel, int32_t *enc_out,
                                     void *stream)
{
    g_err[0] = 0;
    REQUIRE(numel >= 0, DPS_ERR_INVALID_ARG, "numel is negative");
    REQUIRE(enc_out != nullptr, DPS_ERR_INVALID_ARG, "enc_out is NULL");
    REQUIRE(aligned(enc_out, 4), DPS_ERR_ALIGNMENT, "enc_out is not 4-byte aligned");
    REQUIRE(numel == 0 || w != nullptr, DPS_ERR_INVALID_ARG, "w is NULL");
    REQUIRE(aligned(w, 16), DPS_ERR_ALIGNMENT, "w is not 16-byte aligned");
    return launched(dps::launch_select_enc(w, numel, enc_out, (hipStream_t)stream));
}

DPS_EXPORT dps_status dps_split(int enc, const uint16_t *w, int64_t numel, uint8_t *hi,
                                const dps_residual *res, void *stream)
{
    g_err[0] = 0;
    REQUIRE(enc == DPS_ENC_E5M2 || enc == DPS_ENC_E4M3, DPS_ERR_INVALID_ARG,
            "unknown nested encoding");
    REQUIRE(numel >= 0, DPS_ERR_INVALID_ARG, "numel is negative");
    if (numel == 0)
        return DPS_OK;
    REQUIRE(w != nullptr && hi != nullptr, DPS_ERR_INVALID_ARG, "w or hi is NULL");
    REQUIRE(aligned(w, 16) && aligned(hi, 16), DPS_ERR_ALIGNMENT, "w or hi is not 16-byte aligned");
    dps_status s = check_residual(res, numel);
    if (s != DPS_OK)
        return s;
    return launched(dps::launch_split(enc, w, numel, hi, view_of(res), (hipStream_t)stream));
}

DPS_EXPORT dps_status dps_merge(int enc, const uint8_t *hi, const dps_residual *res,
                                int64_t numel, uint16_t *w_out, void *stream)
{
    g_err[0] = 0;
    REQUIRE(enc == DPS_ENC_E5M2 || enc == DPS_ENC_E4M3, DPS_ERR_INVALID_ARG,
            "unknown nested encoding");
    REQUIRE(numel >= 0, DPS_ERR_INVALID_ARG, "numel is negative");
    if (numel == 0)
        return DPS_OK;
    REQUIRE(w_out != nullptr && hi != nullptr, DPS_ERR_INVALID_ARG, "hi or w_out is NULL");
    REQUIRE(aligned(w_out, 16) && aligned(hi, 16), DPS_ERR_ALIGNMENT,
            "hi or w_out is not 16-byte aligned");
    dps_status s = check_residual(res, numel);
    if (s != DPS_OK)
        return s;
    return launched(dps::launch_merge(enc, hi, view_of(res), numel, w_out, (hipStream_t)stream));
}

DPS_EXPORT dps_status dps_restore(const uint8_t *backup, int64_t numel, const dps_residual *res,
                                  const int32_t *slots_host, int64_t chunk_begin,
                                  int64_t chunk_end, int64_t copy_bytes, void *stream)
{
    g_err[0] = 0;
    REQUIRE(numel >= 0, DPS_ERR_INVALID_ARG, "numel is negative");
    REQUIRE(copy_bytes > 0, DPS_ERR_INVALID_ARG, "copy_bytes must be positive");
    dps_status s = check_pool(res, numel);
    if (s != DPS_OK)
        return s;
    const int64_t used = cdiv(numel, int64_t(1) << res->log2_chunk);
    REQUIRE(chunk_begin >= 0 && chunk_begin <= chunk_end && chunk_end <= used,
            DPS_ERR_INVALID_ARG, "chunk range outside the tensor");
    if (chunk_begin == chunk_end)
        return DPS_OK;
    REQUIRE(backup != nullptr, DPS_ERR_INVALID_ARG, "backup is NULL");
    s = check_host_slots(res, slots_host, chunk_begin, chunk_end);
    if (s != DPS_OK)
        return s;
    return launched(dps::launch_restore(backup, numel, view_of(res), slots_host, chunk_begin,
                                        chunk_end, copy_bytes, (hipStream_t)stream));
}

DPS_EXPORT dps_status dps_backup(const dps_residual *res, const int32_t *slots_host,
                                 int64_t numel, uint8_t *backup, int64_t copy_bytes,
                                 void *stream)
{
    g_err[0] = 0;
    REQUIRE(numel >= 0, DPS_ERR_INVALID_ARG, "numel is negative");
    REQUIRE(copy_bytes > 0, DPS_ERR_INVALID_ARG, "copy_bytes must be positive");
    dps_status s = check_pool(res, numel);
    if (s != DPS_OK)
        return s;
    if (numel == 0)
        return DPS_OK;
    REQUIRE(backup != nullptr, DPS_ERR_INVALID_ARG, "backup is NULL");
    s = check_host_slots(res, slots_host, 0, cdiv(numel, int64_t(1) << res->log2_chunk));
    if (s != DPS_OK)
        return s;
    return launched(dps::launch_backup(view_of(res), slots_host, numel, backup, copy_bytes,
                                       (hipStream_t)stream));
}

DPS_EXPORT dps_status dps_quant_rows_e4m3(const uint16_t *x, int64_t m, int64_t k, uint8_t *xq,
                                          float *scale, void *stream)
{
    g_err[0] = 0;
    REQUIRE(m >= 0 && m <= 0x7fffffff, DPS_ERR_INVALID_ARG, "m must be in 0..2^31-1");
    REQUIRE(k > 0 && k % 16 == 0 && k <= (int64_t(1) << 30), DPS_ERR_INVALID_ARG,
            "k must be a positive multiple of 16, at most 2^30");
    if (m == 0)
        return DPS_OK;
    REQUIRE(x != nullptr && xq != nullptr && scale != nullptr, DPS_ERR_INVALID_ARG,
            "x, xq or scale is NULL");
    REQUIRE(aligned(x, 16) && aligned(xq, 16) && aligned(scale, 4), DPS_ERR_ALIGNMENT,
            "x/xq not 16-byte aligned or scale not 4-byte aligned");
    return launched(dps::launch_quant_rows(x, m, k, xq, scale, (hipStream_t)stream));
}

DPS_EXPORT size_t dps_workspace_bytes(int mode, uint32_t flags, int64_t rows, int64_t n,
                                      int64_t k, int64_t experts)
{
    if (rows <= 0 || n <= 0 || k <= 0 || experts < 1)
        return 0;
    const dps::LinearPlan p =
        dps::plan_linear(mode, flags, rows, n, k, experts, 30, current_cu_count(), experts > 1);
    return p.ws_partial + p.ws_quant;
}

DPS_EXPORT dps_status dps_plan_info(int mode, uint32_t flags, int64_t rows, int64_t n, int64_t k,
                                    int64_t experts, int32_t log2_chunk, int64_t *info)
{
    g_err[0] = 0;
    REQUIRE(mode == DPS_MODE_FULL || mode == DPS_MODE_FAST, DPS_ERR_INVALID_ARG, "unknown mode");
    REQUIRE(flags == DPS_ACT_FP16 || flags == DPS_ACT_FP8_ROWSCALE, DPS_ERR_INVALID_ARG,
            "unknown flags");
    REQUIRE(rows > 0 && n > 0 && k > 0 && experts >= 1, DPS_ERR_INVALID_ARG,
            "rows, n, k and experts must be positive");
    REQUIRE(log2_chunk >= 4 && log2_chunk <= 30, DPS_ERR_INVALID_ARG,
            "log2_chunk must be in 4..30");
    REQUIRE(info != nullptr, DPS_ERR_INVALID_ARG, "info is NULL");
    const bool grouped = experts > 1;
    const dps::LinearPlan p =
        dps::plan_linear(mode, flags, rows, n, k, experts,
                         mode == DPS_MODE_FULL ? log2_chunk : 30, current_cu_count(), grouped);
    switch (p.kind) {
    case dps::KIND_GEMV:
        info[0] = DPS_KERNEL_GEMV;
        info[1] = 0;
        info[2] = rows;
        break;
    case dps::KIND_ROWS:
        info[0] = DPS_KERNEL_ROWS;
        info[1] = 16 * p.variant;
        info[2] = 16;
        break;
    case dps::KIND_SKINNY:
        info[0] = DPS_KERNEL_DECODE;
        info[1] = dps::skinny_rows_per_block(p.variant);
        info[2] = dps::skinny_pass_rows(rows, grouped);
        break;
    default:
        info[0] = p.kind == dps::KIND_GEMM_FP8 ? DPS_KERNEL_GEMM_FP8 : DPS_KERNEL_GEMM_F16;
        info[1] = dps::gemm_rows_per_block(p.variant);
        info[2] = dps::gemm_tokens_per_block(p.variant);
        break;
    }
    info[3] = p.splits;
    info[4] = p.ksplit;
    return DPS_OK;
}

namespace {

dps_status run_linear(int mode, uint32_t flags, const uint16_t *x, const int32_t *offsets,
                      int64_t rows, const dps_weight *w, uint16_t *y, void *ws, size_t ws_bytes,
                      hipStream_t stream, bool grouped)
{
    const dps::LinearPlan plan =
        dps::plan_linear(mode, flags, rows, w->n, w->k, w->experts,
                         mode == DPS_MODE_FULL ? w->res.log2_chunk : 30, current_cu_count(),
                         grouped);
    const size_t need = plan.ws_partial + plan.ws_quant;
    if (need > 0) {
        REQUIRE(ws != nullptr && ws_bytes >= need, DPS_ERR_WORKSPACE,
                "workspace is smaller than dps_workspace_bytes()");
        REQUIRE(aligned(ws, 256), DPS_ERR_ALIGNMENT, "workspace is not 256-byte aligned");
    }
    // grouped GEMM grids run one row of blocks per token tile plus one per
    // expert (grid.y); keep every call within that limit
    const bool gemm = plan.kind == dps::KIND_GEMM_F16 || plan.kind == dps::KIND_GEMM_FP8;
    const int64_t token_tiles =
        cdiv(rows, gemm ? dps::gemm_tokens_per_block(plan.variant) : 128) +
        (grouped ? w->experts : 0);
    REQUIRE(token_tiles <= 65535, DPS_ERR_UNSUPPORTED, "too many rows for one call");
    REQUIRE(plan.splits <= 65535, DPS_ERR_UNSUPPORTED, "k too large for one call");
    // dense GEMMs run a 1-D grid of up to 768 threads per block, whose size
    // in threads must fit 32 bits
    if (gemm && !grouped)
        REQUIRE(cdiv(w->n, dps::gemm_rows_per_block(plan.variant)) * plan.splits * token_tiles <=
                    (int64_t)(0xFFFFFFFFu / 768),
                DPS_ERR_UNSUPPORTED, "call too large for one grid");

    float *partial = plan.splits > 1 ? static_cast<float *>(ws) : nullptr;
    dps::LinearProblem p;
    p.mode = mode;
    p.enc = w->enc;
    p.x = x;
    p.offsets = offsets;
    p.rows = rows;
    p.experts = w->experts;
    p.n = w->n;
    p.k = w->k;
    p.hi = w->hi;
    p.res = mode == DPS_MODE_FULL ? view_of(&w->res) : dps::ResidualView{nullptr, nullptr, 0, 0, 0};
    p.y = y;

    dps_status st;
    if (plan.kind == dps::KIND_GEMM_FP8) {
        uint8_t *xq = static_cast<uint8_t *>(ws) + plan.ws_partial;
        float *scale = reinterpret_cast<float *>(xq + align256(rows * w->k));
        st = launched(dps::launch_quant_rows(x, rows, w->k, xq, scale, stream));
        if (st != DPS_OK)
            return st;
        st = launched(dps::launch_gemm_fp8(w->enc, xq, scale, offsets, rows, w->experts, w->n,
                                           w->k, w->hi, y, plan, partial, stream));
    } else if (plan.kind == dps::KIND_GEMV) {
        st = launched(dps::launch_gemv(p, plan, stream));
    } else if (plan.kind == dps::KIND_ROWS) {
        st = launched(dps::launch_rows(p, plan, stream));
    } else if (plan.kind == dps::KIND_SKINNY) {
        st = launched(dps::launch_skinny(p, plan, partial, stream));
    } else {
        st = launched(dps::launch_gemm_f16(p, plan, partial, stream));
    }
    if (st != DPS_OK || plan.splits == 1)
        return st;
    return launched(dps::launch_splitk_reduce(partial, plan.splits, rows, w->n, y, stream));
}

}  // namespace

DPS_EXPORT dps_status dps_linear(int mode, uint32_t flags, const uint16_t *x, int64_t m,
                                 const dps_weight *w, uint16_t *y, void *ws, size_t ws_bytes,
                                 void *stream)
{
    g_err[0] = 0;
    REQUIRE(mode == DPS_MODE_FULL || mode == DPS_MODE_FAST, DPS_ERR_INVALID_ARG, "unknown mode");
    REQUIRE(flags == DPS_ACT_FP16 || flags == DPS_ACT_FP8_ROWSCALE, DPS_ERR_INVALID_ARG,
            "unknown flags");
    REQUIRE(!(flags == DPS_ACT_FP8_ROWSCALE && mode != DPS_MODE_FAST), DPS_ERR_INVALID_ARG,
            "FP8 activations need fast mode");
    dps_status s = check_weight(w, mode);
    if (s != DPS_OK)
        return s;
    REQUIRE(w->experts == 1, DPS_ERR_INVALID_ARG, "dps_linear takes a dense weight (experts == 1)");
    REQUIRE(m >= 0, DPS_ERR_INVALID_ARG, "m is negative");
    if (m == 0)
        return DPS_OK;
    REQUIRE(x != nullptr && y != nullptr, DPS_ERR_INVALID_ARG, "x or y is NULL");
    REQUIRE(aligned(x, 16) && aligned(y, 16), DPS_ERR_ALIGNMENT, "x or y is not 16-byte aligned");
    return run_linear(mode, flags, x, nullptr, m, w, y, ws, ws_bytes, (hipStream_t)stream, false);
}

DPS_EXPORT dps_status dps_linear_grouped(int mode, uint32_t flags, const uint16_t *x_sorted,
                                         const int32_t *offsets, int64_t rows,
                                         const dps_weight *w, uint16_t *y, void *ws,
                                         size_t ws_bytes, void *stream)
{
    g_err[0] = 0;
    REQUIRE(mode == DPS_MODE_FULL || mode == DPS_MODE_FAST, DPS_ERR_INVALID_ARG, "unknown mode");
    REQUIRE(flags == DPS_ACT_FP16 || flags == DPS_ACT_FP8_ROWSCALE, DPS_ERR_INVALID_ARG,
            "unknown flags");
    REQUIRE(!(flags == DPS_ACT_FP8_ROWSCALE && mode != DPS_MODE_FAST), DPS_ERR_INVALID_ARG,
            "FP8 activations need fast mode");
    dps_status s = check_weight(w, mode);
    if (s != DPS_OK)
        return s;
    REQUIRE(rows >= 0, DPS_ERR_INVALID_ARG, "rows is negative");
    if (rows == 0)
        return DPS_OK;
    REQUIRE(offsets != nullptr, DPS_ERR_INVALID_ARG, "offsets is NULL");
    REQUIRE(aligned(offsets, 4), DPS_ERR_ALIGNMENT, "offsets is not 4-byte aligned");
    REQUIRE(x_sorted != nullptr && y != nullptr, DPS_ERR_INVALID_ARG, "x_sorted or y is NULL");
    REQUIRE(aligned(x_sorted, 16) && aligned(y, 16), DPS_ERR_ALIGNMENT,
            "x_sorted or y is not 16-byte aligned");
    // One expert owns every row (offsets = {0, rows}): the dense call, with
    // the dense plan that dps_workspace_bytes reports for experts == 1
    if (w->experts == 1)
        return run_linear(mode, flags, x_sorted, nullptr, rows, w, y, ws, ws_bytes,
                          (hipStream_t)stream, false);
    return run_linear(mode, flags, x_sorted, offsets, rows, w, y, ws, ws_bytes,
                      (hipStream_t)stream, true);
}

// ---- dps_linear_static: dps_linear with library-owned scratch ----------------
// The split-K partials and the FP8 activation staging of a call live in one
// file-scope device array instead of a caller workspace.  Each device that
// loads the library holds its own copy until the process ends; host code
// reaches it only through the address hipGetSymbolAddress returns for the
// current device (the array's name is a host-side stand-in, not a device
// address).  Nothing in it has to start at zero: every byte a kernel reads
// there was written earlier in the same call.
static __device__ __align__(256) uint8_t scratch[DPS_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {nullptr};

// Device address of the current device's scratch array, looked up once per
// device (with that device current) and kept.
dps_status static_scratch(void **out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return launched(e);
    REQUIRE(dev >= 0 && dev < kMaxDevices, DPS_ERR_UNSUPPORTED,
            "device index beyond the static scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr) {
            snprintf(g_err, sizeof(g_err), "hipGetSymbolAddress(scratch) failed: %s",
                     hipGetErrorString(e));
            return DPS_ERR_HIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return DPS_OK;
}

}  // namespace

DPS_EXPORT dps_status dps_linear_static(int mode, uint32_t flags, const uint16_t *x, int64_t m,
                                        const dps_weight *w, uint16_t *y, void *stream)
{
    g_err[0] = 0;
    void *ws = nullptr;
    dps_status s = static_scratch(&ws);
    if (s != DPS_OK)
        return s;
    REQUIRE(mode == DPS_MODE_FULL || mode == DPS_MODE_FAST, DPS_ERR_INVALID_ARG, "unknown mode");
    REQUIRE(flags == DPS_ACT_FP16 || flags == DPS_ACT_FP8_ROWSCALE, DPS_ERR_INVALID_ARG,
            "unknown flags");
    REQUIRE(!(flags == DPS_ACT_FP8_ROWSCALE && mode != DPS_MODE_FAST), DPS_ERR_INVALID_ARG,
            "FP8 activations need fast mode");
    s = check_weight(w, mode);
    if (s != DPS_OK)
        return s;
    REQUIRE(w->experts == 1, DPS_ERR_INVALID_ARG,
            "dps_linear_static takes a dense weight (experts == 1)");
    REQUIRE(m >= 0, DPS_ERR_INVALID_ARG, "m is negative");
    if (m == 0)
        return DPS_OK;
    REQUIRE(x != nullptr && y != nullptr, DPS_ERR_INVALID_ARG, "x or y is NULL");
    REQUIRE(aligned(x, 16) && aligned(y, 16), DPS_ERR_ALIGNMENT, "x or y is not 16-byte aligned");
    const dps::LinearPlan plan =
        dps::plan_linear(mode, flags, m, w->n, w->k, 1,
                         mode == DPS_MODE_FULL ? w->res.log2_chunk : 30, current_cu_count(),
                         false);
    const size_t need = plan.ws_partial + plan.ws_quant;
    if (need > (size_t)DPS_STATIC_SCRATCH_BYTES) {
        snprintf(g_err, sizeof(g_err),
                 "call needs %zu bytes of scratch, above the static scratch of %zu bytes; "
                 "use dps_linear with a workspace",
                 need, (size_t)DPS_STATIC_SCRATCH_BYTES);
        return DPS_ERR_WORKSPACE;
    }
    return run_linear(mode, flags, x, nullptr, m, w, y, ws, DPS_STATIC_SCRATCH_BYTES,
                      (hipStream_t)stream, false);
}
