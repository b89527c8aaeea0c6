/*
 * dps.h -- C ABI of libdps, the MI355X (gfx950) nested-precision linear layer
 * of Dual-Mode Precision Serving (DPS).
 *
 * The method (Sec. IV of the paper) keeps every FP16 weight as two bytes held
 * in two places:
 *   - the upper byte -- an FP8 number, the FP16 value truncated to E5M2 or,
 *     for layers of small range, to E4M3 scaled by 2^8 -- in a persistent
 *     region (Sec. IV-B "Persistent Region");
 *   - the lower byte, the residual, in a shared region whose physical memory
 *     is made of relocatable units that may instead hold paged KV-cache
 *     blocks (Sec. IV-B "Shared Region"; Sec. IV-C, restoration paragraph).
 * Full mode rebuilds the original FP16 weights from both bytes during the
 * product; fast mode reads the upper byte only and never touches the
 * residual, whose memory may hold KV data at that time (Sec. IV-C "Overall
 * concept").  One kernel family serves dense layers and MoE expert groups
 * (Sec. IV-C, GroupedGEMM paragraph).
 *
 * Conventions for every entry point:
 *   - Tensor pointers are HIP device memory owned by the caller; the library
 *     never allocates, frees, synchronizes or keeps a pointer after return.
 *     Buffers must stay alive until the enqueued work completes.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  All work
 *     is enqueued on it, asynchronously.
 *   - Arguments are validated on the host before anything is enqueued; on
 *     any error nothing is launched and a status other than DPS_OK is
 *     returned (dps_last_error() then names the offending argument).
 *   - Faults inside kernels surface at the caller's next synchronization.
 *   - Calls are reentrant.  Two calls that share a workspace must be
 *     ordered (same stream, or synchronized).
 *   - Matrices are row-major.  Y = X . W^T: X is [m][k], W is [n][k],
 *     Y is [m][n].
 */
#ifndef DPS_H
#define DPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DPS_OK = 0,
    DPS_ERR_INVALID_ARG = 1, /* null/negative/inconsistent argument         */
    DPS_ERR_ALIGNMENT = 2,   /* a tensor pointer is not 16-byte aligned      */
    DPS_ERR_UNSUPPORTED = 3, /* valid request the library does not implement */
    DPS_ERR_WORKSPACE = 4,   /* workspace missing or smaller than required   */
    DPS_ERR_HIP = 5,         /* the HIP runtime reported an error on launch  */
    DPS_ERR_NO_SPACE = 6,    /* SUM manager: not enough room for the request */
    DPS_ERR_TIMEOUT = 7      /* restore worker: still busy when the wait ended */
} dps_status;

/* Precision mode of one call; a whole forward pass runs in one mode
 * (batch-aligned switching, Sec. IV-C "Overall concept" and "Granularity of
 * the precision switch"). */
typedef enum {
    DPS_MODE_FULL = 0, /* FP16 rebuilt from upper byte + residual byte       */
    DPS_MODE_FAST = 1  /* FP8 upper byte only; residual never read           */
} dps_mode;

/* Nested encodings (Sec. IV-B "Persistent Region"), chosen per layer
 * (Sec. IV-C, "Dual-mode serving" paragraph).  FP16 word w = sign s,
 * exponent e (5 bits), mantissa m (10 bits):
 *   DPS_ENC_E5M2: upper byte = s | e | m[9:8]   (w >> 8, E5M2 by truncation),
 *                 residual byte = m[7:0];  fast-mode weight = E5M2(upper).
 *   DPS_ENC_E4M3: upper byte = s | e[3:0] | m[9:7], residual byte = m[6:0]
 *                 (top bit 0 when written, ignored when read); exact only
 *                 when e's MSB is 0.  Fast-mode weight = OCP E4M3(upper) *
 *                 2^-8, a number only when |w| < 1.875.  dps_select_enc
 *                 says whether a whole layer qualifies.  The linear calls,
 *                 in both modes, assume an E4M3 layer that qualifies: words
 *                 of 1.875 <= |w| < 2 (upper byte an E4M3 NaN code) give
 *                 NaN there; dps_merge restores every word. */
enum { DPS_ENC_E5M2 = 0, DPS_ENC_E4M3 = 1 };

/* Activation handling, `flags` argument of the linear calls.
 *   DPS_ACT_FP16: activations stay FP16; weights enter the FP16 matrix cores
 *     (fast mode: the fast-mode weight is an exact FP16 word).
 *   DPS_ACT_FP8_ROWSCALE (fast mode only): each activation row is first
 *     quantized to OCP FP8 E4M3 with its own power-of-two scale (see
 *     dps_quant_rows_e4m3) and the product runs on the FP8 matrix cores with
 *     the weights' upper byte (E5M2 or E4M3) as the second operand. */
enum { DPS_ACT_FP16 = 0u, DPS_ACT_FP8_ROWSCALE = 1u };

/* Residual plane of one weight tensor (Sec. IV-B "Shared Region": physical
 * units behind one contiguous virtual tensor).  The residual bytes form a
 * logical stream in the weight's row-major element order; the stream is cut
 * into chunks of C = 2^log2_chunk bytes and logical chunk c is stored in
 * pool slot slots[c], i.e. logical byte i lives at
 *     pool + slots[i >> log2_chunk] * C + (i & (C - 1)).
 * Other pool slots may hold anything (e.g. paged KV blocks).
 *   pool        device, 16-byte aligned, pool_bytes bytes.
 *   pool_bytes  >= C; slots address pool_bytes / C whole chunks.
 *   slots       device int32[n_chunks].  Entries should be distinct; an entry
 *               outside [0, pool_bytes / C) is never dereferenced: reads
 *               through it return zero bytes and writes through it are
 *               dropped.
 *   n_chunks    >= ceil(numel / C) for the tensor it describes.
 *   log2_chunk  4..30 (chunks of 16 B .. 1 GiB).
 * In fast mode the whole descriptor is ignored and may be zero/NULL. */
typedef struct {
    uint8_t *pool;
    int64_t pool_bytes;
    const int32_t *slots;
    int64_t n_chunks;
    int32_t log2_chunk;
} dps_residual;

/* A nested weight: `experts` stacked [n][k] matrices (experts = 1 for a dense
 * layer).  Element (e, r, c) is logical element (e * n + r) * k + c of both
 * the upper-byte plane `hi` and the residual stream.
 *   hi   device uint8[experts][n][k], 16-byte aligned.
 *   k    multiple of 16, 16..2^30.   n in 1..2^31-1.   experts in 1..65535.
 *   enc  DPS_ENC_E5M2 or DPS_ENC_E4M3: the encoding hi and the residual were
 *        split with. */
typedef struct {
    const uint8_t *hi;
    dps_residual res;
    int64_t experts;
    int64_t n;
    int64_t k;
    int32_t enc;
} dps_weight;

/* Per-layer encoding choice (Sec. IV-C, "Dual-mode serving" paragraph: E5M2
 * for layers E4M3 cannot express): *enc_out = DPS_ENC_E4M3 if every word of
 * w has |w| < 1.875 (exponent MSB zero and E4M3 part a number; NaN and
 * infinities do not qualify), else DPS_ENC_E5M2.  numel == 0 gives E4M3.
 *   w        device uint16 (FP16 bit patterns) [numel], 16-byte aligned.
 *   enc_out  device int32, written by the enqueued work (read it after
 *            synchronizing the stream). */
dps_status dps_select_enc(const uint16_t *w, int64_t numel, int32_t *enc_out, void *stream);

/* Split FP16 weights into the nested pair (Sec. IV-A "Dynamic Networks and a
 * Nested Model"; Sec. IV-B "Persistent Region"): hi[i] and residual byte i of
 * w[i] under encoding `enc` (see the encoding table above), the residual
 * written through the chunk table.  E4M3 on a word whose exponent MSB is set
 * keeps the listed fields all the same and loses that bit.
 *   enc    DPS_ENC_E5M2 or DPS_ENC_E4M3.
 *   w      device uint16 (FP16 bit patterns) [numel], 16-byte aligned.
 *   hi     device uint8[numel], 16-byte aligned.
 *   res    host pointer to the residual descriptor (its pool is written).
 * numel == 0 is a no-op.  Bit-exact. */
dps_status dps_split(int enc, const uint16_t *w, int64_t numel, uint8_t *hi,
                     const dps_residual *res, void *stream);

/* Rebuild the FP16 words (Sec. IV-C "Overall concept": full mode
 * reconstructs the original FP16 values) from hi and the residual bytes
 * under encoding `enc`: E5M2 w = hi << 8 | residual; E4M3 w = sign | 0 |
 * hi's seven low bits | the residual byte's seven low bits.  Same layouts as
 * dps_split.  Bit-exact. */
dps_status dps_merge(int enc, const uint8_t *hi, const dps_residual *res, int64_t numel,
                     uint16_t *w_out, void *stream);

/* Residual restore (Sec. IV-B "Residual Backup": a pinned host copy of every
 * residual, the source for reloading residuals whose pool units KV blocks
 * have overwritten; Sec. IV-C, restoration paragraph: host-to-device copies
 * in fixed-size pieces on a copy stream of their own, overlapped with the
 * passes that run in fast mode meanwhile).  Copies logical chunks
 * [chunk_begin, chunk_end) of a residual's byte stream from `backup` into the
 * pool slots the table names, as hipMemcpyAsync host-to-device copies of at
 * most copy_bytes each (4 MiB in the paper), enqueued in order on `stream`.
 * Chunks in consecutive slots are joined before the stream is cut into
 * copies.  Other pool bytes are not touched.
 *   backup       host memory, the logical stream (numel bytes).  Allocate it
 *                pinned (hipHostMalloc) for the copies to be asynchronous.
 *   numel        bytes in the stream (elements of the weight).
 *   res          host pointer to the residual descriptor; res->slots is not
 *                read (the copies need the table on the host).
 *   slots_host   host int32[>= chunk_end], the same entries as res->slots;
 *                every entry in [chunk_begin, chunk_end) must lie in
 *                [0, pool_bytes / C) (checked; DPS_ERR_INVALID_ARG).
 *   0 <= chunk_begin <= chunk_end <= ceil(numel / C); an empty range is a
 *   no-op.  copy_bytes > 0.
 * Completion is the stream's: record an event on it for the compute stream
 * to wait on before a full-mode pass.  Bit-exact. */
dps_status dps_restore(const uint8_t *backup, int64_t numel, const dps_residual *res,
                       const int32_t *slots_host, int64_t chunk_begin, int64_t chunk_end,
                       int64_t copy_bytes, void *stream);

/* Residual backup (Sec. IV-B "Residual Backup", built once at start-up): the
 * whole logical stream (numel bytes) copied from the pool into `backup`
 * (host, pinned for asynchronous copies) with device-to-host copies of at
 * most copy_bytes on `stream`.  Arguments as dps_restore; every table entry
 * of the tensor's chunks must lie in the pool.  Bit-exact. */
dps_status dps_backup(const dps_residual *res, const int32_t *slots_host, int64_t numel,
                      uint8_t *backup, int64_t copy_bytes, void *stream);

/* Per-row FP8 quantization of activations for fast-mode prefill (this
 * reading taken here of the dynamic per-token activations of Sec. V-A
 * "Baselines"): for row r, a = max_k |x[r][k]|, scale[r] = the smallest power
 * of two s with a <= 448 * s (1 when a == 0), xq[r][k] = OCP E4M3 nearest to
 * x[r][k] / s, ties to even.  The division is exact, so this is bit-exact.
 *   x      device FP16 [m][k], 16-byte aligned, finite values.
 *   xq     device uint8 [m][k] (E4M3 codes), 16-byte aligned.
 *   scale  device float [m].
 * k must be a multiple of 16, at most 2^30. */
dps_status dps_quant_rows_e4m3(const uint16_t *x, int64_t m, int64_t k,
                               uint8_t *xq, float *scale, void *stream);

/* Workspace bytes that dps_linear (experts == 1, rows = m) or
 * dps_linear_grouped (rows = total routed rows) needs for these arguments on
 * the current device.  0 means no workspace is needed.  The workspace is
 * scratch: its contents on entry do not matter. */
size_t dps_workspace_bytes(int mode, uint32_t flags, int64_t rows, int64_t n,
                           int64_t k, int64_t experts);

/* Nested linear layer, dense (Sec. IV-C, GroupedGEMM paragraph, dense case):
 *   full mode: Y = X . merge(hi, residual)^T   (exact FP16 weights)
 *   fast mode: Y = X . fast(hi)^T              (residual not read), fast =
 *              E5M2(hi) or E4M3(hi) * 2^-8 per w->enc
 * fp32 accumulation, Y rounded to FP16 (round to nearest even).
 *   mode   DPS_MODE_FULL or DPS_MODE_FAST.
 *   flags  DPS_ACT_FP16, or DPS_ACT_FP8_ROWSCALE with DPS_MODE_FAST.
 *   x      device FP16 [m][w->k], 16-byte aligned.   m >= 0 (0: no-op).
 *   w      host pointer; w->experts must be 1.
 *   y      device FP16 [m][w->n], 16-byte aligned.
 *   ws     device scratch of ws_bytes >= dps_workspace_bytes(...), 256-byte
 *          aligned; may be NULL when that is 0. */
dps_status dps_linear(int mode, uint32_t flags, const uint16_t *x, int64_t m,
                      const dps_weight *w, uint16_t *y, void *ws, size_t ws_bytes,
                      void *stream);

/* Kernel families of the linear calls (dps_plan_info). */
enum {
    DPS_KERNEL_GEMV = 0,     /* 1-4 tokens: whole weight rows per wave, vector ALUs  */
    DPS_KERNEL_ROWS = 1,     /* up to 16 tokens: 16-row groups, whole K per block    */
    DPS_KERNEL_DECODE = 2,   /* a few tokens per expert: LDS-ring decode kernel      */
    DPS_KERNEL_GEMM_F16 = 3, /* FP16 matrix cores, weight tile x token tile          */
    DPS_KERNEL_GEMM_FP8 = 4  /* FP8 matrix cores (DPS_ACT_FP8_ROWSCALE)              */
};

/* The launch plan of a dps_linear (experts == 1) or dps_linear_grouped call
 * with these arguments on the current device, for introspection (which
 * kernel runs, how the work is tiled):
 *   info[0]  DPS_KERNEL_* family;
 *   info[1]  weight rows per block (0 for DPS_KERNEL_GEMV: whole rows per
 *            wave);
 *   info[2]  token rows per block tile (per pass for DPS_KERNEL_DECODE);
 *   info[3]  K splits (> 1: fp32 partials in the workspace, summed in a
 *            second launch);
 *   info[4]  K elements per split.
 * log2_chunk is the residual chunk size of a full-mode call (ignored in fast
 * mode).  Host only; enqueues nothing.  info: host int64[5]. */
dps_status dps_plan_info(int mode, uint32_t flags, int64_t rows, int64_t n, int64_t k,
                         int64_t experts, int32_t log2_chunk, int64_t *info);

/* Upper bound of the scratch dps_linear_static may use: 64 MiB per device.
 * dps_workspace_bytes() at or below it means the call fits. */
#define DPS_STATIC_SCRATCH_BYTES (((size_t)64) << 20)

/* dps_linear without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses that
 * forbid hipMalloc).  Same arguments, kernels and results as dps_linear; the
 * split-K partials and FP8 activation staging go to a static device array of
 * DPS_STATIC_SCRATCH_BYTES that every device the library runs on holds until
 * the process ends.  The first call on a device looks the array's address up
 * (hipGetSymbolAddress, no allocation); no call allocates or frees anything.
 * A call whose dps_workspace_bytes() exceeds DPS_STATIC_SCRATCH_BYTES returns
 * DPS_ERR_WORKSPACE with nothing enqueued.  Every call on one device shares
 * that device's array: calls that may overlap on one device (different
 * streams without ordering, several host threads) race on it and give wrong
 * results; order them on one stream. */
dps_status dps_linear_static(int mode, uint32_t flags, const uint16_t *x, int64_t m,
                             const dps_weight *w, uint16_t *y, void *stream);

/* Grouped nested linear for MoE experts (Sec. IV-C, GroupedGEMM paragraph,
 * MoE case): rows [offsets[e], offsets[e+1]) of x_sorted are multiplied by
 * expert e's weights; Y rows follow the same order.
 *   x_sorted  device FP16 [rows][w->k], rows grouped by expert.
 *   offsets   device int32[w->experts + 1]; offsets[0] = 0, nondecreasing,
 *             offsets[experts] = rows.  Read on the device only, so the call
 *             does not synchronize; rows outside [0, rows) are never touched
 *             even if the array breaks this contract.
 *   y         device FP16 [rows][w->n].
 * With w->experts == 1 the call is the dense one (dps_linear on all rows,
 * same kernels and results); offsets is then checked but not read.
 * Other arguments as dps_linear.  With DPS_ACT_FP8_ROWSCALE (fast mode only)
 * every row of x_sorted is quantized to E4M3 with its own power-of-two scale,
 * as in dps_quant_rows_e4m3, and multiplied on the FP8 matrix cores against
 * its expert's upper bytes (Sec. IV-C: fast-mode prefill, MoE case). */
dps_status dps_linear_grouped(int mode, uint32_t flags, const uint16_t *x_sorted,
                              const int32_t *offsets, int64_t rows, const dps_weight *w,
                              uint16_t *y, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------------------
 * SUM manager (Sec. IV-B "SUM manager"; Sec. IV-D, Algorithm 1): host-side
 * bookkeeping of the shared region's physical units.  A unit holds either
 * one residual tensor (BACKED) or KV blocks (AVAIL: some free, FULL: none
 * free), or nothing (FREE); RESTORING units are held for a residual being
 * copied back.  Residual r starts bound to unit r.  Taking a BACKED unit for
 * KV evicts its residual: the mapping goes stale, the data lives only in the
 * host backup, and the mode is fast until every evicted residual is back.
 * Sets are ordered by unit id; a pop takes the lowest id and a unit hands out
 * its lowest free block indices first.  Block id = unit * blocks_per_unit +
 * index.  Not thread-safe: one caller (the serving loop) drives it.
 * ------------------------------------------------------------------------ */
enum { DPS_UNIT_FREE = 0, DPS_UNIT_BACKED = 1, DPS_UNIT_AVAIL = 2, DPS_UNIT_FULL = 3,
       DPS_UNIT_RESTORING = 4 };

typedef struct dps_sum dps_sum;

/* n_units >= 1 units of blocks_per_unit >= 1 KV blocks; n_res (0..n_units)
 * residuals bound to units 0 .. n_res-1, the other units FREE, mode full.
 * *out receives the manager (free it with dps_sum_destroy). */
dps_status dps_sum_create(int64_t n_units, int64_t blocks_per_unit, int64_t n_res,
                          dps_sum **out);
void dps_sum_destroy(dps_sum *s);

/* AllocKVBlock(n) of Algorithm 1: blocks from AVAIL units first, then a FREE
 * unit, then a BACKED unit (evicting its residual, switching to fast mode).
 * The n block ids go to blocks[0..n).  A request larger than the room left
 * in AVAIL, FREE and BACKED units takes nothing and returns
 * DPS_ERR_NO_SPACE. */
dps_status dps_sum_alloc(dps_sum *s, int64_t n, int64_t *blocks);

/* FreeKVBlock(blocks) of Algorithm 1: FULL units with a freed block become
 * AVAIL, units with no block left become FREE, and *wake (may be NULL) is
 * set to 1 if that happened while residuals wait for restoration.  Blocks
 * that are not allocated, or listed twice, fail the whole call with
 * DPS_ERR_INVALID_ARG and change nothing. */
dps_status dps_sum_free(dps_sum *s, const int64_t *blocks, int64_t n, int32_t *wake);

/* Restore worker, first step: the lowest stale residual is bound to the
 * lowest FREE unit, which turns RESTORING.  *residual and *unit receive them,
 * or -1 when nothing is stale or no unit is free.  The caller then copies
 * the residual's bytes into that unit (dps_sum_slots, dps_restore) and calls
 * dps_sum_restore_done once the copy has completed. */
dps_status dps_sum_restore_begin(dps_sum *s, int64_t *residual, int64_t *unit);

/* The copy of `residual` has completed: its unit becomes BACKED; when no
 * residual is left evicted the mode returns to full. */
dps_status dps_sum_restore_done(dps_sum *s, int64_t residual);

/* DPS_MODE_FULL or DPS_MODE_FAST (-1 for NULL). */
int32_t dps_sum_mode(const dps_sum *s);
/* DPS_UNIT_* state of a unit (-1 if out of range). */
int32_t dps_sum_unit_state(const dps_sum *s, int64_t unit);
/* Unit a residual is bound to or being restored into; -1 while evicted. */
int64_t dps_sum_unit_of(const dps_sum *s, int64_t residual);
/* counts[0..8): |FREE|, |BACKED|, |AVAIL|, |FULL|, |RESTORING|, |STALE|,
 * |EVICTED|, free blocks in AVAIL units. */
dps_status dps_sum_counts(const dps_sum *s, int64_t *counts);
/* Host slot table of a residual of n_chunks <= chunks_per_unit chunks in
 * its unit u, where unit u spans pool slots [u * chunks_per_unit,
 * (u + 1) * chunks_per_unit): slots_host[c] = u * chunks_per_unit + c.  The
 * residual must be bound or being restored (else DPS_ERR_INVALID_ARG). */
dps_status dps_sum_slots(const dps_sum *s, int64_t residual, int64_t chunks_per_unit,
                         int64_t n_chunks, int32_t *slots_host);

/* ------------------------------------------------------------------------
 * Restore worker (Sec. IV-B "SUM manager": a background thread drains the
 * restore queue; Sec. IV-C restoration paragraph: copies on their own
 * stream, beside fast-mode passes).  A host thread that, each time it is
 * woken, takes restores from the SUM manager for as long as it hands them
 * out (dps_sum_restore_begin): it rewrites the residual's device chunk table
 * (res.slots, chunks_per_unit slots per unit, dps_sum_slots) to the unit it
 * was given, copies the host backup into those slots (as dps_restore, in
 * copies of at most copy_bytes) on a stream of its own, waits for them and
 * reports dps_sum_restore_done.  The SUM manager is safe to call from the
 * serving loop meanwhile; it must outlive the worker.  Only full-mode calls
 * read a residual, and the mode is full only after every copy completed.
 * ------------------------------------------------------------------------ */
typedef struct {
    const uint8_t *backup; /* host backup of the residual's logical stream
                              (dps_backup), pinned for asynchronous copies  */
    int64_t numel;         /* its bytes                                       */
    dps_residual res;      /* the descriptor the linear calls use; the worker
                              rewrites the device table res.slots points to   */
} dps_restore_target;

typedef struct dps_restore_worker dps_restore_worker;

/* A worker for the SUM manager's residuals 0 .. n_targets-1 (targets: host
 * array, copied; each residual's n_chunks at most chunks_per_unit), on the
 * current device.  Free it with dps_restore_worker_destroy. */
dps_status dps_restore_worker_create(dps_sum *sum, const dps_restore_target *targets,
                                     int64_t n_targets, int64_t chunks_per_unit,
                                     int64_t copy_bytes, dps_restore_worker **out);
/* Wake the worker (after KV blocks were freed, or any time). */
dps_status dps_restore_worker_kick(dps_restore_worker *w);
/* Wait until the worker has taken up every wake-up and has nothing left it
 * can restore: DPS_OK, DPS_ERR_TIMEOUT after timeout_ms, or the error that
 * stopped the worker (it then restores nothing more). */
dps_status dps_restore_worker_wait_idle(dps_restore_worker *w, int64_t timeout_ms);
/* Residuals restored so far (-1 for NULL). */
int64_t dps_restore_worker_restored(dps_restore_worker *w);
/* Stop the thread (a restore in progress completes first) and free it. */
void dps_restore_worker_destroy(dps_restore_worker *w);
/* Detail of the last dps_restore_worker_* error on the calling thread. */
const char *dps_restore_worker_last_error(void);

/* ------------------------------------------------------------------------
 * Shared region through the HIP virtual memory API (Sec. IV-B "Shared
 * Region", dual-mapping property): n_units physical units of unit_bytes
 * each, mapped once in unit order into the KV view and again, per residual
 * tensor, into a residual view whose piece i maps the unit holding the
 * tensor's chunk i.  The residual view is contiguous, so the residual
 * descriptor {pool = view, pool_bytes = count * unit_bytes, slots = the
 * identity table 0 .. count-1, log2_chunk = log2(unit_bytes)} addresses it
 * in every call above, and a byte written through either view is the same
 * physical byte.  This is the optional allocator of the region (the linear
 * path itself never allocates).  Mapping changes are not ordered with work
 * queued on any stream: nothing that uses a view may run while the view is
 * remapped or unmapped.  Host calls; they work on the device current at
 * dps_vmm_create and leave the caller's current device as it was.  A HIP
 * runtime without VMM support gives DPS_ERR_UNSUPPORTED.
 * ------------------------------------------------------------------------ */
typedef struct dps_vmm dps_vmm;

/* Minimum VMM allocation granularity of the current device, bytes. */
dps_status dps_vmm_granularity(int64_t *bytes_out);

/* n_units (1..2^20) units of unit_bytes (a power of two, 4 KiB..1 GiB, a
 * multiple of the granularity) on the current device, all mapped into the
 * KV view.  *out is owned by the caller (dps_vmm_destroy). */
dps_status dps_vmm_create(int64_t n_units, int64_t unit_bytes, dps_vmm **out);

/* The KV view: device address of n_units * unit_bytes bytes, unit u at
 * u * unit_bytes (NULL for a NULL region). */
void *dps_vmm_kv_view(const dps_vmm *v);
int64_t dps_vmm_unit_bytes(const dps_vmm *v);

/* A new residual view of count (1..64 * n_units) pieces, piece i mapping
 * unit units_host[i] (host int32, each in 0..n_units-1); *view_out its
 * device address. */
dps_status dps_vmm_map_residual(dps_vmm *v, const int32_t *units_host, int64_t count,
                                void **view_out);

/* Map unit `unit` at piece `piece` of a residual view instead of the unit
 * there (a residual restored into another unit).  If mapping the new unit
 * fails, the piece is left unmapped (the call returns the error): nothing
 * may read the view until a later remap of that piece succeeds. */
dps_status dps_vmm_remap(dps_vmm *v, void *view, int64_t piece, int32_t unit);

/* Unmap a residual view and free its address range. */
dps_status dps_vmm_unmap_residual(dps_vmm *v, void *view);

/* Unmap every view and release the units (NULL: no-op). */
void dps_vmm_destroy(dps_vmm *v);

/* Detail of the last dps_vmm_* error on the calling thread ("" if none). */
const char *dps_vmm_last_error(void);

/* Static description of a status code. */
const char *dps_status_str(dps_status s);

/* Detail of the last error returned on the calling thread ("" if none). */
const char *dps_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DPS_H */
