/*
 * dps_probe.h -- measured ceilings of the MI355X units the nested linear
 * layer is bound by (HBM streaming, FP16 and FP8 matrix cores), so roofline
 * fractions can be stated against what the part delivers as well as against
 * its published peaks.  A separate library (libdps_probe.so), not part of the
 * nested-linear boundary in dps.h.
 *
 * Each call enqueues one kernel on `stream` (a hipStream_t) and returns 0, or
 * 1 for a bad argument (nothing enqueued), or 5 if the launch failed.  Time
 * them with events around the enqueued work.
 */
#ifndef DPS_PROBE_H
#define DPS_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Read every byte of buf once with 16-byte loads (1 KiB per wave
 * instruction; nontemporal != 0: nontemporal loads) over `blocks` blocks of
 * 256 threads, block b over the b-th of `blocks` equal contiguous chunks.  buf: device, 16-byte aligned, bytes a positive
 * multiple of 16.  out: device uint32[blocks], one folded word per block. */
int dps_probe_stream_read(const void *buf, int64_t bytes, int nontemporal, uint32_t *out,
                          int64_t blocks, void *stream);

/* `blocks` blocks of four waves, each wave issuing 8 * iters MFMAs on
 * register operands (fp8 == 0: v_mfma_f32_16x16x32_f16, 16384 flops each;
 * fp8 != 0: v_mfma_f32_16x16x128_f8f6f4 with E4M3 operands, 65536 flops
 * each).  out: device float[blocks * 256]. */
int dps_probe_mfma(int fp8, int iters, int64_t blocks, float *out, void *stream);

/* The FP16 GEMMs' compute loop alone: `blocks` blocks, shape 0: eight waves
 * of 64 x 128 wave tiles (the 256 x 256 tile's grid), shape 1: four waves of
 * 128 x 64 (one wave per SIMD); per 64-element stage every wave reads its weight and token
 * fragments from LDS (merge != 0: weight fragments from two byte planes
 * interleaved into FP16, as full mode does) and runs 2 x (TN/16) x (TM/16)
 * v_mfma_f32_16x16x32_f16 (16384 flops each); barrier != 0 ends every stage
 * at a block barrier.  iters stages; no global memory inside the loop.
 * out: device float[blocks * 64 * waves]. */
int dps_probe_mfma_lds(int shape, int merge, int barrier, int iters, int64_t blocks, float *out,
                       void *stream);

/* The global -> LDS fill of the GEMMs, alone: `blocks` blocks (one per CU
 * when blocks = CUs; 128 KiB of LDS each) of `loaders` waves (4, 8 or 16),
 * which fill iters stages of 64 KiB by direct-to-LDS loads of 8 rows x 128
 * bytes per instruction from rows 4 KiB apart inside the first window_bytes
 * of buf, into a two-slot ring with one barrier per stage.  Bytes moved:
 * 65536 * iters * blocks.  buf: device, 16-byte aligned; window_bytes a
 * multiple of 4096, at least 1 MiB.  out: device uint32[blocks]. */
int dps_probe_lds_fill(const void *buf, int64_t window_bytes, int loaders, int iters,
                       int64_t blocks, uint32_t *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DPS_PROBE_H */
