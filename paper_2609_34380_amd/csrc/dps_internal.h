// dps_internal.h -- host-side launch interface between the C ABI (dps_api.hip)
// and the kernel files.  Every launcher enqueues on `stream` and returns the
// hipError_t of the launch; arguments are already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dps_device.h"

namespace dps {

// ---- elementwise ------------------------------------------------------------
hipError_t launch_split(int enc, const uint16_t *w, int64_t numel, uint8_t *hi,
                        const ResidualView &res, hipStream_t stream);
hipError_t launch_merge(int enc, const uint8_t *hi, const ResidualView &res, int64_t numel,
                        uint16_t *w_out, hipStream_t stream);
// *enc_out = ENC_E4M3 if every word nests losslessly into E4M3 with a finite
// E4M3 part, else ENC_E5M2 (two launches: set, then clear on any misfit).
hipError_t launch_select_enc(const uint16_t *w, int64_t numel, int32_t *enc_out,
                             hipStream_t stream);
hipError_t launch_quant_rows(const uint16_t *x, int64_t m, int64_t k, uint8_t *xq, float *scale,
                             hipStream_t stream);
// y[r][c] = fp16(sum_s partial[s][r][c]) for r < rows, c < n, s in order.
hipError_t launch_splitk_reduce(const float *partial, int splits, int64_t rows, int64_t n,
                                uint16_t *y, hipStream_t stream);

// ---- residual backup / restore (host-issued DMA copies) ----------------------
// Logical chunks [c0, c1) of the stream `backup` (numel bytes, host) into the
// pool slots slots_host names, as copies of at most copy_bytes on `stream`.
hipError_t launch_restore(const uint8_t *backup, int64_t numel, const ResidualView &r,
                          const int32_t *slots_host, int64_t c0, int64_t c1,
                          int64_t copy_bytes, hipStream_t stream);
// The whole logical stream from the pool into `backup` (host).
hipError_t launch_backup(const ResidualView &r, const int32_t *slots_host, int64_t numel,
                         uint8_t *backup, int64_t copy_bytes, hipStream_t stream);

// ---- linear -------------------------------------------------------------------
// A linear problem: rows of x grouped by expert (offsets == nullptr: one
// expert owning rows [0, rows)), weights [experts][n][k].
struct LinearProblem {
    int mode;
    int enc;
    const uint16_t *x;
    const int32_t *offsets;  // device, experts + 1 entries, or nullptr
    int64_t rows;
    int64_t experts, n, k;
    const uint8_t *hi;
    ResidualView res;
    uint16_t *y;
};

enum KernelKind { KIND_SKINNY = 0, KIND_GEMM_F16 = 1, KIND_GEMM_FP8 = 2, KIND_GEMV = 3, KIND_ROWS = 4 };
// GEMM tile variants (weight rows x tokens per block).
enum GemmVariant {
    // FP8 activations: eight-wave LDS-DMA kernel
    GEMM_G3_256x256 = 0,
    GEMM_G3_256x128 = 1,
    // FP16 activations: 128-element stages with wide-row loads, K split over
    // waves; up to 32 tokens the eight compute waves issue the DMA, from 64
    // tokens on four dedicated DMA waves do (the planner's three tiles)
    GEMM_G4_128x32 = 2,
    GEMM_G4S_128x64 = 3,
    GEMM_G4S_128x128 = 4,
    // FP16 activations, prefill: 256 weight rows x 256 tokens, 64-element
    // stages, 128 x 64 wave tiles
    GEMM_G5_256x256 = 5
};
// Decode-kernel variants 0 and 1 keep the weight stream in registers (16 or
// 32 weight rows per wave); SKINNY_RING streams it through per-wave LDS rings.
enum { SKINNY_RING = 2 };

// Kernel choice and work split for one call.  plan_linear is the single
// place that decides; dps_workspace_bytes and the launch both call it.
struct LinearPlan {
    int kind;
    int variant;       // kernel-family specific tile variant
    int splits;        // K is cut into `splits` ranges of `ksplit` elements
    int64_t ksplit;
    bool range_addr;   // each row's residual range in a split spans <= 2 chunks
    size_t ws_partial; // fp32 split-K partials, bytes
    size_t ws_quant;   // E4M3 activations + row scales, bytes
};

LinearPlan plan_linear(int mode, uint32_t flags, int64_t rows, int64_t n, int64_t k,
                       int64_t experts, int log2c, int cu_count, bool grouped);

hipError_t launch_skinny(const LinearProblem &p, const LinearPlan &plan, float *partial,
                         hipStream_t stream);
// Dense 1-4 token calls on the vector ALUs, whole rows per wave (no K split).
hipError_t launch_gemv(const LinearProblem &p, const LinearPlan &plan, hipStream_t stream);
// Dense calls of up to 16 tokens on the matrix cores, plan.variant = 16-row
// groups per block (1-8), whole K per block (no K split).
hipError_t launch_rows(const LinearProblem &p, const LinearPlan &plan, hipStream_t stream);
hipError_t launch_gemm_f16(const LinearProblem &p, const LinearPlan &plan, float *partial,
                           hipStream_t stream);
// FP8 activations (E4M3 codes and row scales from launch_quant_rows) against
// the upper bytes; offsets == nullptr: dense, else rows grouped by expert as
// in LinearProblem (weights [experts][n][k]).
hipError_t launch_gemm_fp8(int enc, const uint8_t *xq, const float *scale, const int32_t *offsets,
                           int64_t m, int64_t experts, int64_t n, int64_t k, const uint8_t *hi,
                           uint16_t *y, const LinearPlan &plan, float *partial, hipStream_t stream);

}  // namespace dps
