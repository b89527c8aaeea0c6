// dps_internal.h -- host-side launch interface between the C ABI (dps_api.hip)
// and the kernel files.  Every launcher enqueues on `stream` and returns the
// hipError_t of the launch; arguments are already validated.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dps_device.h"

namespace dps {

// ---- elementwise ------------------------------------------------------------
hipError_t launch_split(const uint16_t *w, int64_t numel, uint8_t *hi, const ResidualView &res,
                        hipStream_t stream);
hipError_t launch_merge(const uint8_t *hi, const ResidualView &res, int64_t numel,
                        uint16_t *w_out, hipStream_t stream);
hipError_t launch_quant_rows(const uint16_t *x, int64_t m, int64_t k, uint8_t *xq, float *scale,
                             hipStream_t stream);
// y[r][c] = fp16(sum_s partial[s][r][c]) for r < rows, c < n, s in order.
hipError_t launch_splitk_reduce(const float *partial, int splits, int64_t rows, int64_t n,
                                uint16_t *y, hipStream_t stream);

// ---- linear -------------------------------------------------------------------
// A linear problem: rows of x grouped by expert (offsets == nullptr: one
// expert owning rows [0, rows)), weights [experts][n][k].
struct LinearProblem {
    int mode;
    const uint16_t *x;
    const int32_t *offsets;  // device, experts + 1 entries, or nullptr
    int64_t rows;
    int64_t experts, n, k;
    const uint8_t *hi;
    ResidualView res;
    uint16_t *y;
};

enum KernelKind { KIND_SKINNY = 0, KIND_GEMM_F16 = 1, KIND_GEMM_FP8 = 2 };
// FP16 GEMM variants: register-staged 128-token tiles, or the LDS-DMA pipeline
// with 128- or 256-token tiles (128 weight rows each).
enum GemmVariant {
    GEMM_REG_128 = 0,
    GEMM_DMA_128 = 1,
    GEMM_DMA_256 = 2,
    // eight-wave LDS-DMA kernels: weight rows x tokens per block
    GEMM_G3_256x256 = 3,
    GEMM_G3_128x256 = 4,
    GEMM_G3_256x128 = 5,
    GEMM_G3_128x128 = 6,
    GEMM_G3_256x256_W16 = 7,  // 256 x 256 with sixteen waves (four per SIMD)
    // 128 weight rows x 128/64/32 tokens, 128-element stages with wide-row
    // loads, K split over waves
    GEMM_G4_128x128 = 8,
    GEMM_G4_128x64 = 9,
    GEMM_G4_128x32 = 10,
    // the same with four dedicated DMA waves
    GEMM_G4S_128x128 = 11,
    GEMM_G4S_128x64 = 12,
    GEMM_G4S_128x32 = 13
};
// Decode-kernel variants 0..3 keep the weight stream in registers (tile
// shapes differ); SKINNY_RING streams it through per-wave LDS rings.
enum { SKINNY_RING = 4, SKINNY_RING_HALF = 5 };

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
hipError_t launch_gemm_f16(const LinearProblem &p, const LinearPlan &plan, float *partial,
                           hipStream_t stream);
hipError_t launch_gemm_fp8(const uint8_t *xq, const float *scale, int64_t m, int64_t n,
                           int64_t k, const uint8_t *hi, uint16_t *y, const LinearPlan &plan,
                           float *partial, hipStream_t stream);

}  // namespace dps
