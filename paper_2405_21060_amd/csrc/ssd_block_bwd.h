// Internal interface of the block-gradient kernels (ssd_block_bwd.hip) for the
// C-ABI host layer.  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ssd {

struct BlockBwdParams {
    int64_t rows;          // b * T
    int64_t H, C;          // heads; channels per row (H * P)
    int64_t group;         // normalisation group (channels), 0 = none
    // dt step
    const void* dt_raw;    // (rows, H) dtype
    const float* bias;     // (H) or null
    int softplus;
    float lo, hi;
    void* dt;              // (rows, H) float32: the step's output (workspace)
    const void* ddt;       // (rows, H) float32: gradient of the layer's dt
    void* ddt_raw;         // (rows, H) dtype: output
    float* dbias_part;     // (row chunks, H) workspace, or null
    float* ddt_bias;       // (H) output, or null
    // gate and normalisation
    const void* y;         // (rows, C) float32: the layer's output (workspace)
    const void* z;         // (rows, C) dtype, or null
    const float* w;        // (C), or null
    float eps;
    const void* dout;      // (rows, C) dtype: gradient of the block's output
    void* dy;              // (rows, C) float32: gradient of the layer's output (workspace)
    void* dz;              // (rows, C) dtype output, or null
    float* inv_rms;        // (rows, C / group) workspace
    float* dw_part;        // (row chunks, C) workspace
    float* dw;             // (C) output, or null
};

// Row chunks of the per-chunk partial sums (dbias_part, dw_part).
int64_t block_bwd_row_chunks(int64_t rows);

hipError_t launch_block_dt_apply(const BlockBwdParams& p, bool bf16, hipStream_t stream);
// dy (and dz, dw) from dout: gate and / or normalisation (at least one active).
hipError_t launch_block_out_bwd(const BlockBwdParams& p, bool bf16, hipStream_t stream);
// ddt_raw (and ddt_bias) from ddt.
hipError_t launch_block_dt_bwd(const BlockBwdParams& p, bool bf16, hipStream_t stream);

// n bf16 values to float32 (exact), and float32 to bf16 (nearest even).
hipError_t launch_widen(const void* src, float* dst, int64_t n, hipStream_t stream);
hipError_t launch_narrow(const float* src, void* dst, int64_t n, hipStream_t stream);

}  // namespace ssd
