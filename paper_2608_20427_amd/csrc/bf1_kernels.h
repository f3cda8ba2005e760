// Internal interface between the C-ABI shim and the device kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bf1 {

struct AttnArgs {
    const void* Q;
    const void* K;
    const void* V;
    void* O;
    float* LSE;             // may be null
    const int32_t* row_ptr; // null for the dense route
    const int32_t* col_idx;
    int64_t nnz;
    int32_t batch;
    int64_t n;
    int32_t Hq;
    int32_t Hkv;
    int32_t head_dim;       // 64 or 128
    int32_t B;              // block width 64 or 128 (BF1 route)
    bool dense;             // implicit route {0..j} over 64-token blocks
};

// Route planner: row_ptr[0..NB], col_idx[0..nnz) on `stream`.
hipError_t launch_plan(int32_t NB, int32_t L, int32_t* row_ptr, int32_t* col_idx,
                       hipStream_t stream);

// Attention forward (validated arguments only).
hipError_t launch_attention(const AttnArgs& a, hipStream_t stream);

}  // namespace bf1
