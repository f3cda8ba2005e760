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
    int32_t key_split = 0;  // 0 automatic, 1 one key group, 2 two key groups per workgroup
};

// Backward (head_dim 64 or 128; G * B >= 128).  All pointers are device memory.
struct BwdArgs {
    const void* Q;
    const void* K;
    const void* V;
    const void* O;
    const void* dO;
    const float* LSE;
    float* dQ;               // [batch, Hq, n, head_dim] fp32
    float* dK;               // [batch, Hkv, n, head_dim] fp32
    float* dV;
    float* delta;            // workspace: [batch, Hq, n] fp32 (D = rowsum(dO * O))
    float* lse2;             // workspace: [batch, Hq, n] fp32 (LSE * log2 e)
    float* part;             // workspace: [batch * Hkv, nslots, 2, 64, head_dim] fp32
    void* ds;                // workspace: dS units, [batch * Hkv, nusers, B/64, B/64, Hq/Hkv] x 8 KB bf16
    const int32_t* row_ptr;  // forward route (CSR)
    const int32_t* col_idx;
    int64_t nnz;
    const int32_t* users;    // transposed route entries (query blocks per key block)
    const int32_t* uoffs;    // [NB + 1]: first entry of each key block's list in users
    int64_t nusers;          // entries of the transposed route
    const int32_t* segs;     // [nseg][8]: key block, sub-tile, first entry, count, slot
    int32_t nseg;
    const int32_t* reds;     // [nred][4]: key block, sub-tile, first slot, slot count
    int32_t nred;
    int32_t nslots;
    int32_t batch;
    int64_t n;
    int32_t Hq;
    int32_t Hkv;
    int32_t B;               // block width 64 or 128
    int32_t head_dim;        // 64 or 128
    int32_t L;               // local width of the route
};

hipError_t launch_backward(const BwdArgs& a, hipStream_t stream);

// One-token decode over a paged cache (validated arguments only).
struct DecodePlanArgs {
    int32_t batch;
    const int32_t* seq_lens;    // [batch]
    const int32_t* page_table;  // [batch, max_pages]
    int32_t max_pages;
    int32_t num_pages;
    int32_t B;                  // page = block width
    int32_t L;
    int32_t dense;              // 1: every earlier block (dense comparator)
    int32_t* plan;              // [batch, stride]
    int32_t stride;
    int32_t cap;                // stride - 3
};
hipError_t launch_decode_plan(const DecodePlanArgs& a, hipStream_t stream);

struct DecodeArgs {
    const void* Q;              // [batch, Hq, head_dim] bf16
    const void* K;              // [num_pages, Hkv, B, head_dim] bf16
    const void* V;
    const int32_t* seq_lens;
    int32_t num_pages;
    const int32_t* plan;
    int32_t stride;
    int32_t cap;
    void* O;                    // [batch, Hq, head_dim] bf16
    float* LSE;                 // [batch, Hq] or null
    float* ws;                  // [batch * Hkv * nsplit, G * (head_dim + 2)] fp32
    int32_t batch;
    int32_t Hq;
    int32_t Hkv;
    int32_t head_dim;           // 64 or 128
    int32_t B;                  // 64 or 128
    int32_t nsplit;             // splits per (sequence, kv-head), <= 256
    int32_t ppw;                // pages per split
};
hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);

// Fixed device scratch of the forward that allocates nothing: capacity in
// int32 entries (row_ptr and col_idx of one route table), and the address of
// the current device's copy (looked up once per device, then cached).
constexpr int64_t kNoallocInts = int64_t(1) << 20;  // 4 MiB
hipError_t noalloc_scratch(int32_t** ptr);

// Route planner: row_ptr[0..NB], col_idx[0..nnz) on `stream`.
hipError_t launch_plan(int32_t NB, int32_t L, int32_t* row_ptr, int32_t* col_idx,
                       hipStream_t stream);

// Attention forward (validated arguments only).
hipError_t launch_attention(const AttnArgs& a, hipStream_t stream);

}  // namespace bf1
