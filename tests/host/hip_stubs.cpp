// Host-only stand-ins for the HIP runtime calls and kernel launchers that the
// C-ABI shim (bf1_api.cpp) makes, for a sanitizer build that loads no GPU
// runtime.  Mode "fail": every call reports an error (the shim must map it to
// BF1_ERR_HIP).  Mode "host": allocations are host heap blocks, launches
// record their arguments and succeed, and the capture status is settable.
#include <hip/hip_runtime_api.h>

#include <cstdlib>
#include <cstring>

#include "../../paper_2608_20427_amd/csrc/bf1_kernels.h"
#include "hip_stubs.h"

StubState g_stub;

extern "C" {
hipError_t hipGetDevice(int* d) {
    if (g_stub.fail) return hipErrorNoDevice;
    *d = 0;
    return hipSuccess;
}
hipError_t hipMalloc(void** p, size_t n) {
    if (g_stub.fail) return hipErrorOutOfMemory;
    ++g_stub.mallocs;
    *p = std::malloc(n ? n : 1);
    return *p ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipFree(void* p) {
    if (p) ++g_stub.frees;
    std::free(p);
    return hipSuccess;
}
hipError_t hipMemcpy(void* dst, const void* src, size_t n, hipMemcpyKind) {
    if (g_stub.fail) return hipErrorInvalidValue;
    std::memcpy(dst, src, n);
    return hipSuccess;
}
hipError_t hipStreamIsCapturing(hipStream_t, hipStreamCaptureStatus* st) {
    if (g_stub.fail) return hipErrorInvalidValue;
    *st = g_stub.capturing ? hipStreamCaptureStatusActive : hipStreamCaptureStatusNone;
    return hipSuccess;
}
hipError_t hipStreamCreateWithFlags(hipStream_t* s, unsigned int) {
    if (g_stub.fail) return hipErrorInvalidValue;
    static int token;
    *s = reinterpret_cast<hipStream_t>(&token);
    return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return g_stub.fail ? hipErrorInvalidValue : hipSuccess; }
hipError_t hipDeviceSynchronize(void) { return g_stub.fail ? hipErrorInvalidValue : hipSuccess; }
}

namespace bf1 {
hipError_t launch_plan(int32_t NB, int32_t, int32_t* row_ptr, int32_t* col_idx, hipStream_t) {
    if (g_stub.fail) return hipErrorLaunchFailure;
    ++g_stub.plans;
    // touch the whole table the shim sized, so the sanitizer checks the sizes
    for (int32_t j = 0; j <= NB; ++j) row_ptr[j] = 0;
    (void)col_idx;
    return hipSuccess;
}
hipError_t launch_attention(const AttnArgs& a, hipStream_t) {
    if (g_stub.fail) return hipErrorLaunchFailure;
    ++g_stub.attns;
    g_stub.last_nnz = a.nnz;
    return hipSuccess;
}
hipError_t launch_backward(const BwdArgs& a, hipStream_t) {
    if (g_stub.fail) return hipErrorLaunchFailure;
    ++g_stub.bwds;
    // read every host-built descriptor the shim uploaded
    long sum = 0;
    for (int64_t e = 0; e < a.nusers; ++e) sum += a.users[e];
    for (int32_t s = 0; s < a.nseg * 8; ++s) sum += a.segs[s];
    for (int32_t r = 0; r < a.nred * 4; ++r) sum += a.reds[r];
    g_stub.last_nnz = sum;
    return hipSuccess;
}
hipError_t launch_decode_plan(const DecodePlanArgs&, hipStream_t) {
    return g_stub.fail ? hipErrorLaunchFailure : hipSuccess;
}
hipError_t launch_decode(const DecodeArgs&, hipStream_t) {
    return g_stub.fail ? hipErrorLaunchFailure : hipSuccess;
}
hipError_t noalloc_scratch(int32_t** ptr) {
    if (g_stub.fail) return hipErrorInvalidSymbol;
    static int32_t table[kNoallocInts];
    *ptr = table;
    return hipSuccess;
}
}  // namespace bf1
