// State of the host-only HIP stand-ins (hip_stubs.cpp).
#pragma once
#include <cstdint>

struct StubState {
    bool fail = false;       // every runtime call and launch reports an error
    bool capturing = false;  // hipStreamIsCapturing reports an active capture
    long mallocs = 0, frees = 0, plans = 0, attns = 0, bwds = 0;
    int64_t last_nnz = 0;
};
extern StubState g_stub;
