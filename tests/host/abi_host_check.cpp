// Host-side checks of the C-ABI shim under AddressSanitizer / UBSan and the
// checked standard library (built by tests/test_host_sanitized.py with the
// HIP runtime and the kernel launchers replaced by hip_stubs.cpp).
//
// Every buffer the host-only entry points write or read is a heap block of
// exactly the size the interface states, so any access past it is reported.
// Prints the host-built tables as "table <kind> <n> <B> <L> <row_ptr...> | <col_idx...>"
// lines for comparison with the oracle, and "ALL OK" at the end.
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "../../include/bf1.h"
#include "hip_stubs.h"

static int g_failures = 0;
#define CHECK(cond)                                                         \
    do {                                                                    \
        if (!(cond)) {                                                      \
            std::printf("FAIL line %d: %s\n", __LINE__, #cond);             \
            ++g_failures;                                                   \
        }                                                                   \
    } while (0)

static void print_table(const char* kind, long n, int B, int L, const std::vector<int32_t>& rp,
                        const std::vector<int32_t>& ci) {
    std::printf("table %s %ld %d %d", kind, n, B, L);
    for (int32_t x : rp) std::printf(" %d", x);
    std::printf(" |");
    for (int32_t x : ci) std::printf(" %d", x);
    std::printf("\n");
}

static void host_tables(long n, int B, int L) {
    int32_t NB = 0;
    int64_t nnz = 0, pairs = 0;
    CHECK(bf1_plan_size(n, B, L, &NB, &nnz, &pairs) == BF1_OK);
    // transposed route, exact-size buffers; one entry short is refused untouched
    {
        std::vector<int32_t> rp(NB + 1), ci(nnz > 0 ? nnz : 0);
        CHECK(bf1_plan_transposed(n, B, L, rp.data(), ci.data(), nnz) == BF1_OK);
        print_table("transposed", n, B, L, rp, ci);
        if (nnz > 0) {
            // (at least one element, so the pointer is never null: a null
            // col_idx with entries to write is an invalid argument instead)
            std::vector<int32_t> rp2(NB + 1, -7), ci2(nnz > 1 ? nnz - 1 : 1, -7);
            CHECK(bf1_plan_transposed(n, B, L, rp2.data(), ci2.data(), nnz - 1) == BF1_ERR_BUFFER_TOO_SMALL);
            bool untouched = true;
            for (int32_t x : ci2) untouched = untouched && x == -7;
            for (int32_t x : rp2) untouched = untouched && x == -7;
            CHECK(untouched);
        }
    }
    static const char* names[3] = {"bf1", "sliding", "static_random"};
    for (int kind = 0; kind < 3; ++kind) {
        std::vector<int32_t> rp(NB + 1), ci(nnz > 0 ? nnz : 0);
        CHECK(bf1_plan_variant(kind, n, B, L, 17, rp.data(), ci.data(), nnz) == BF1_OK);
        print_table(names[kind], n, B, L, rp, ci);
        if (NB <= 16384) {
            int32_t depth = -2;
            CHECK(bf1_route_depth(rp.data(), nnz > 0 ? ci.data() : nullptr, NB, &depth) == BF1_OK);
            std::printf("depth %s %ld %d %d %d\n", names[kind], n, B, L, depth);
        }
        if (nnz > 0) {
            std::vector<int32_t> ci2(nnz > 1 ? nnz - 1 : 1);
            CHECK(bf1_plan_variant(kind, n, B, L, 17, rp.data(), ci2.data(), nnz - 1) ==
                  BF1_ERR_BUFFER_TOO_SMALL);
        }
    }
    CHECK(bf1_plan_variant(3, n, B, L, 17, nullptr, nullptr, 0) == BF1_ERR_INVALID_ARG);
}

static void malformed_depth_tables() {
    int32_t d = 0;
    {   // row_ptr must start at 0
        std::vector<int32_t> rp = {1, 1, 2}, ci = {0, 0};
        CHECK(bf1_route_depth(rp.data(), ci.data(), 2, &d) == BF1_ERR_INVALID_ARG);
    }
    {   // decreasing row_ptr
        std::vector<int32_t> rp = {0, 2, 1, 3}, ci = {0, 0, 1};
        CHECK(bf1_route_depth(rp.data(), ci.data(), 3, &d) == BF1_ERR_INVALID_ARG);
    }
    {   // an entry after its own row (not causal)
        std::vector<int32_t> rp = {0, 1, 3}, ci = {0, 0, 2};
        CHECK(bf1_route_depth(rp.data(), ci.data(), 2, &d) == BF1_ERR_INVALID_ARG);
    }
    {   // a negative entry
        std::vector<int32_t> rp = {0, 1, 3}, ci = {0, -1, 1};
        CHECK(bf1_route_depth(rp.data(), ci.data(), 2, &d) == BF1_ERR_INVALID_ARG);
    }
    {   // entries but no col_idx
        std::vector<int32_t> rp = {0, 1};
        CHECK(bf1_route_depth(rp.data(), nullptr, 1, &d) == BF1_ERR_INVALID_ARG);
    }
    {   // too many blocks, negative count, missing output
        std::vector<int32_t> rp(16386, 0);
        CHECK(bf1_route_depth(rp.data(), nullptr, 16385, &d) == BF1_ERR_INVALID_ARG);
        CHECK(bf1_route_depth(rp.data(), nullptr, -1, &d) == BF1_ERR_INVALID_ARG);
        CHECK(bf1_route_depth(rp.data(), nullptr, 3, nullptr) == BF1_ERR_INVALID_ARG);
    }
    {   // an unreachable later block gives -1, not an error
        std::vector<int32_t> rp = {0, 1, 2}, ci = {0, 1};
        CHECK(bf1_route_depth(rp.data(), ci.data(), 2, &d) == BF1_OK);
        CHECK(d == -1);
    }
}

static void sizes() {
    int64_t bytes = 0;
    const int cfgs[][7] = {{1, 32768, 16, 8, 128, 64, 2}, {2, 30001, 16, 8, 128, 64, 2},
                           {1, 512, 2, 1, 64, 64, 1},     {2, 1300, 8, 2, 128, 128, 2}};
    for (const auto& c : cfgs) {
        CHECK(bf1_attn_bwd_workspace_size(c[0], c[1], c[2], c[3], c[4], c[5], c[6], &bytes) == BF1_OK);
        std::printf("bwd_ws %d %d %d %d %d %d %d %lld\n", c[0], c[1], c[2], c[3], c[4], c[5], c[6],
                    (long long)bytes);
    }
    int32_t stride = 0;
    CHECK(bf1_decode_plan_stride(65536, 64, 2, 0, &stride) == BF1_OK);
    CHECK(bf1_decode_workspace_size(32, 16, 8, 128, stride, &bytes) == BF1_OK);
    std::printf("decode %d %lld\n", stride, (long long)bytes);
    CHECK(bf1_decode_plan_stride(0, 64, 2, 0, &stride) == BF1_ERR_INVALID_ARG);
    CHECK(bf1_decode_workspace_size(1, 3, 2, 128, stride, &bytes) == BF1_ERR_INVALID_ARG);
}

// A dummy, suitably aligned address: the shim never dereferences caller
// pointers and the stubs do not either.
static void* const P = reinterpret_cast<void*>(uintptr_t(1) << 16);
static float* const PF = reinterpret_cast<float*>(uintptr_t(1) << 16);

static void runtime_errors_map_to_bf1_err_hip() {
    g_stub = StubState{};
    g_stub.fail = true;
    int32_t* ip = reinterpret_cast<int32_t*>(P);
    CHECK(bf1_plan(4096, 64, 2, ip, ip, 1 << 20, nullptr) == BF1_ERR_HIP);
    CHECK(bf1_attn_fwd(P, P, P, P, PF, 1, 4096, 16, 8, 128, 64, 2, nullptr) == BF1_ERR_HIP);
    CHECK(bf1_attn_fwd_noalloc(P, P, P, P, PF, 1, 4096, 16, 8, 128, 64, 2, nullptr) == BF1_ERR_HIP);
    CHECK(bf1_attn_fwd_csr(P, P, P, P, PF, 1, 4096, 16, 8, 128, 64, ip, ip, 442, nullptr) == BF1_ERR_HIP);
    CHECK(bf1_dense_causal_fwd(P, P, P, P, PF, 1, 4096, 16, 8, 128, nullptr) == BF1_ERR_HIP);
    CHECK(bf1_attn_bwd(P, P, P, P, P, PF, PF, PF, PF, 1, 4096, 16, 8, 128, 64, 2, P, int64_t(1) << 40,
                       nullptr) == BF1_ERR_HIP);
    CHECK(bf1_decode_plan(1, ip, ip, 8, 8, 64, 2, 0, ip, 16, nullptr) == BF1_ERR_HIP);
    CHECK(bf1_decode_attn(P, P, P, ip, 8, ip, 16, P, PF, 1, 16, 8, 128, 64, P, int64_t(1) << 30,
                          nullptr) == BF1_ERR_HIP);
    CHECK(g_stub.mallocs == 0);
    // argument errors still win over runtime errors: nothing is called
    CHECK(bf1_attn_fwd(nullptr, P, P, P, PF, 1, 4096, 16, 8, 128, 64, 2, nullptr) == BF1_ERR_INVALID_ARG);
    g_stub.fail = false;
}

static void plan_cache_and_capture() {
    g_stub = StubState{};
    CHECK(bf1_attn_fwd(P, P, P, P, PF, 1, 4096, 16, 8, 128, 64, 2, nullptr) == BF1_OK);
    CHECK(g_stub.plans == 1 && g_stub.attns == 1 && g_stub.last_nnz == 442);
    CHECK(bf1_attn_fwd(P, P, P, P, PF, 1, 4096, 16, 8, 128, 64, 2, nullptr) == BF1_OK);
    CHECK(g_stub.plans == 1 && g_stub.attns == 2);   // cached
    // under capture: an existing plan is used, a new one is refused untouched
    g_stub.capturing = true;
    const long m0 = g_stub.mallocs;
    CHECK(bf1_attn_fwd(P, P, P, P, PF, 1, 4096, 16, 8, 128, 64, 2, nullptr) == BF1_OK);
    CHECK(bf1_attn_fwd(P, P, P, P, PF, 1, 8192, 16, 8, 128, 64, 2, nullptr) == BF1_ERR_CAPTURE);
    CHECK(bf1_attn_bwd(P, P, P, P, P, PF, PF, PF, PF, 1, 4096, 16, 8, 128, 64, 2, P, int64_t(1) << 40,
                       nullptr) == BF1_ERR_CAPTURE);   // its transposed plan is new
    CHECK(g_stub.mallocs == m0 && g_stub.attns == 3 && g_stub.bwds == 0);
    g_stub.capturing = false;
    // backward: host-built descriptors uploaded through the (stub) allocator
    int64_t need = 0;
    CHECK(bf1_attn_bwd_workspace_size(1, 4096, 16, 8, 128, 64, 2, &need) == BF1_OK);
    CHECK(bf1_attn_bwd(P, P, P, P, P, PF, PF, PF, PF, 1, 4096, 16, 8, 128, 64, 2, P, need - 1, nullptr) ==
          BF1_ERR_BUFFER_TOO_SMALL);
    CHECK(bf1_attn_bwd(P, P, P, P, P, PF, PF, PF, PF, 1, 4096, 16, 8, 128, 64, 2, P, need, nullptr) == BF1_OK);
    CHECK(bf1_attn_bwd(P, P, P, P, P, PF, PF, PF, PF, 1, 30001, 16, 8, 128, 64, 2, P, int64_t(1) << 40,
                       nullptr) == BF1_OK);
    CHECK(g_stub.bwds == 2);
    // the forward that allocates nothing: no allocation, and an oversized
    // table is refused before any call
    const long m1 = g_stub.mallocs;
    CHECK(bf1_attn_fwd_noalloc(P, P, P, P, PF, 2, 30001, 16, 8, 128, 64, 2, nullptr) == BF1_OK);
    CHECK(bf1_attn_fwd_noalloc(P, P, P, P, PF, 1, int64_t(1) << 23, 2, 1, 128, 64, 2, nullptr) ==
          BF1_ERR_BUFFER_TOO_SMALL);
    CHECK(g_stub.mallocs == m1);
    bf1_release_plans();
    CHECK(g_stub.mallocs == g_stub.frees);
    std::printf("allocations %ld frees %ld\n", g_stub.mallocs, g_stub.frees);
}

int main() {
    const long cases[][3] = {{0, 64, 2}, {1, 64, 2}, {257, 64, 2}, {512, 64, 1}, {4096, 64, 2},
                             {30001, 64, 2}, {1500, 128, 2}, {777, 5, 0}, {20000, 16, 3}, {700, 64, 9}};
    for (const auto& c : cases) host_tables(c[0], (int)c[1], (int)c[2]);
    malformed_depth_tables();
    sizes();
    runtime_errors_map_to_bf1_err_hip();
    plan_cache_and_capture();
    std::printf(g_failures == 0 ? "ALL OK\n" : "FAILURES %d\n", g_failures);
    return g_failures == 0 ? 0 : 1;
}
