// C-ABI shim of libbf1.so: argument validation, the plan cache, stream
// handling and the mapping of HIP errors to status codes.  Every argument
// check happens before any HIP call, so invalid calls touch no device.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "../../include/bf1.h"
#include "bf1_kernels.h"
#include "bf1_route.h"

namespace {

constexpr int kVersion = 10200;  // 1.2.0

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Route sizes; false if the table would not fit int32 indices.
bool route_sizes(int64_t n, int64_t B, int64_t L, int64_t* NB, int64_t* nnz) {
    *NB = (n + B - 1) / B;
    if (*NB >= 0x7fffffff) return false;
    *nnz = bf1::route_row_start(*NB, L);
    return *nnz >= 0 && *nnz < 0x7fffffff;
}

// ---- plan cache: (device, n, B, L) -> device CSR --------------------------
// A plan is complete before it enters the cache (built on a private stream
// that the host waits for), so later calls use it with no stream ordering at
// all -- which also makes them safe to capture into a HIP graph.  Building a
// plan is refused while the caller's stream is being captured.
struct Plan {
    int32_t* row_ptr = nullptr;
    int32_t* col_idx = nullptr;
    int64_t nnz = 0;
};

std::mutex g_mu;
std::map<std::tuple<int, int64_t, int32_t, int32_t>, Plan> g_plans;
std::map<int, hipStream_t> g_plan_streams;  // per device, created on first use

int status_of(hipError_t e) { return e == hipSuccess ? BF1_OK : BF1_ERR_HIP; }

// Forward key split (bf1_set_forward_key_split): 0 automatic, 1 never, 2 always.
std::atomic<int> g_key_split{0};

// True (and BF1_OK) if `s` is being captured into a graph.
int capturing(hipStream_t s, bool* yes) {
    hipStreamCaptureStatus st = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &st) != hipSuccess) return BF1_ERR_HIP;
    *yes = st != hipStreamCaptureStatusNone;
    return BF1_OK;
}

// Validation shared by the attention entry points.
int check_attn(const void* Q, const void* K, const void* V, void* O, float* LSE, int32_t batch,
               int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim) {
    if (batch < 0 || n < 0 || Hq < 1 || Hkv < 1) return BF1_ERR_INVALID_ARG;
    if (Hq % Hkv != 0) return BF1_ERR_INVALID_ARG;
    if (n > 0x7fffffffLL - 256) return BF1_ERR_INVALID_ARG;
    // one head's K or V rows are addressed through a 32-bit buffer range
    if (n >= (int64_t(1) << 24)) return BF1_ERR_UNSUPPORTED;
    const int32_t G = Hq / Hkv;
    if (head_dim != 64 && head_dim != 128) return BF1_ERR_UNSUPPORTED;
    if (G != 1 && G != 2 && G != 4 && G != 8) return BF1_ERR_UNSUPPORTED;
    if (batch == 0 || n == 0) return BF1_OK;
    if (!Q || !K || !V || !O) return BF1_ERR_INVALID_ARG;
    if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16))
        return BF1_ERR_INVALID_ARG;
    if (LSE && !aligned(LSE, 4)) return BF1_ERR_INVALID_ARG;
    // element counts must fit comfortably in int64 byte offsets
    const double elems = (double)batch * (double)Hq * (double)n * (double)head_dim;
    if (elems > 4.0e18) return BF1_ERR_INVALID_ARG;
    return BF1_OK;
}

// ---- decode ----------------------------------------------------------------
// Earlier selected pages any token of a sequence of at most max_seq_len
// tokens can need: the largest c(j) over j < NB, which is c(NB - 1) because
// c never decreases (j <= L: c = j; beyond, the locals stay L, the dyadic
// count only grows, and where block 0 stops being a separate entry (j a power
// of two) the dyadic count has just grown by one), or NB - 1 if dense.
bool decode_cap(int64_t max_seq_len, int64_t B, int64_t L, bool dense, int64_t* cap) {
    const int64_t NB = (max_seq_len + B - 1) / B;
    if (NB < 1 || NB >= 0x7fffffff) return false;
    *cap = dense ? NB - 1 : bf1::route_pred_count(NB - 1, L);
    return true;
}

// Splits per (sequence, kv-head) and pages per split for lists of up to P
// pages: about 1024 workgroups (four per CU; more or fewer measured no
// faster for the selected lists and slower for long dense ones), at most 256
// splits, splits as even as possible.
void decode_splits(int64_t batch, int64_t Hkv, int64_t P, int32_t* nsplit, int32_t* ppw) {
    const int64_t units = std::max<int64_t>(1, batch * Hkv);
    const int64_t want = std::max<int64_t>(1, (1024 + units - 1) / units);
    int64_t ns = std::min<int64_t>(std::min<int64_t>(P, want), 256);
    ns = std::max<int64_t>(ns, 1);
    const int64_t pp = (P + ns - 1) / ns;
    *nsplit = (int32_t)((P + pp - 1) / pp);
    *ppw = (int32_t)pp;
}

int64_t decode_ws_bytes(int64_t batch, int64_t Hq, int64_t Hkv, int64_t D, int64_t nsplit) {
    const int64_t G = Hq / Hkv;
    const int64_t b = batch * Hkv * nsplit * G * (D + 2) * 4;
    return (b + 255) / 256 * 256;
}

int run_attn(bf1::AttnArgs a, hipStream_t s) {
    a.key_split = g_key_split.load(std::memory_order_relaxed);
    return status_of(bf1::launch_attention(a, s));
}

// Cached forward route of (current device, n, B, L), built by the planner
// kernel on first use and complete on return.  `s` is the caller's stream
// (only checked for capture).
int get_plan(int64_t n, int32_t B, int32_t L, hipStream_t s, Plan* out) {
    int64_t NB, nnz;
    if (!route_sizes(n, B, L, &NB, &nnz)) return BF1_ERR_INVALID_ARG;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return BF1_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_mu);
    auto key = std::make_tuple(dev, n, B, L);
    auto it = g_plans.find(key);
    if (it != g_plans.end()) {
        *out = it->second;
        return BF1_OK;
    }
    bool cap = false;
    int st = capturing(s, &cap);
    if (st != BF1_OK) return st;
    if (cap) return BF1_ERR_CAPTURE;
    hipStream_t ps = nullptr;
    auto ps_it = g_plan_streams.find(dev);
    if (ps_it == g_plan_streams.end()) {
        if (hipStreamCreateWithFlags(&ps, hipStreamNonBlocking) != hipSuccess) return BF1_ERR_HIP;
        g_plan_streams.emplace(dev, ps);
    } else {
        ps = ps_it->second;
    }
    Plan p;
    p.nnz = nnz;
    if (hipMalloc((void**)&p.row_ptr, sizeof(int32_t) * (NB + 1)) != hipSuccess) return BF1_ERR_NOMEM;
    if (hipMalloc((void**)&p.col_idx, sizeof(int32_t) * (nnz > 0 ? nnz : 1)) != hipSuccess) {
        (void)hipFree(p.row_ptr);
        return BF1_ERR_NOMEM;
    }
    hipError_t e = bf1::launch_plan((int32_t)NB, L, p.row_ptr, p.col_idx, ps);
    if (e == hipSuccess) e = hipStreamSynchronize(ps);
    if (e != hipSuccess) {
        (void)hipFree(p.row_ptr);
        (void)hipFree(p.col_idx);
        return BF1_ERR_HIP;
    }
    g_plans.emplace(key, p);
    *out = p;
    return BF1_OK;
}

// ---- backward plan: transposed route cut into segments ---------------------
// Every 64-key tile (key block i, sub-tile u, starting before n) gets the list
// of query blocks that select block i; lists longer than SEG_MAX entries are
// cut into segments whose partial dK/dV go to numbered workspace slots and are
// summed by the reduce kernel.  Segments are ordered longest first.
constexpr int64_t SEG_MAX = 16;

struct BwdLayout {
    std::vector<int32_t> users, uoffs, segs, reds;
    int32_t nslots = 0;
    int64_t nusers = 0;
};

bool bwd_layout(int64_t n, int32_t B, int32_t L, BwdLayout* lay, bool fill) {
    const int64_t NB = (n + B - 1) / B;
    const int nsub = B / 64;
    std::vector<int32_t> tmp;
    std::vector<std::array<int32_t, 8>> segs;
    int64_t nslots = 0, total = 0;
    for (int64_t i = 0; i < NB; ++i) {
        const int64_t cnt = bf1::route_users(NB, L, i, nullptr);
        const int64_t off = total;
        if (fill) lay->uoffs.push_back((int32_t)off);
        if (fill) {
            tmp.resize(cnt);
            bf1::route_users(NB, L, i, tmp.data());
            lay->users.insert(lay->users.end(), tmp.begin(), tmp.end());
        }
        total += cnt;
        const int64_t nch = (cnt + SEG_MAX - 1) / SEG_MAX;
        for (int u = 0; u < nsub; ++u) {
            if (i * B + u * 64 >= n) break;
            const int64_t slot0 = nch > 1 ? nslots : -1;
            for (int64_t c = 0; c < nch; ++c) {
                const int64_t m = std::min(SEG_MAX, cnt - SEG_MAX * c);
                if (fill)
                    segs.push_back({(int32_t)i, u, (int32_t)(off + SEG_MAX * c), (int32_t)m,
                                    (int32_t)(nch > 1 ? slot0 + c : -1), 0, 0, 0});
            }
            if (nch > 1) {
                if (fill) lay->reds.insert(lay->reds.end(), {(int32_t)i, u, (int32_t)slot0, (int32_t)nch});
                nslots += nch;
            }
            if (nslots > 0x3fffffff || total > 0x3fffffff) return false;
        }
    }
    if (fill) {
        lay->uoffs.push_back((int32_t)total);
        std::stable_sort(segs.begin(), segs.end(),
                         [](const std::array<int32_t, 8>& a, const std::array<int32_t, 8>& b) {
                             return a[3] > b[3];
                         });
        for (auto& sg : segs) lay->segs.insert(lay->segs.end(), sg.begin(), sg.end());
    }
    lay->nslots = (int32_t)nslots;
    lay->nusers = total;
    return true;
}

struct BwdPlan {
    int32_t* users = nullptr;
    int32_t* uoffs = nullptr;
    int64_t nusers = 0;
    int32_t* segs = nullptr;
    int32_t* reds = nullptr;
    int32_t nseg = 0, nred = 0, nslots = 0;
};
std::map<std::tuple<int, int64_t, int32_t, int32_t>, BwdPlan> g_bwd_plans;

int bwd_workspace_bytes(int32_t batch, int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim, int32_t B,
                        int32_t L, int64_t* bytes) {
    BwdLayout lay;
    if (!bwd_layout(n, B, L, &lay, false)) return BF1_ERR_INVALID_ARG;
    const int64_t delta = ((int64_t)batch * Hq * n * 4 + 255) / 256 * 256;
    const int64_t part = (int64_t)batch * Hkv * lay.nslots * 2 * 64 * head_dim * 4;
    const int64_t nsub = B / 64;
    const int64_t ds = (int64_t)batch * Hq * lay.nusers * nsub * nsub * 64 * 64 * 2;
    *bytes = 2 * delta + part + ds;  // D, LSE * log2 e, partial tiles, dS units
    return BF1_OK;
}

int get_bwd_plan(int64_t n, int32_t B, int32_t L, hipStream_t s, BwdPlan* out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return BF1_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_mu);
    auto key = std::make_tuple(dev, n, B, L);
    auto it = g_bwd_plans.find(key);
    if (it == g_bwd_plans.end()) {
        bool cap = false;
        int st = capturing(s, &cap);
        if (st != BF1_OK) return st;
        if (cap) return BF1_ERR_CAPTURE;
        BwdLayout lay;
        if (!bwd_layout(n, B, L, &lay, true)) return BF1_ERR_INVALID_ARG;
        BwdPlan p;
        p.nseg = (int32_t)(lay.segs.size() / 8);
        p.nred = (int32_t)(lay.reds.size() / 4);
        p.nslots = lay.nslots;
        p.nusers = lay.nusers;
        auto up = [](const std::vector<int32_t>& v, int32_t** d) -> bool {
            const size_t bytes = sizeof(int32_t) * (v.empty() ? 1 : v.size());
            if (hipMalloc((void**)d, bytes) != hipSuccess) return false;
            if (!v.empty() && hipMemcpy(*d, v.data(), sizeof(int32_t) * v.size(),
                                        hipMemcpyHostToDevice) != hipSuccess)
                return false;
            return true;
        };
        if (!up(lay.users, &p.users) || !up(lay.uoffs, &p.uoffs) || !up(lay.segs, &p.segs) ||
            !up(lay.reds, &p.reds)) {
            (void)hipFree(p.users);
            (void)hipFree(p.uoffs);
            (void)hipFree(p.segs);
            (void)hipFree(p.reds);
            return BF1_ERR_NOMEM;
        }
        it = g_bwd_plans.emplace(key, p).first;
    }
    *out = it->second;
    return BF1_OK;
}

}  // namespace

extern "C" {

int bf1_version(void) { return kVersion; }

const char* bf1_status_string(int status) {
    switch (status) {
        case BF1_OK: return "BF1_OK";
        case BF1_ERR_INVALID_ARG: return "BF1_ERR_INVALID_ARG: invalid argument";
        case BF1_ERR_UNSUPPORTED: return "BF1_ERR_UNSUPPORTED: configuration not supported";
        case BF1_ERR_BUFFER_TOO_SMALL: return "BF1_ERR_BUFFER_TOO_SMALL: route table capacity too small";
        case BF1_ERR_HIP: return "BF1_ERR_HIP: HIP runtime or launch error";
        case BF1_ERR_NOMEM: return "BF1_ERR_NOMEM: device allocation failed";
        case BF1_ERR_CAPTURE:
            return "BF1_ERR_CAPTURE: the route plan is not built yet and cannot be built while the "
                   "stream is being captured (call once outside capture first)";
        default: return "BF1: unknown status";
    }
}

int bf1_plan_size(int64_t n, int32_t B, int32_t L, int32_t* num_blocks, int64_t* nnz,
                  int64_t* pairs) {
    if (n < 0 || B < 1 || L < 0) return BF1_ERR_INVALID_ARG;
    int64_t NB, z;
    if (!route_sizes(n, B, L, &NB, &z)) return BF1_ERR_INVALID_ARG;
    if (num_blocks) *num_blocks = (int32_t)NB;
    if (nnz) *nnz = z;
    if (pairs) *pairs = bf1::route_selected_pairs(n, B, L);
    return BF1_OK;
}

int bf1_plan(int64_t n, int32_t B, int32_t L, int32_t* row_ptr, int32_t* col_idx,
             int64_t col_capacity, void* stream) {
    if (n < 0 || B < 1 || L < 0 || col_capacity < 0) return BF1_ERR_INVALID_ARG;
    int64_t NB, nnz;
    if (!route_sizes(n, B, L, &NB, &nnz)) return BF1_ERR_INVALID_ARG;
    if (!row_ptr) return BF1_ERR_INVALID_ARG;
    if (nnz > 0 && !col_idx) return BF1_ERR_INVALID_ARG;
    if (!aligned(row_ptr, 4) || (col_idx && !aligned(col_idx, 4))) return BF1_ERR_INVALID_ARG;
    if (col_capacity < nnz) return BF1_ERR_BUFFER_TOO_SMALL;
    return status_of(bf1::launch_plan((int32_t)NB, L, row_ptr, col_idx, (hipStream_t)stream));
}

int bf1_attn_fwd(const void* Q, const void* K, const void* V, void* O, float* LSE, int32_t batch,
                 int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim, int32_t B, int32_t L,
                 void* stream) {
    int st = check_attn(Q, K, V, O, LSE, batch, n, Hq, Hkv, head_dim);
    if (st != BF1_OK) return st;
    if (L < 0) return BF1_ERR_INVALID_ARG;
    if (B != 64 && B != 128) return BF1_ERR_UNSUPPORTED;
    if (batch == 0 || n == 0) return BF1_OK;
    hipStream_t s = (hipStream_t)stream;
    Plan plan;
    st = get_plan(n, B, L, s, &plan);
    if (st != BF1_OK) return st;
    bf1::AttnArgs a{Q, K, V, O, LSE, plan.row_ptr, plan.col_idx, plan.nnz,
                    batch, n, Hq, Hkv, head_dim, B, false};
    return run_attn(a, s);
}

int bf1_attn_fwd_noalloc(const void* Q, const void* K, const void* V, void* O, float* LSE,
                         int32_t batch, int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim,
                         int32_t B, int32_t L, void* stream) {
    int st = check_attn(Q, K, V, O, LSE, batch, n, Hq, Hkv, head_dim);
    if (st != BF1_OK) return st;
    if (L < 0) return BF1_ERR_INVALID_ARG;
    if (B != 64 && B != 128) return BF1_ERR_UNSUPPORTED;
    if (batch == 0 || n == 0) return BF1_OK;
    int64_t NB, nnz;
    if (!route_sizes(n, B, L, &NB, &nnz)) return BF1_ERR_INVALID_ARG;
    if (NB + 1 + nnz > bf1::kNoallocInts) return BF1_ERR_BUFFER_TOO_SMALL;
    int32_t* table = nullptr;
    if (bf1::noalloc_scratch(&table) != hipSuccess) return BF1_ERR_HIP;
    int32_t* row_ptr = table;
    int32_t* col_idx = table + (NB + 1);
    hipStream_t s = (hipStream_t)stream;
    // The planner rewrites every entry the attention kernel reads, so nothing
    // left in the scratch by an earlier call matters.
    if (bf1::launch_plan((int32_t)NB, L, row_ptr, col_idx, s) != hipSuccess) return BF1_ERR_HIP;
    bf1::AttnArgs a{Q, K, V, O, LSE, row_ptr, col_idx, nnz, batch, n, Hq, Hkv, head_dim, B, false};
    return run_attn(a, s);
}

int bf1_attn_fwd_csr(const void* Q, const void* K, const void* V, void* O, float* LSE,
                     int32_t batch, int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim,
                     int32_t B, const int32_t* row_ptr, const int32_t* col_idx, int64_t nnz,
                     void* stream) {
    int st = check_attn(Q, K, V, O, LSE, batch, n, Hq, Hkv, head_dim);
    if (st != BF1_OK) return st;
    if (B != 64 && B != 128) return BF1_ERR_UNSUPPORTED;
    if (nnz < 0 || nnz >= 0x7fffffff) return BF1_ERR_INVALID_ARG;
    if (batch == 0 || n == 0) return BF1_OK;
    if (!row_ptr || (nnz > 0 && !col_idx)) return BF1_ERR_INVALID_ARG;
    if (!aligned(row_ptr, 4) || (col_idx && !aligned(col_idx, 4))) return BF1_ERR_INVALID_ARG;
    bf1::AttnArgs a{Q, K, V, O, LSE, row_ptr, col_idx, nnz, batch, n, Hq, Hkv, head_dim, B, false};
    return run_attn(a, (hipStream_t)stream);
}

int bf1_dense_causal_fwd(const void* Q, const void* K, const void* V, void* O, float* LSE,
                         int32_t batch, int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim,
                         void* stream) {
    int st = check_attn(Q, K, V, O, LSE, batch, n, Hq, Hkv, head_dim);
    if (st != BF1_OK) return st;
    if (batch == 0 || n == 0) return BF1_OK;
    bf1::AttnArgs a{Q, K, V, O, LSE, nullptr, nullptr, 0, batch, n, Hq, Hkv, head_dim, 64, true};
    return run_attn(a, (hipStream_t)stream);
}

int bf1_plan_transposed(int64_t n, int32_t B, int32_t L, int32_t* row_ptr, int32_t* col_idx,
                        int64_t col_capacity) {
    if (n < 0 || B < 1 || L < 0 || col_capacity < 0 || !row_ptr) return BF1_ERR_INVALID_ARG;
    int64_t NB, nnz;
    if (!route_sizes(n, B, L, &NB, &nnz)) return BF1_ERR_INVALID_ARG;
    if (nnz > 0 && !col_idx) return BF1_ERR_INVALID_ARG;
    if (col_capacity < nnz) return BF1_ERR_BUFFER_TOO_SMALL;
    int64_t e = 0;
    for (int64_t i = 0; i < NB; ++i) {
        row_ptr[i] = (int32_t)e;
        e += bf1::route_users(NB, L, i, col_idx ? col_idx + e : nullptr);
    }
    row_ptr[NB] = (int32_t)e;
    return e == nnz ? BF1_OK : BF1_ERR_INVALID_ARG;
}

int bf1_plan_variant(int32_t kind, int64_t n, int32_t B, int32_t L, uint64_t seed, int32_t* row_ptr,
                     int32_t* col_idx, int64_t col_capacity) {
    if (kind != BF1_ROUTE_BF1 && kind != BF1_ROUTE_SLIDING && kind != BF1_ROUTE_STATIC_RANDOM)
        return BF1_ERR_INVALID_ARG;
    if (n < 0 || B < 1 || L < 0 || col_capacity < 0 || !row_ptr) return BF1_ERR_INVALID_ARG;
    int64_t NB, nnz;
    if (!route_sizes(n, B, L, &NB, &nnz)) return BF1_ERR_INVALID_ARG;
    if (nnz > 0 && !col_idx) return BF1_ERR_INVALID_ARG;
    if (col_capacity < nnz) return BF1_ERR_BUFFER_TOO_SMALL;
    int64_t e = 0;
    for (int64_t j = 0; j < NB; ++j) {
        row_ptr[j] = (int32_t)e;
        if (kind == BF1_ROUTE_BF1) {
            // Eq. 1, ascending: block 0, dyadics from the farthest, locals, self
            const int64_t start = e;
            if (j > L) col_idx[e++] = 0;
            int r = 2;
            while (r < 62 && (int64_t(1) << (r + 1)) <= j) ++r;
            for (; r >= 2; --r) {
                const int64_t off = int64_t(1) << r;
                if (off <= j && off > L && j - off > 0) col_idx[e++] = (int32_t)(j - off);
            }
            for (int64_t t = (j - L > 0 ? j - L : 0); t <= j; ++t) col_idx[e++] = (int32_t)t;
            if (e - start != 1 + bf1::route_pred_count(j, L)) return BF1_ERR_INVALID_ARG;
        } else if (kind == BF1_ROUTE_SLIDING) {
            e += bf1::route_sliding_row(j, L, col_idx + e);
        } else {
            e += bf1::route_static_random_row(j, L, seed, col_idx + e);
        }
    }
    row_ptr[NB] = (int32_t)e;
    return e == nnz ? BF1_OK : BF1_ERR_INVALID_ARG;
}

int bf1_route_depth(const int32_t* row_ptr, const int32_t* col_idx, int32_t num_blocks,
                    int32_t* max_depth) {
    if (num_blocks < 0 || num_blocks > 16384 || !row_ptr || !max_depth) return BF1_ERR_INVALID_ARG;
    const int32_t NB = num_blocks;
    if (row_ptr[0] != 0) return BF1_ERR_INVALID_ARG;
    for (int32_t j = 0; j < NB; ++j)
        if (row_ptr[j + 1] < row_ptr[j]) return BF1_ERR_INVALID_ARG;
    if (row_ptr[NB] > 0 && !col_idx) return BF1_ERR_INVALID_ARG;
    // successor lists: edge i -> j for every earlier block i in row j
    std::vector<int32_t> deg(NB + 1, 0);
    for (int32_t j = 0; j < NB; ++j)
        for (int32_t e = row_ptr[j]; e < row_ptr[j + 1]; ++e) {
            const int32_t i = col_idx[e];
            if (i < 0 || i > j) return BF1_ERR_INVALID_ARG;
            if (i < j) ++deg[i + 1];
        }
    for (int32_t i = 0; i < NB; ++i) deg[i + 1] += deg[i];
    std::vector<int32_t> succ(deg[NB]), fill(deg.begin(), deg.end() - 1);
    for (int32_t j = 0; j < NB; ++j)
        for (int32_t e = row_ptr[j]; e < row_ptr[j + 1]; ++e)
            if (col_idx[e] < j) succ[fill[col_idx[e]]++] = j;
    // breadth-first search from every source; edges only go forward, so a
    // source's search touches blocks src..NB-1 only
    std::vector<int32_t> dist(NB), queue(NB);
    int32_t worst = 0;
    for (int32_t src = 0; src < NB; ++src) {
        std::fill(dist.begin() + src, dist.end(), -1);
        dist[src] = 0;
        int32_t head = 0, tail = 0;
        queue[tail++] = src;
        while (head < tail) {
            const int32_t u = queue[head++];
            for (int32_t e = deg[u]; e < deg[u + 1]; ++e) {
                const int32_t w = succ[e];
                if (dist[w] < 0) {
                    dist[w] = dist[u] + 1;
                    queue[tail++] = w;
                }
            }
        }
        if (tail != NB - src) {
            *max_depth = -1;
            return BF1_OK;
        }
        worst = std::max(worst, dist[queue[tail - 1]]);
    }
    *max_depth = worst;
    return BF1_OK;
}

int bf1_attn_bwd_workspace_size(int32_t batch, int64_t n, int32_t Hq, int32_t Hkv,
                                int32_t head_dim, int32_t B, int32_t L, int64_t* bytes) {
    if (!bytes) return BF1_ERR_INVALID_ARG;
    int st = check_attn(nullptr, nullptr, nullptr, nullptr, nullptr, 0, n, Hq, Hkv, head_dim);
    if (st != BF1_OK) return st;
    if (batch < 0 || L < 0) return BF1_ERR_INVALID_ARG;
    if ((B != 64 && B != 128) || (Hq / Hkv) * B < 128) return BF1_ERR_UNSUPPORTED;
    return bwd_workspace_bytes(batch, n, Hq, Hkv, head_dim, B, L, bytes);
}

int bf1_attn_bwd(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const float* LSE, float* dQ, float* dK, float* dV, int32_t batch, int64_t n,
                 int32_t Hq, int32_t Hkv, int32_t head_dim, int32_t B, int32_t L, void* workspace,
                 int64_t workspace_bytes, void* stream) {
    int st = check_attn(Q, K, V, const_cast<void*>(O), nullptr, batch, n, Hq, Hkv, head_dim);
    if (st != BF1_OK) return st;
    if (L < 0 || workspace_bytes < 0) return BF1_ERR_INVALID_ARG;
    if ((B != 64 && B != 128) || (Hq / Hkv) * B < 128) return BF1_ERR_UNSUPPORTED;
    if (batch == 0 || n == 0) return BF1_OK;
    if (!dO || !LSE || !dQ || !dK || !dV || !workspace) return BF1_ERR_INVALID_ARG;
    if (!aligned(dO, 16) || !aligned(dQ, 16) || !aligned(dK, 16) || !aligned(dV, 16) ||
        !aligned(LSE, 4) || !aligned(workspace, 256))
        return BF1_ERR_INVALID_ARG;
    int64_t need = 0;
    st = bwd_workspace_bytes(batch, n, Hq, Hkv, head_dim, B, L, &need);
    if (st != BF1_OK) return st;
    if (workspace_bytes < need) return BF1_ERR_BUFFER_TOO_SMALL;
    hipStream_t s = (hipStream_t)stream;
    Plan plan;
    st = get_plan(n, B, L, s, &plan);
    if (st != BF1_OK) return st;
    BwdPlan bp;
    st = get_bwd_plan(n, B, L, s, &bp);
    if (st != BF1_OK) return st;
    const int64_t delta_bytes = ((int64_t)batch * Hq * n * 4 + 255) / 256 * 256;
    float* delta = (float*)workspace;
    float* lse2 = (float*)((char*)workspace + delta_bytes);
    float* part = (float*)((char*)workspace + 2 * delta_bytes);
    void* ds = (char*)workspace + 2 * delta_bytes +
               (int64_t)batch * Hkv * bp.nslots * 2 * 64 * head_dim * 4;
    bf1::BwdArgs a{Q, K, V, O, dO, LSE, dQ, dK, dV, delta, lse2, part, ds,
                   plan.row_ptr, plan.col_idx, plan.nnz, bp.users, bp.uoffs, bp.nusers, bp.segs, bp.nseg,
                   bp.reds, bp.nred, bp.nslots, batch, n, Hq, Hkv, B, head_dim, L};
    return status_of(bf1::launch_backward(a, s));
}

int bf1_set_forward_key_split(int32_t mode) {
    if (mode < 0 || mode > 2) return BF1_ERR_INVALID_ARG;
    g_key_split.store(mode, std::memory_order_relaxed);
    return BF1_OK;
}

void bf1_release_plans(void) {
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_plans.empty() || !g_bwd_plans.empty()) (void)hipDeviceSynchronize();
    for (auto& kv : g_plans) {
        (void)hipFree(kv.second.row_ptr);
        (void)hipFree(kv.second.col_idx);
    }
    g_plans.clear();
    for (auto& kv : g_bwd_plans) {
        (void)hipFree(kv.second.users);
        (void)hipFree(kv.second.uoffs);
        (void)hipFree(kv.second.segs);
        (void)hipFree(kv.second.reds);
    }
    g_bwd_plans.clear();
}

int bf1_decode_plan_stride(int64_t max_seq_len, int32_t B, int32_t L, int32_t dense, int32_t* stride) {
    if (!stride || max_seq_len < 1 || L < 0 || L > 32 || (dense != 0 && dense != 1))
        return BF1_ERR_INVALID_ARG;
    if (B != 64 && B != 128) return BF1_ERR_UNSUPPORTED;
    if (max_seq_len >= (int64_t(1) << 31)) return BF1_ERR_INVALID_ARG;
    int64_t cap;
    if (!decode_cap(max_seq_len, B, L, dense != 0, &cap)) return BF1_ERR_INVALID_ARG;
    *stride = (int32_t)(3 + cap);
    return BF1_OK;
}

int bf1_decode_plan(int32_t batch, const int32_t* seq_lens, const int32_t* page_table,
                    int32_t max_pages_per_seq, int32_t num_pages, int32_t B, int32_t L, int32_t dense,
                    int32_t* plan, int32_t plan_stride, void* stream) {
    if (batch < 0 || L < 0 || L > 32 || (dense != 0 && dense != 1)) return BF1_ERR_INVALID_ARG;
    if (B != 64 && B != 128) return BF1_ERR_UNSUPPORTED;
    if (max_pages_per_seq < 1 || num_pages < 1 || plan_stride < 3) return BF1_ERR_INVALID_ARG;
    if (batch == 0) return BF1_OK;
    if (!seq_lens || !page_table || !plan) return BF1_ERR_INVALID_ARG;
    if (!aligned(seq_lens, 4) || !aligned(page_table, 4) || !aligned(plan, 4)) return BF1_ERR_INVALID_ARG;
    bf1::DecodePlanArgs a{batch, seq_lens, page_table, max_pages_per_seq, num_pages, B, L, dense,
                          plan, plan_stride, plan_stride - 3};
    return status_of(bf1::launch_decode_plan(a, (hipStream_t)stream));
}

int bf1_decode_workspace_size(int32_t batch, int32_t Hq, int32_t Hkv, int32_t head_dim,
                              int32_t plan_stride, int64_t* bytes) {
    if (!bytes || batch < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0 || plan_stride < 3)
        return BF1_ERR_INVALID_ARG;
    if (head_dim != 64 && head_dim != 128) return BF1_ERR_UNSUPPORTED;
    int32_t nsplit, ppw;
    decode_splits(batch, Hkv, (int64_t)plan_stride - 2, &nsplit, &ppw);
    *bytes = decode_ws_bytes(batch, Hq, Hkv, head_dim, nsplit);
    return BF1_OK;
}

int bf1_decode_attn(const void* Q, const void* K_pages, const void* V_pages, const int32_t* seq_lens,
                    int32_t num_pages, const int32_t* plan, int32_t plan_stride, void* O, float* LSE,
                    int32_t batch, int32_t Hq, int32_t Hkv, int32_t head_dim, int32_t B,
                    void* workspace, int64_t workspace_bytes, void* stream) {
    if (batch < 0 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return BF1_ERR_INVALID_ARG;
    if (num_pages < 1 || plan_stride < 3) return BF1_ERR_INVALID_ARG;
    const int32_t G = Hq / Hkv;
    if (head_dim != 64 && head_dim != 128) return BF1_ERR_UNSUPPORTED;
    if (B != 64 && B != 128) return BF1_ERR_UNSUPPORTED;
    if (G != 1 && G != 2 && G != 4 && G != 8) return BF1_ERR_UNSUPPORTED;
    if ((int64_t)batch * Hkv > (int64_t(1) << 22)) return BF1_ERR_INVALID_ARG;
    if ((double)num_pages * Hkv * B * head_dim > 4.0e18) return BF1_ERR_INVALID_ARG;
    if (batch == 0) return BF1_OK;
    if (!Q || !K_pages || !V_pages || !seq_lens || !plan || !O || !workspace) return BF1_ERR_INVALID_ARG;
    if (!aligned(Q, 16) || !aligned(K_pages, 16) || !aligned(V_pages, 16) || !aligned(O, 16) ||
        !aligned(workspace, 16) || !aligned(seq_lens, 4) || !aligned(plan, 4))
        return BF1_ERR_INVALID_ARG;
    if (LSE && !aligned(LSE, 4)) return BF1_ERR_INVALID_ARG;
    int32_t nsplit, ppw;
    decode_splits(batch, Hkv, (int64_t)plan_stride - 2, &nsplit, &ppw);
    if (workspace_bytes < decode_ws_bytes(batch, Hq, Hkv, head_dim, nsplit)) return BF1_ERR_BUFFER_TOO_SMALL;
    bf1::DecodeArgs a{Q, K_pages, V_pages, seq_lens, num_pages, plan, plan_stride, plan_stride - 3, O,
                      LSE, (float*)workspace, batch, Hq, Hkv, head_dim, B, nsplit, ppw};
    return status_of(bf1::launch_decode(a, (hipStream_t)stream));
}

}  // extern "C"
