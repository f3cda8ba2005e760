// BF1 one-token decode over a paged key/value cache, for gfx950.
//
// The newest token of a sequence (position t = seq_len - 1, query block
// j = t / B) attends to the keys of row t of the paper's §3.1 mask: every key
// of the earlier selected blocks of P(j) (Eq. 1) and the keys j*B .. t of its
// own block.  §3.2 notes that such a token reads only O(log NB) blocks; here a
// block is one cache page of B tokens, so a step reads |P(j)| pages per
// kv-head.  The selected pages stay the same for all B tokens of block j
// (§5.4: a plan can persist across the 64-token route epoch), so they are
// listed once per epoch by the plan kernel and reused by every step.
//
// Cache layout: K and V pages [num_pages, Hkv, B, D] bf16 (a page holds B
// consecutive tokens of one sequence; one (page, kv-head) slice is contiguous,
// B * D * 2 bytes).  A page table [batch, max_pages] maps each sequence's
// logical block i to its physical page; only the planner reads it.
//
// Plan row of a sequence (int32, `stride` = 3 + cap entries):
//   [0]                 block j the plan was made for (-1: not plannable)
//   [1]                 c, the number of earlier selected pages
//   [2, 2 + c)          their physical pages, ascending logical block
//   [2 + c]             the page of block j itself
// A step reads only its sequence length and this row, two independent loads,
// before it can address the cache.
//
// Split kernel: one workgroup of four waves per (sequence, kv-head, split);
// a split is `ppw` consecutive pages of the sequence's list (earlier pages,
// then the self page).  Each wave takes a quarter of every page's keys: lanes
// read 16-byte chunks of key rows (D / 8 lanes per row), form the G scores of
// a row by a cross-lane sum, and keep an online softmax (log2 units) with the
// matching V chunks.  The four waves merge in LDS; a split that covers the
// whole list writes O and LSE at once, otherwise it writes a partial record
// (per q-head: max, sum, unnormalised O row).  Merge kernel: one workgroup
// per (sequence, kv-head) with more than one split sums the records in split
// order (deterministic).  The kernel boundary orders the records before their
// readers; a single kernel with a completion counter would need device-scope
// release/acquire fences per workgroup, which write back and invalidate the
// whole L2 of an XCD each time and cost far more than the second launch.
// Masked keys (past t in the self page) contribute exactly nothing, whatever
// the page holds there.
#include <hip/hip_runtime.h>
#include <math.h>

#include "bf1_device.h"
#include "bf1_kernels.h"

namespace bf1 {
namespace {

constexpr int DEC_THREADS = 256;
constexpr int DEC_WAVES = DEC_THREADS / 64;
constexpr int PLAN_THREADS = 64;
constexpr int MAX_ROUTE = 64;  // bound on |P(j)| - 1 for any j < 2^31 and L <= 32

// ---------------------------------------------------------------------------
// Plan: one workgroup per sequence.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(PLAN_THREADS) void decode_plan_kernel(
    int32_t batch, const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ page_table,
    int32_t max_pages, int32_t num_pages, int32_t B, int32_t L, int32_t dense,
    int32_t* __restrict__ plan, int32_t stride, int32_t cap) {
    __shared__ int32_t blocks[MAX_ROUTE];
    __shared__ int32_t count;
    __shared__ int32_t bad;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    if (b >= batch) return;
    int32_t* row = plan + (int64_t)b * stride;
    const int64_t t = (int64_t)seq_lens[b] - 1;
    const int64_t j = t >= 0 ? t / B : -1;
    if (tid == 0) {
        bad = (t < 0 || j >= max_pages) ? 1 : 0;
        int c = 0;
        if (!bad && !dense) {
            // earlier blocks of P(j), ascending: 0, j - 2^r (r from high to
            // low, 2^r > L, skipping j - 2^r = 0), then j-L .. j-1
            if (j > L) blocks[c++] = 0;
            int r = 2;
            while (r < 30 && (int64_t(1) << (r + 1)) <= j) ++r;
            for (; r >= 2; --r) {
                const int64_t off = int64_t(1) << r;
                if (off <= j && off > L && j - off > 0) blocks[c++] = (int32_t)(j - off);
            }
            for (int64_t i = (j - L > 0 ? j - L : 0); i < j; ++i) blocks[c++] = (int32_t)i;
        } else if (!bad) {
            c = (int)j;
        }
        if (c > cap) bad = 1;
        count = c;
    }
    __syncthreads();
    const int c = count;
    const int32_t* pt = page_table + (int64_t)b * max_pages;
    if (!bad) {
        for (int e = tid; e < c; e += PLAN_THREADS) {
            const int32_t i = dense ? e : blocks[e];
            const int32_t p = pt[i];
            if (p < 0 || p >= num_pages) atomicOr(&bad, 1);
            row[2 + e] = p;
        }
        if (tid == 0) {
            const int32_t p = pt[j];  // the self page must exist as well
            if (p < 0 || p >= num_pages) atomicOr(&bad, 1);
            row[2 + c] = p;
        }
    }
    __syncthreads();
    if (tid == 0) {
        row[0] = bad ? -1 : (int32_t)j;
        row[1] = bad ? 0 : c;
    }
}

__device__ __forceinline__ void bf16x8_to_float(u32x4 w, float* f) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        f[2 * k] = __uint_as_float(w[k] << 16);
        f[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
    }
}

// ---------------------------------------------------------------------------
// Decode attention.
// ---------------------------------------------------------------------------

// What one step of sequence b reads: its newest position t, block j and the
// number c of earlier pages in its plan row.  False if the plan row was made
// for another block or is not a planner row; both kernels take the same
// decision from the same data.
struct StepView {
    int64_t t, j;
    int c;
};

__device__ __forceinline__ bool step_view(const int32_t* __restrict__ seq_lens, const int32_t* row,
                                          int32_t cap, int PW, int b, StepView* v) {
    const int32_t n = seq_lens[b];
    const int32_t pj = row[0];
    const int32_t pc = row[1];
    v->t = (int64_t)n - 1;
    v->j = v->t >= 0 ? v->t / PW : -1;
    v->c = pc;
    return v->t >= 0 && pj == v->j && pc >= 0 && pc <= cap;
}

template <int D, int G>
__device__ __forceinline__ void write_nan(__bf16* O, float* LSE, int b, int Hq, int h, int tid, int nthreads) {
    for (int x = tid; x < G * D; x += nthreads)
        O[((int64_t)b * Hq + h * G + x / D) * D + x % D] = (__bf16)__builtin_nanf("");
    if (LSE != nullptr && tid < G) LSE[(int64_t)b * Hq + h * G + tid] = __builtin_nanf("");
}

// A unit of decode work for one wave: a quarter of a page (KPW consecutive
// keys), read as NI wave-wide loads of K rows and of V rows; lane `lane` holds
// the 16-byte chunk cch of key row rg of every load.
template <int D, int PW>
struct Unit {
    static constexpr int LPR = D / 8;    // lanes per key row (16 bytes each)
    static constexpr int RPI = 64 / LPR;  // key rows per wave-wide load
    static constexpr int KPW = PW / 4;    // keys per unit (a quarter page)
    static constexpr int NI = KPW / RPI;  // loads per unit (for K, and for V)
    static_assert(NI >= 1 && KPW % RPI == 0, "page width and head_dim mismatch");
};

// K and V page rows are read once per decode step (a page is not shared
// between the workgroups of a step), so the loads are non-temporal: they do
// not displace other lines in L2.
template <int D, int PW>
__device__ __forceinline__ void load_unit(const __bf16* __restrict__ Kp, const __bf16* __restrict__ Vp,
                                          int64_t page_base, int quarter, int rg, int cch, u32x4* kr,
                                          u32x4* vr) {
    using U = Unit<D, PW>;
#pragma unroll
    for (int i = 0; i < U::NI; ++i) {
        const int key = quarter * U::KPW + i * U::RPI + rg;
        kr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(Kp + page_base + (int64_t)key * D + cch * 8));
    }
#pragma unroll
    for (int i = 0; i < U::NI; ++i) {
        const int key = quarter * U::KPW + i * U::RPI + rg;
        vr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(Vp + page_base + (int64_t)key * D + cch * 8));
    }
}

// Online softmax over one unit: the G scores of each key row (cross-lane sum
// over the LPR lanes of the row), masked past nvalid keys of the page (their
// V chunks zeroed), folded into the wave's running max / sum / row.
template <int D, int G, int PW>
__device__ __forceinline__ void consume_unit(const u32x4* kr, const u32x4* vr, int quarter, int rg, int nvalid,
                                             const float (&qv)[G][8], float (&m_run)[G], float (&l_run)[G],
                                             float (&o_acc)[G][8]) {
    using U = Unit<D, PW>;
    constexpr int NI = U::NI;
    float sc[G][NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
        float kf[8];
        bf16x8_to_float(kr[i], kf);
#pragma unroll
        for (int e = 0; e < G; ++e) {
            float acc = 0.f;
#pragma unroll
            for (int k = 0; k < 8; ++k) acc = fmaf(qv[e][k], kf[k], acc);
            sc[e][i] = acc;
        }
    }
#pragma unroll
    for (int x = 1; x < U::LPR; x <<= 1)
#pragma unroll
        for (int e = 0; e < G; ++e)
#pragma unroll
            for (int i = 0; i < NI; ++i) sc[e][i] += __shfl_xor(sc[e][i], x);
    bool valid[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) valid[i] = quarter * U::KPW + i * U::RPI + rg < nvalid;
#pragma unroll
    for (int e = 0; e < G; ++e) {
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < NI; ++i) mx = fmaxf(mx, valid[i] ? sc[e][i] : -INFINITY);
#pragma unroll
        for (int x = U::LPR; x < 64; x <<= 1) mx = fmaxf(mx, __shfl_xor(mx, x));
        const float m_new = fmaxf(m_run[e], mx);
        if (m_new == -INFINITY) continue;  // no visible key for this wave so far
        const float alpha = exp2f(m_run[e] - m_new);
        m_run[e] = m_new;
        l_run[e] *= alpha;
#pragma unroll
        for (int k = 0; k < 8; ++k) o_acc[e][k] *= alpha;
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const float pr = valid[i] ? exp2f(sc[e][i] - m_new) : 0.f;
            l_run[e] += pr;
            float vf[8];
            bf16x8_to_float(valid[i] ? vr[i] : u32x4{0u, 0u, 0u, 0u}, vf);
#pragma unroll
            for (int k = 0; k < 8; ++k) o_acc[e][k] = fmaf(pr, vf[k], o_acc[e][k]);
        }
    }
}

// The wave's totals (sums over the RPI key rows of each load) into LDS slot
// red[wave]: max, sum, unnormalised row.
template <int D, int G>
__device__ __forceinline__ void wave_totals_to_lds(float (&red)[G][D + 2], int lane, int rg, int cch,
                                                   float (&m_run)[G], float (&l_run)[G], float (&o_acc)[G][8]) {
    constexpr int LPR = D / 8;
#pragma unroll
    for (int x = LPR; x < 64; x <<= 1)
#pragma unroll
        for (int e = 0; e < G; ++e) {
            l_run[e] += __shfl_xor(l_run[e], x);
#pragma unroll
            for (int k = 0; k < 8; ++k) o_acc[e][k] += __shfl_xor(o_acc[e][k], x);
        }
    if (rg == 0) {
#pragma unroll
        for (int e = 0; e < G; ++e)
#pragma unroll
            for (int k = 0; k < 8; ++k) red[e][2 + cch * 8 + k] = o_acc[e][k];
    }
    if (lane == 0) {
#pragma unroll
        for (int e = 0; e < G; ++e) {
            red[e][0] = m_run[e];
            red[e][1] = l_run[e];
        }
    }
}

template <int D, int G>
__device__ __forceinline__ void load_query(const __bf16* __restrict__ Q, int b, int Hq, int h, int cch,
                                           float c_log2, float (&qv)[G][8]) {
#pragma unroll
    for (int e = 0; e < G; ++e) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(Q + ((int64_t)b * Hq + h * G + e) * D + cch * 8);
        bf16x8_to_float(w, qv[e]);
#pragma unroll
        for (int k = 0; k < 8; ++k) qv[e][k] *= c_log2;
    }
}

template <int G>
__device__ __forceinline__ void init_running(float (&m_run)[G], float (&l_run)[G], float (&o_acc)[G][8]) {
#pragma unroll
    for (int e = 0; e < G; ++e) {
        m_run[e] = -INFINITY;
        l_run[e] = 0.f;
#pragma unroll
        for (int k = 0; k < 8; ++k) o_acc[e][k] = 0.f;
    }
}

template <int D, int G, int PW>
__global__ __launch_bounds__(DEC_THREADS) void decode_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ Kp, const __bf16* __restrict__ Vp,
    const int32_t* __restrict__ seq_lens, int32_t num_pages, const int32_t* __restrict__ plan,
    int32_t stride, int32_t cap, __bf16* __restrict__ O, float* __restrict__ LSE,
    float* __restrict__ ws, int32_t Hkv, int32_t nsplit, int32_t ppw, float c_log2) {
    using U = Unit<D, PW>;
    constexpr int NI = U::NI;
    constexpr int REC = G * (D + 2);      // floats per partial record

    __shared__ float red[DEC_WAVES][G][D + 2];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int rg = lane / U::LPR;
    const int cch = lane % U::LPR;
    const int s = blockIdx.x % nsplit;
    const int bh = blockIdx.x / nsplit;
    const int h = bh % Hkv;
    const int b = bh / Hkv;
    const int Hq = Hkv * G;
    const int32_t* row = plan + (int64_t)b * stride;

    StepView sv;
    if (!step_view(seq_lens, row, cap, PW, b, &sv)) {
        // stale or unplannable: the outputs of this (sequence, kv-head) are NaN
        if (s == 0) write_nan<D, G>(O, LSE, b, Hq, h, tid, DEC_THREADS);
        return;
    }
    const int c = sv.c;
    const int npages = c + 1;
    const int nsb = (npages + ppw - 1) / ppw;
    if (s >= nsb) return;
    const int p0 = s * ppw;
    const int p1 = min(npages, p0 + ppw);

    float qv[G][8];
    load_query<D, G>(Q, b, Hq, h, cch, c_log2, qv);
    float m_run[G], l_run[G], o_acc[G][8];
    init_running<G>(m_run, l_run, o_acc);

    // Wave w takes quarter w of every page of the split; with PREFETCH the
    // next page's loads are issued before the current page is consumed (where
    // registers allow), so a wave keeps two pages of loads in flight.  Pages
    // written by the planner are in range; the clamp only keeps a foreign plan
    // row from addressing memory outside the cache.
    constexpr bool PREFETCH = G * NI <= 16;
    auto page_base = [&](int p) {
        return ((int64_t)min(max(row[2 + p], 0), num_pages - 1) * Hkv + h) * PW * D;
    };
    u32x4 kr[NI], vr[NI];
    if constexpr (PREFETCH) load_unit<D, PW>(Kp, Vp, page_base(p0), wave, rg, cch, kr, vr);
    for (int p = p0; p < p1; ++p) {
        const int nvalid = p < c ? PW : (int)(sv.t - sv.j * PW + 1);
        u32x4 kn[NI], vn[NI];
        if constexpr (PREFETCH) {
            if (p + 1 < p1) load_unit<D, PW>(Kp, Vp, page_base(p + 1), wave, rg, cch, kn, vn);
        } else {
            load_unit<D, PW>(Kp, Vp, page_base(p), wave, rg, cch, kr, vr);
        }
        consume_unit<D, G, PW>(kr, vr, wave, rg, nvalid, qv, m_run, l_run, o_acc);
        if constexpr (PREFETCH) {
#pragma unroll
            for (int i = 0; i < NI; ++i) {
                kr[i] = kn[i];
                vr[i] = vn[i];
            }
        }
    }
    wave_totals_to_lds<D, G>(red[wave], lane, rg, cch, m_run, l_run, o_acc);
    __syncthreads();

    const bool single = nsb == 1;
    float* rec = ws + ((int64_t)bh * nsplit + s) * REC;
    for (int x = tid; x < G * D; x += DEC_THREADS) {
        const int e = x / D, d = x % D;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < DEC_WAVES; ++w) M = fmaxf(M, red[w][e][0]);
        float o = 0.f, l = 0.f;
#pragma unroll
        for (int w = 0; w < DEC_WAVES; ++w) {
            const float sw = red[w][e][0] == -INFINITY ? 0.f : exp2f(red[w][e][0] - M);
            o = fmaf(red[w][e][2 + d], sw, o);
            l = fmaf(red[w][e][1], sw, l);
        }
        if (single) {
            O[((int64_t)b * Hq + h * G + e) * D + d] = (__bf16)(o / l);
            if (d == 0 && LSE != nullptr) LSE[(int64_t)b * Hq + h * G + e] = (M + log2f(l)) * LN2;
        } else {
            rec[e * (D + 2) + 2 + d] = o;
            if (d == 0) {
                rec[e * (D + 2)] = M;
                rec[e * (D + 2) + 1] = l;
            }
        }
    }
}

// Merge of the split records of one (sequence, kv-head), in split order:
// every thread owns one (q-head, dim) output and folds the records in groups
// of sixteen (their loads issued together, so a selected list of up to 16
// splits costs one load round trip) into a running max / sum / row.
template <int D, int G, int PW>
__global__ __launch_bounds__(DEC_THREADS) void decode_merge_kernel(
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ plan, int32_t stride,
    int32_t cap, __bf16* __restrict__ O, float* __restrict__ LSE, const float* __restrict__ ws,
    int32_t Hkv, int32_t nsplit, int32_t ppw) {
    constexpr int REC = G * (D + 2);
    constexpr int U = 16;
    const int tid = threadIdx.x;
    const int bh = blockIdx.x;
    const int h = bh % Hkv;
    const int b = bh / Hkv;
    const int Hq = Hkv * G;
    StepView sv;
    if (!step_view(seq_lens, plan + (int64_t)b * stride, cap, PW, b, &sv))
        return;  // the split kernel wrote NaN
    const int nsb = (sv.c + 1 + ppw - 1) / ppw;
    if (nsb <= 1) return;  // the split kernel wrote the result
    const float* recs = ws + (int64_t)bh * nsplit * REC;
    for (int x = tid; x < G * D; x += DEC_THREADS) {
        const int e = x / D, d = x % D;
        float M = -INFINITY, l = 0.f, o = 0.f;
        for (int q0 = 0; q0 < nsb; q0 += U) {
            float mq[U], lq[U], oq[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const bool in = q0 + u < nsb;
                const float* r = recs + (int64_t)(in ? q0 + u : 0) * REC + e * (D + 2);
                mq[u] = in ? r[0] : -INFINITY;
                lq[u] = in ? r[1] : 0.f;
                oq[u] = in ? r[2 + d] : 0.f;
            }
            float mm = M;
#pragma unroll
            for (int u = 0; u < U; ++u) mm = fmaxf(mm, mq[u]);
            if (mm == -INFINITY) continue;
            const float a = exp2f(M - mm);  // 0 while nothing is accumulated
            l *= a;
            o *= a;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const float w = mq[u] == -INFINITY ? 0.f : exp2f(mq[u] - mm);
                l = fmaf(lq[u], w, l);
                o = fmaf(oq[u], w, o);
            }
            M = mm;
        }
        O[((int64_t)b * Hq + h * G + e) * D + d] = (__bf16)(o / l);
        if (d == 0 && LSE != nullptr) LSE[(int64_t)b * Hq + h * G + e] = (M + log2f(l)) * LN2;
    }
}

template <int D, int G, int PW>
hipError_t launch_decode_pw(const DecodeArgs& a, hipStream_t st) {
    const float c_log2 = LOG2E / sqrtf((float)D);
    hipLaunchKernelGGL((decode_kernel<D, G, PW>), dim3((unsigned)((int64_t)a.batch * a.Hkv * a.nsplit)),
                       dim3(DEC_THREADS), 0, st, (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V,
                       a.seq_lens, a.num_pages, a.plan, a.stride, a.cap, (__bf16*)a.O, a.LSE, a.ws, a.Hkv,
                       a.nsplit, a.ppw, c_log2);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.nsplit <= 1) return e;
    hipLaunchKernelGGL((decode_merge_kernel<D, G, PW>), dim3((unsigned)((int64_t)a.batch * a.Hkv)),
                       dim3(DEC_THREADS), 0, st, a.seq_lens, a.plan, a.stride, a.cap, (__bf16*)a.O, a.LSE,
                       a.ws, a.Hkv, a.nsplit, a.ppw);
    return hipGetLastError();
}

template <int D, int G>
hipError_t launch_decode_g(const DecodeArgs& a, hipStream_t st) {
    return a.B == 64 ? launch_decode_pw<D, G, 64>(a, st) : launch_decode_pw<D, G, 128>(a, st);
}

template <int D>
hipError_t launch_decode_d(const DecodeArgs& a, hipStream_t st) {
    switch (a.Hq / a.Hkv) {
        case 1: return launch_decode_g<D, 1>(a, st);
        case 2: return launch_decode_g<D, 2>(a, st);
        case 4: return launch_decode_g<D, 4>(a, st);
        default: return launch_decode_g<D, 8>(a, st);
    }
}

}  // namespace

hipError_t launch_decode_plan(const DecodePlanArgs& a, hipStream_t st) {
    hipLaunchKernelGGL(decode_plan_kernel, dim3((unsigned)a.batch), dim3(PLAN_THREADS), 0, st, a.batch,
                       a.seq_lens, a.page_table, a.max_pages, a.num_pages, a.B, a.L, a.dense, a.plan,
                       a.stride, a.cap);
    return hipGetLastError();
}

hipError_t launch_decode(const DecodeArgs& a, hipStream_t st) {
    return a.head_dim == 64 ? launch_decode_d<64>(a, st) : launch_decode_d<128>(a, st);
}

}  // namespace bf1
