// BF1 causal dyadic block-sparse attention: device kernels for gfx950.
//
// Two kernels:
//  * bf1_plan_kernel -- the integer route planner (paper §3.1, Eq. 1): one
//    thread per query block writes its CSR row in closed form.
//  * attn_fwd_kernel -- flash-style prefill forward over a block route.  The
//    BF1 instance walks the CSR row of its query block; the dense instance
//    walks every block 0..j (the dense causal comparator).
//
// Work decomposition.  One workgroup handles one (batch, kv-head, query
// block, row chunk): the G q-heads of a GQA group are stacked, so G*B query
// rows share every K/V tile that is staged in LDS; a chunk is up to 128 of
// those stacked rows and each wave owns 32 of them.
//
// Matrix-core layout (v_mfma_f32_32x32x16_bf16).  The kernel computes the
// TRANSPOSED score tile S^T = K Q^T (rows = keys, columns = queries), so a
// lane owns one query column and 16 of the 32 key rows of a tile; the row max
// and row sum of the softmax are then in-lane reductions plus one exchange
// with the lane 32 apart.  The same lane then holds exactly the P^T values it
// must feed as the B operand of O^T = V^T P^T, so P never leaves registers.
// V^T is produced in LDS by a register transpose while staging the tile.
//
// Accumulator layout of a 32x32 MFMA tile (lane l, register r):
//   row = 8*(r/4) + 4*(l/32) + (r%4), column = l%32.
// A operand: row l%32, 8 consecutive k for lane half l/32; B operand:
// column l%32, the same 8 k.  Any fixed relabelling of k applied to both
// operands leaves the contraction unchanged, which the P^T/V^T pairing uses.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bf1_kernels.h"
#include "bf1_route.h"

namespace bf1 {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int KT = 64;  // keys per LDS tile
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr float RESCALE_LOG2 = 8.0f;  // lazy-rescale threshold (log2 units)

// ---------------------------------------------------------------------------
// Route planner
// ---------------------------------------------------------------------------

__global__ void bf1_plan_kernel(int32_t NB, int32_t L, int32_t* __restrict__ row_ptr,
                                int32_t* __restrict__ col_idx) {
    const int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j > NB) return;
    const int64_t start = route_row_start(j, L);
    row_ptr[j] = (int32_t)start;
    if (j == NB) return;
    // Ascending emission: global block 0, dyadic predecessors j - 2^r for
    // descending r (offsets above L only; smaller ones are local), the local
    // window j-min(j,L) .. j-1, then the self block.  Values that repeat the
    // last one written (block 0 reached again) are dropped.
    // Writes stop at the closed-form end of the row, so the table can never
    // be overrun.
    const int64_t end = route_row_start(j + 1, L);
    int64_t e = start;
    int32_t last = 0;
    if (e < end) col_idx[e++] = 0;
    if (j == 0) return;
    int rmax = 31 - __builtin_clz((unsigned)j);
    for (int r = rmax; r >= 2; --r) {
        const int32_t off = 1 << r;
        if (off > L) {
            const int32_t v = j - off;
            if (v > last && e < end) { col_idx[e++] = v; last = v; }
        }
    }
    const int32_t nloc = j < L ? j : L;
    for (int32_t l = nloc; l >= 1; --l) {
        const int32_t v = j - l;
        if (v > last && e < end) { col_idx[e++] = v; last = v; }
    }
    if (e < end) col_idx[e] = j;
}

// ---------------------------------------------------------------------------
// LDS tile layouts
// ---------------------------------------------------------------------------
// K tile : KT rows (keys) x D bf16, stored as 16-byte chunks; chunk c of key
//          row k sits at physical chunk c ^ kswz(k) so that the 16 lanes of
//          one LDS cycle (consecutive keys, same logical chunk) hit 16
//          distinct 4-bank groups.
// V^T tile: D rows x KT key slots.  Inside each group of 16 keys, key
//          16g + 8a + 4h + c (a,h in {0,1}, c in 0..3) is stored at slot
//          16g + 8h + 4a + c, so the 8 keys that lane half h feeds to one PV
//          MFMA k-step are one contiguous 16-byte chunk.  Chunks are swizzled
//          by vswz(d) for the same reason as K.
template <int D>
__device__ __forceinline__ int kswz(int key) {
    return D == 128 ? (key & 15) : ((key >> 1) & 7);
}
__device__ __forceinline__ int vswz(int d) { return (d >> 1) & 7; }

template <int D>
struct TileSmem {
    u32x4 k[2][KT * D / 8];
    u32x4 v[2][D * KT / 8];
};

// ---------------------------------------------------------------------------
// Attention forward
// ---------------------------------------------------------------------------

template <int D, int G, int BW, int NW, bool DENSE>
__global__ __launch_bounds__(NW * 64, 2) void attn_fwd_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    __bf16* __restrict__ O, float* __restrict__ LSE, const int32_t* __restrict__ row_ptr,
    const int32_t* __restrict__ col_idx, int64_t nnz, int32_t n, int32_t NB, int32_t batch_hkv,
    int32_t Hkv, float c_log2) {
    constexpr int NT = NW * 64;
    constexpr int ROWS = NW * 32;             // stacked query rows per workgroup
    constexpr int NCHUNK = (G * BW + ROWS - 1) / ROWS;
    constexpr int NSUB = BW / KT;             // LDS tiles per key block
    constexpr int DCH = D / 8;                // 16-byte chunks per K row
    constexpr int KS = D / 16;                // MFMA k-steps for S
    constexpr int DT = D / 32;                // 32-wide d tiles of O
    static_assert(ROWS * NCHUNK == G * BW, "rows must tile the stacked group");
    static_assert((KT * DCH) % NT == 0, "K tile chunks must split evenly");
    static_assert((16 * DCH) % NT == 0 || NT % (16 * DCH) == 0, "V jobs must split");

    __shared__ TileSmem<D> sm;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
    const int col = lane & 31;   // query column owned by this lane
    const int half = lane >> 5;  // lane half: selects k-range / row group

    // ---- work item (heaviest query blocks first) --------------------------
    const int32_t x = blockIdx.x;
    const int chunk = x % NCHUNK;
    const int32_t y = x / NCHUNK;
    const int32_t bh = y % batch_hkv;
    const int32_t j = NB - 1 - y / batch_hkv;
    const int32_t beta = bh / Hkv;
    const int32_t g = bh % Hkv;
    const int Hq = Hkv * G;

    const int srow = chunk * ROWS + wave * 32;  // first stacked row of this wave
    const int gi = srow / BW;                   // q-head within the group
    const int p0 = srow % BW;                   // first position in the block
    const int head = g * G + gi;
    const int32_t qpos = j * BW + p0 + col;     // token of this lane's query
    const bool qvalid = qpos < n;

    const __bf16* Qh = Q + ((int64_t)beta * Hq + head) * (int64_t)n * D;
    const __bf16* Kh = K + ((int64_t)beta * Hkv + g) * (int64_t)n * D;
    const __bf16* Vh = V + ((int64_t)beta * Hkv + g) * (int64_t)n * D;

    // ---- Q fragments (B operand of S^T = K Q^T), zero past n ---------------
    bf16x8 qf[KS];
    {
        const u32x4* src = reinterpret_cast<const u32x4*>(Qh + (int64_t)qpos * D);
#pragma unroll
        for (int s = 0; s < KS; ++s) {
            u32x4 w = {0u, 0u, 0u, 0u};
            if (qvalid) w = src[2 * s + half];
            qf[s] = __builtin_bit_cast(bf16x8, w);
        }
    }

    // ---- route walk ---------------------------------------------------------
    int32_t pos, pos_end;
    if (DENSE) {
        pos = 0;
        pos_end = j + 1;
    } else {
        int64_t e0 = row_ptr[j], e1 = row_ptr[j + 1];
        e0 = e0 < 0 ? 0 : (e0 > nnz ? nnz : e0);
        e1 = e1 < e0 ? e0 : (e1 > nnz ? nnz : e1);
        pos = (int32_t)e0;
        pos_end = (int32_t)e1;
    }
    // Advance (p, u) to the next tile that exists: a valid block i in [0, j]
    // whose sub-tile u starts before n.  All quantities fit in 32 bits
    // (i * BW < n + BW < 2^31).
    auto seek = [&](int32_t& p, int& u, int32_t& i) -> bool {
        for (; p < pos_end; ++p, u = 0) {
            i = DENSE ? p : col_idx[p];
            if (i < 0 || i > j) continue;
            for (; u < NSUB; ++u)
                if (i * BW + u * KT < n) return true;
        }
        return false;
    };

    // ---- global -> register staging of one K/V tile ------------------------
    constexpr int KLD = KT * DCH / NT;                              // K chunks per thread
    constexpr int VJOBS = 16 * DCH;                                 // (4 keys x 8 d) jobs
    constexpr int VLD = VJOBS >= NT ? VJOBS / NT : 1;
    u32x4 kreg[KLD];
    u32x4 vreg[VLD][4];

    // Keys at or past n occur only in the self block of the last query block,
    // where every query that exists sees them with probability exactly 0.
    // Their rows are therefore loaded from a clamped, valid row of the same
    // tile (finite data, 0 * finite = 0) instead of being zeroed, so the
    // loaded registers are never touched before they are stored to LDS and
    // the loads stay in flight across the compute of the current tile.
    auto load_tile = [&](int32_t i, int u) {
        const int32_t key0 = i * BW + u * KT;
        const __bf16* kb = Kh + (int64_t)key0 * D;
        const __bf16* vb = Vh + (int64_t)key0 * D;
        const int32_t last = n - key0 - 1;  // last valid row of the tile (>= 0)
#pragma unroll
        for (int it = 0; it < KLD; ++it) {
            const int idx = tid + it * NT;
            const int kr = min(idx / DCH, last), c = idx % DCH;
            kreg[it] = *reinterpret_cast<const u32x4*>(kb + kr * D + c * 8);
        }
#pragma unroll
        for (int it = 0; it < VLD; ++it) {
            const int job = (VJOBS % NT == 0) ? tid + it * NT : (tid % VJOBS);
            const int kg = job & 15, dc = job >> 4;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int kr = min(4 * kg + q, last);
                vreg[it][q] = *reinterpret_cast<const u32x4*>(vb + kr * D + dc * 8);
            }
        }
    };

    auto store_tile = [&](int buf) {
#pragma unroll
        for (int it = 0; it < KLD; ++it) {
            const int idx = tid + it * NT;
            const int kr = idx / DCH, c = idx % DCH;
            sm.k[buf][kr * DCH + (c ^ kswz<D>(kr))] = kreg[it];
        }
        u32x2* vt = reinterpret_cast<u32x2*>(&sm.v[buf][0]);
#pragma unroll
        for (int it = 0; it < VLD; ++it) {
            const int job = (VJOBS % NT == 0) ? tid + it * NT : (tid % VJOBS);
            const int kg = job & 15, dc = job >> 4;
            const int lchunk = 2 * (kg >> 2) + (kg & 1);  // logical 16-B chunk of the 4 keys
            const int hsel = (kg >> 1) & 1;                // which 8-B half of it
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const uint32_t w0 = vreg[it][0][p], w1 = vreg[it][1][p];
                const uint32_t w2 = vreg[it][2][p], w3 = vreg[it][3][p];
                // row d = 8 dc + 2p (low halves) and 8 dc + 2p + 1 (high halves)
                const u32x2 lo = {(w0 & 0xffffu) | (w1 << 16), (w2 & 0xffffu) | (w3 << 16)};
                const u32x2 hi = {(w0 >> 16) | (w1 & 0xffff0000u), (w2 >> 16) | (w3 & 0xffff0000u)};
                const int d0 = 8 * dc + 2 * p, d1 = d0 + 1;
                vt[2 * (d0 * 8 + (lchunk ^ vswz(d0))) + hsel] = lo;
                vt[2 * (d1 * 8 + (lchunk ^ vswz(d1))) + hsel] = hi;
            }
        }
    };

    // ---- accumulators -------------------------------------------------------
    f32x16 acc[DT];
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
    float m_run = -1e30f;     // running max, log2 units (finite: masked scores give 0)
    float l_run = 0.f;        // this lane's partial row sum (its 32 keys of each tile)

    auto compute_tile = [&](int buf, int32_t i, int u) {
        const bool diag = (i == j);
        const int kin = u * KT;  // first key position of the tile inside block i
        if (diag && kin > p0 + 31) return;  // every key is in this wave's future
        f32x16 s[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r) s[kt][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
                const int kr = 32 * kt + col;
                const u32x4 w = sm.k[buf][kr * DCH + ((2 * ks + half) ^ kswz<D>(kr))];
                s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w),
                                                                qf[ks], s[kt], 0, 0, 0);
            }
        }
        if (diag) {
            const int qin = p0 + col;  // query position inside the block
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int kp = kin + 32 * kt + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (kp > qin) s[kt][r] = -INFINITY;
                }
        }
        // Online softmax in the log2 domain (c_log2 = scale * log2 e).  A row's
        // running max m_run only moves when a score exceeds it by more than
        // 2^RESCALE_LOG2; otherwise the stale max is kept for numerator and
        // denominator alike, which is exact and keeps every p <= 2^RESCALE_LOG2.
        // The decision is per row (per lane), so a row's arithmetic never
        // depends on other rows' data; the wave only skips the rescale work
        // when no row needs it (alpha = 1 exactly for the others).
        float mx = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kt][r]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_cand = mx * c_log2;
        const bool need = m_cand > m_run + RESCALE_LOG2;
        if (__any(need)) {
            const float alpha = need ? __builtin_amdgcn_exp2f(m_run - m_cand) : 1.0f;
            m_run = need ? m_cand : m_run;
            l_run *= alpha;
#pragma unroll
            for (int t = 0; t < DT; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[t][r] *= alpha;
        }
        float ls = 0.f;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float p = __builtin_amdgcn_exp2f(fmaf(s[kt][r], c_log2, -m_run));
                s[kt][r] = p;
                ls += p;
            }
        l_run += ls;
        // O^T += V^T P^T
        bf16x8 pb[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            f32x8 pf;
#pragma unroll
            for (int m = 0; m < 8; ++m) pf[m] = s[t >> 1][8 * (t & 1) + m];
            pb[t] = __builtin_convertvector(pf, bf16x8);
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const int d = 32 * dt + col;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const u32x4 w = sm.v[buf][d * 8 + ((2 * t + half) ^ vswz(d))];
                acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w),
                                                                  pb[t], acc[dt], 0, 0, 0);
            }
        }
    };

    // ---- software pipeline: global loads of tile k+1 overlap compute of k ---
    int32_t cur_p = pos, cur_i = 0;
    int cur_u = 0;
    if (!seek(cur_p, cur_u, cur_i)) {
        // A row with no usable key block (possible only for a caller route
        // table): O = 0, LSE = -inf.
        if (qvalid) {
            __bf16* Orow = O + (((int64_t)beta * Hq + head) * (int64_t)n + qpos) * D;
#pragma unroll
            for (int c = 0; c < D / 2; c += 8)
                *reinterpret_cast<u32x4*>(Orow + half * (D / 2) + c) = u32x4{0u, 0u, 0u, 0u};
            if (LSE != nullptr && half == 0)
                LSE[((int64_t)beta * Hq + head) * (int64_t)n + qpos] = -INFINITY;
        }
        return;
    }
    load_tile(cur_i, cur_u);
    store_tile(0);
    __syncthreads();
    int buf = 0;
    bool have = true;
    do {
        int32_t nxt_p = cur_p, nxt_i = 0;
        int nxt_u = cur_u + 1;
        const bool have_n = seek(nxt_p, nxt_u, nxt_i);
        if (have_n) load_tile(nxt_i, nxt_u);
        compute_tile(buf, cur_i, cur_u);
        if (have_n) store_tile(buf ^ 1);
        __syncthreads();
        buf ^= 1;
        cur_p = nxt_p;
        cur_u = nxt_u;
        cur_i = nxt_i;
        have = have_n;
    } while (have);

    // ---- epilogue: O = acc / l, LSE = (m + log2 l) ln 2 ---------------------
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (!qvalid) return;
    const float inv = 1.f / l_tot;
    __bf16* Orow = O + (((int64_t)beta * Hq + head) * (int64_t)n + qpos) * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
            f32x4 v4;
#pragma unroll
            for (int c = 0; c < 4; ++c) v4[c] = acc[dt][4 * gq + c] * inv;
            *reinterpret_cast<bf16x4*>(Orow + 32 * dt + 8 * gq + 4 * half) =
                __builtin_convertvector(v4, bf16x4);
        }
    if (LSE != nullptr && half == 0)
        LSE[((int64_t)beta * Hq + head) * (int64_t)n + qpos] = (m_run + log2f(l_tot)) * LN2;
}

template <int D, int G, int BW, bool DENSE>
hipError_t launch_attn(const AttnArgs& a, hipStream_t stream) {
    constexpr int NW = (G * BW) >= 128 ? 4 : (G * BW) / 32;
    constexpr int ROWS = NW * 32;
    constexpr int NCHUNK = (G * BW + ROWS - 1) / ROWS;
    const int32_t NB = (int32_t)((a.n + BW - 1) / BW);
    const int64_t items = (int64_t)NB * a.batch * a.Hkv * NCHUNK;
    if (items == 0) return hipSuccess;
    if (items > 0x7fffffff) return hipErrorInvalidValue;
    const float c_log2 = (1.0f / sqrtf((float)D)) * LOG2E;
    hipLaunchKernelGGL((attn_fwd_kernel<D, G, BW, NW, DENSE>), dim3((unsigned)items), dim3(NW * 64),
                       0, stream, (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V,
                       (__bf16*)a.O, a.LSE, a.row_ptr, a.col_idx, a.nnz, (int32_t)a.n, NB,
                       a.batch * a.Hkv, a.Hkv, c_log2);
    return hipGetLastError();
}

template <int D, int G>
hipError_t dispatch_bw(const AttnArgs& a, hipStream_t s) {
    if (a.dense) return launch_attn<D, G, 64, true>(a, s);
    if (a.B == 64) return launch_attn<D, G, 64, false>(a, s);
    return launch_attn<D, G, 128, false>(a, s);
}

template <int D>
hipError_t dispatch_g(const AttnArgs& a, hipStream_t s) {
    switch (a.Hq / a.Hkv) {
        case 1: return dispatch_bw<D, 1>(a, s);
        case 2: return dispatch_bw<D, 2>(a, s);
        case 4: return dispatch_bw<D, 4>(a, s);
        default: return dispatch_bw<D, 8>(a, s);
    }
}

}  // namespace

hipError_t launch_plan(int32_t NB, int32_t L, int32_t* row_ptr, int32_t* col_idx,
                       hipStream_t stream) {
    const int threads = 256;
    const int blocks = (NB + 1 + threads - 1) / threads;
    hipLaunchKernelGGL(bf1_plan_kernel, dim3(blocks), dim3(threads), 0, stream, NB, L, row_ptr,
                       col_idx);
    return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, hipStream_t stream) {
    if (a.head_dim == 64) return dispatch_g<64>(a, stream);
    return dispatch_g<128>(a, stream);
}

}  // namespace bf1
