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

#include <map>
#include <mutex>
#include <type_traits>

#include "bf1_device.h"
#include "bf1_kernels.h"
#include "bf1_route.h"

namespace bf1 {
namespace {

constexpr float RESCALE_LOG2 = 8.0f;  // lazy-rescale threshold (log2 units)
constexpr int KPF = 3;                // K operand reads in flight ahead of the score MFMAs

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
// LDS tile layouts (both tiles keep the natural [key][d] row order)
// ---------------------------------------------------------------------------
// K tile: KT rows x D bf16 in 16-byte chunks; logical chunk c of key row k
//   sits at physical chunk c ^ kswz(k), so the lanes of one LDS cycle of the
//   score MFMA's operand read (consecutive keys, same chunk) hit distinct banks.
// V tile: KT rows x D bf16 in 32-byte slots (16 d values); logical slot s of
//   key row k sits at physical slot s ^ vswz(k).  The PV operand is read with
//   the LDS transpose load (ds_read_b64_tr_b16): in each 16-lane group, lanes
//   4e..4e+3 address 8 consecutive bytes (4 d values) of key row e and lane i
//   receives the 4 keys' values of its own d.  vswz spreads the 4 key rows and
//   the 2 neighbouring slots read in one cycle over distinct banks.
// Both tiles are filled by direct global->LDS loads: one wave instruction
//   writes a contiguous 1 KB segment (16 bytes per lane, lane order), so each
//   lane fetches the global chunk whose swizzled position is its lane slot.
template <int D>
__device__ __forceinline__ int kswz(int key) {
    return D == 128 ? (key & 15) : ((key >> 1) & 7);
}
template <int D>
__device__ __forceinline__ int vswz(int key) {
    return D == 128 ? ((key & 3) << 1) : (((key >> 1) & 1) << 1);
}

template <int D>
struct TileSmem {
    u32x4 k[2][KT * D / 8];
    u32x4 v[2][KT * D / 8];
};

// Eight 64-bit LDS transpose reads (see the V tile layout above) at constant
// offsets O0 + k * STEP from one lane address, followed by the wait for them,
// all in ONE inline-assembly statement.  Keeping the wait inside the statement
// matters: the hardware writes the destination registers asynchronously, so
// the compiler must not see the values (or be free to reuse or copy their
// registers) before they have landed; the early-clobber outputs also keep
// them apart from the address register.  Inline assembly is used because the
// compiler's builtin for this instruction carries no memory-alias information
// and would make it wait for every in-flight buffer->LDS load of the other
// LDS buffer first.  LDS operations complete in order, so the extra wait never
// weakens the compiler's own lgkmcnt accounting.
template <int O0, int STEP>
__device__ __forceinline__ void lds_read_tr16_x8(uint32_t addr, u32x2 (&v)[8]) {
    static_assert(O0 >= 0 && O0 + 7 * STEP < 65536, "DS offsets are 16 bits");
    asm volatile(
        "ds_read_b64_tr_b16 %0, %8 offset:%9\n\t"
        "ds_read_b64_tr_b16 %1, %8 offset:%10\n\t"
        "ds_read_b64_tr_b16 %2, %8 offset:%11\n\t"
        "ds_read_b64_tr_b16 %3, %8 offset:%12\n\t"
        "ds_read_b64_tr_b16 %4, %8 offset:%13\n\t"
        "ds_read_b64_tr_b16 %5, %8 offset:%14\n\t"
        "ds_read_b64_tr_b16 %6, %8 offset:%15\n\t"
        "ds_read_b64_tr_b16 %7, %8 offset:%16\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]),
          "=&v"(v[6]), "=&v"(v[7])
        : "v"(addr), "i"(O0), "i"(O0 + STEP), "i"(O0 + 2 * STEP), "i"(O0 + 3 * STEP),
          "i"(O0 + 4 * STEP), "i"(O0 + 5 * STEP), "i"(O0 + 6 * STEP), "i"(O0 + 7 * STEP)
        : "memory");
}

// ---------------------------------------------------------------------------
// Attention forward
// ---------------------------------------------------------------------------

// KSPLIT = 2 (short sequences, at most one work item per compute unit): the
// workgroup holds two groups of NW waves that cover the same query rows and
// walk alternate tiles of the route (group 0 the even positions, group 1 the
// odd ones), each with its own LDS tiles; group 1 hands its running max, sums
// and unnormalised rows to group 0 through LDS, which merges and stores.  An
// item's chain of key tiles is halved, and two waves share each SIMD where a
// single workgroup would otherwise leave one.
template <int D, int G, int BW, int NW, bool DENSE, int KSPLIT>
__global__ __launch_bounds__(NW * 64 * KSPLIT, KSPLIT == 1 ? 2 : 1) void attn_fwd_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    __bf16* __restrict__ O, float* __restrict__ LSE, const int32_t* __restrict__ row_ptr,
    const int32_t* __restrict__ col_idx, int64_t nnz, int32_t n, int32_t NB, int32_t batch_hkv,
    int32_t Hkv, float c_log2) {
    constexpr int ROWS = NW * 32;             // stacked query rows per workgroup
    constexpr int NCHUNK = (G * BW + ROWS - 1) / ROWS;
    constexpr int NSUB = BW / KT;             // LDS tiles per key block
    constexpr int KS = D / 16;                // MFMA k-steps of the score product
    constexpr int DT = D / 32;                // 32-wide d tiles of O
    constexpr int RB = D * 2;                 // bytes per key row in LDS
    constexpr int TILE_B = KT * RB;           // bytes per K (or V) tile
    constexpr int SEGS = TILE_B / 1024;       // 1 KB direct-load segments per tile
    constexpr int ROWS_PER_SEG = 1024 / RB;
    constexpr int SEG_PER_WAVE = SEGS / NW;
    static_assert(ROWS * NCHUNK == G * BW, "rows must tile the stacked group");
    static_assert(SEGS % NW == 0, "segments must split over the waves");
    static_assert(KSPLIT == 1 || KSPLIT == 2, "one or two key groups");

    __shared__ TileSmem<D> smem[KSPLIT];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
    const int grp = wid / NW;     // key group (0 unless KSPLIT = 2)
    const int wave = wid % NW;    // wave within its group
    TileSmem<D>& sm = smem[grp];
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
    int32_t pos_end, cur_p;
    if (DENSE) {
        cur_p = 0;
        pos_end = j + 1;
    } else {
        int64_t e0 = row_ptr[j], e1 = row_ptr[j + 1];
        e0 = e0 < 0 ? 0 : (e0 > nnz ? nnz : e0);
        e1 = e1 < e0 ? e0 : (e1 > nnz ? nnz : e1);
        cur_p = (int32_t)e0;
        pos_end = (int32_t)e1;
    }
    int cur_u = 0;
    // Next tile of the route: a block i in [0, j] (caller tables may hold
    // anything else; such entries are skipped) and a 64-key sub-tile of it
    // that starts before n.  All quantities fit in 32 bits.  The table entry
    // at cur_p is fetched one call ahead (pref), so the scalar load latency
    // is hidden behind a pipeline step.
    int32_t pref = (!DENSE && cur_p < pos_end) ? col_idx[cur_p] : -1;
    auto advance = [&]() {
        ++cur_p;
        cur_u = 0;
        if (!DENSE) pref = (cur_p < pos_end) ? col_idx[cur_p] : -1;
    };
    auto next_tile = [&](int32_t& ti, int& tu) -> bool {
        while (cur_p < pos_end) {
            const int32_t i = DENSE ? cur_p : pref;
            if (i >= 0 && i <= j) {
                for (; cur_u < NSUB; ++cur_u)
                    if (i * BW + cur_u * KT < n) {
                        ti = i;
                        tu = cur_u++;
                        if (cur_u >= NSUB) advance();
                        return true;
                    }
            }
            advance();
        }
        return false;
    };
    // This group's next tile.  With two key groups the route's tiles are
    // taken in pairs: a pair exists if its first tile does (both groups see
    // the same walk, so they agree on the number of steps), and the group
    // whose tile of the pair is missing runs that step on a dummy tile whose
    // scores are all masked (it contributes exactly nothing).
    auto next_own = [&](int32_t& ti, int& tu, bool& real) -> bool {
        if (KSPLIT == 1) {
            real = next_tile(ti, tu);
            return real;
        }
        int32_t t0 = 0, t1 = 0;
        int u0 = 0, u1 = 0;
        if (!next_tile(t0, u0)) return false;
        const bool has1 = next_tile(t1, u1);
        ti = grp == 0 ? t0 : t1;
        tu = grp == 0 ? u0 : u1;
        real = grp == 0 || has1;
        return true;
    };

    // ---- direct buffer -> LDS staging ----------------------------------------
    // Keys at or past n occur only in the self block of the last query block,
    // where every query that exists sees them with probability exactly 0; the
    // buffer range check returns zeros for those rows (0 * 0 = 0 in P V, and
    // the zero scores are masked).  A tile that does not exist is "loaded"
    // from past the end: all lanes read zeros and no memory is touched.
    const uint32_t head_bytes = (uint32_t)n * RB;
    const __amdgpu_buffer_rsrc_t k_rsrc = head_rsrc(Kh, head_bytes);
    const __amdgpu_buffer_rsrc_t v_rsrc = head_rsrc(Vh, head_bytes);
    const int lrow = lane / (RB / 16);   // row inside a 1 KB segment
    const int pc = lane % (RB / 16);     // physical 16-byte chunk in the row
    uint32_t kgo[SEG_PER_WAVE], vgo[SEG_PER_WAVE];  // lane byte offsets inside a tile
#pragma unroll
    for (int it = 0; it < SEG_PER_WAVE; ++it) {
        const int row = (it * NW + wave) * ROWS_PER_SEG + lrow;
        kgo[it] = row * RB + (pc ^ kswz<D>(row)) * 16;
        vgo[it] = row * RB + (2 * ((pc >> 1) ^ vswz<D>(row)) + (pc & 1)) * 16;
    }
    auto tile_off = [&](bool exists, int32_t i, int u) -> uint32_t {
        return exists ? (uint32_t)(i * BW + u * KT) * RB : head_bytes;
    };
    auto load_k = [&](int kbuf, uint32_t soff) {
#pragma unroll
        for (int it = 0; it < SEG_PER_WAVE; ++it)
            load_lds16(k_rsrc, &sm.k[kbuf][(it * NW + wave) * 64], kgo[it], soff);
    };
    auto load_v = [&](int vbuf, uint32_t soff) {
#pragma unroll
        for (int it = 0; it < SEG_PER_WAVE; ++it)
            load_lds16(v_rsrc, &sm.v[vbuf][(it * NW + wave) * 64], vgo[it], soff);
    };

    // ---- lane-constant LDS read offsets -------------------------------------
    // Score operand: key row 32 kt + col, logical chunk 2 ks + half.  kswz
    // depends only on col, so kt adds a constant 32 rows.
    int kofs[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kofs[ks] = col * RB + 16 * ((2 * ks + half) ^ kswz<D>(col));
    // PV operand (transpose reads): group gq = lane/16 covers d 32 dt + 16 (gq%2)
    // .. +15 and keys 16 t + 4 (gq/2) + e (+8 for the second read); vswz of
    // those rows does not depend on t, so t and the +8 are constant offsets.
    const int gq = lane >> 4, kk = lane & 15;
    const int r0 = 4 * (gq >> 1) + (kk >> 2);
    int vofs[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
        vofs[dt] = r0 * RB + 32 * ((2 * dt + (gq & 1)) ^ vswz<D>(r0)) + 8 * (kk & 3);

    auto score_mfma = [&](auto kbuf_c, f32x16 (&s)[2]) {
        constexpr int KB = decltype(kbuf_c)::value;
        const char* kb = reinterpret_cast<const char*>(&sm.k[KB][0]);
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int r = 0; r < 16; ++r) s[kt][r] = 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
                const u32x4 w = *reinterpret_cast<const u32x4*>(kb + kofs[ks] + kt * 32 * RB);
                s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w),
                                                                qf[ks], s[kt], 0, 0, 0);
            }
    };

    // ---- accumulators -------------------------------------------------------
    f32x16 acc[DT];
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;
    float m_run = -1e30f;  // running max, log2 units (finite: masked scores give 0)
    float l_run = 0.f;     // this lane's partial row sum (its 32 keys of each tile)
    float l_bf = 0.f;      // the same sum over the bf16-rounded weights the PV product uses

    // ---- prologue: K0, V0 and K1 resident, S0 computed ----------------------
    int32_t ti0 = 0, ti1 = 0, ti2 = 0;
    int tu0 = 0, tu1 = 0, tu2 = 0;
    bool rl0 = true, rl1 = true, rl2 = true;  // tile k, k+1, k+2 is real (not a dummy)
    if (!next_own(ti0, tu0, rl0)) {
        // A row with no usable key block (possible only for a caller route
        // table): O = 0, LSE = -inf.
        if (qvalid && grp == 0) {
            __bf16* Orow = O + (((int64_t)beta * Hq + head) * (int64_t)n + qpos) * D;
#pragma unroll
            for (int c = 0; c < D / 2; c += 8)
                *reinterpret_cast<u32x4*>(Orow + half * (D / 2) + c) = u32x4{0u, 0u, 0u, 0u};
            if (LSE != nullptr && half == 0)
                LSE[((int64_t)beta * Hq + head) * (int64_t)n + qpos] = -INFINITY;
        }
        return;
    }
    bool h1 = next_own(ti1, tu1, rl1);
    load_k(0, tile_off(rl0, ti0, tu0));
    load_v(0, tile_off(rl0, ti0, tu0));
    if (h1) load_k(1, tile_off(rl1, ti1, tu1));
    __builtin_amdgcn_s_waitcnt(VMCNT0);
    __syncthreads();

    // Row statistics of a score tile: the self-block causal mask, then the
    // row max in log2 units (m_cand) and whether the running max must move.
    // Online softmax in the log2 domain (c_log2 = scale * log2 e): a row's
    // running max m_run only moves when a score exceeds it by more than
    // 2^RESCALE_LOG2; otherwise the stale max is kept for numerator and
    // denominator alike, which is exact and keeps every p <= 2^RESCALE_LOG2.
    // The decision is per row (per lane), so a row's arithmetic never depends
    // on other rows' data; the wave only skips the rescale work when no row
    // needs it (alpha = 1 exactly for the others).
    auto tile_stats = [&](f32x16 (&sc)[2], int32_t ti, int tu, bool real, float& m_cand) -> bool {
        if (KSPLIT > 1 && !real) {  // dummy tile: every score masked
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r) sc[kt][r] = -INFINITY;
        } else if (ti == j) {  // self block: token-level causal triangle
            const int kin = tu * KT, qin = p0 + col;
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int kp = kin + 32 * kt + 8 * (r >> 2) + 4 * half + (r & 3);
                    if (kp > qin) sc[kt][r] = -INFINITY;
                }
        }
        // maximum (not fmaxf): the scores are never NaN, and without NaN
        // quieting the compiler emits three-input v_maximum3 directly instead
        // of canonicalising every MFMA output first
        float mq[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};  // independent chains
#pragma unroll
        for (int r = 0; r < 16; ++r)
            mq[r & 3] = __builtin_elementwise_maximum(mq[r & 3], __builtin_elementwise_maximum(sc[0][r], sc[1][r]));
        m_cand = pair_max(__builtin_elementwise_maximum(__builtin_elementwise_maximum(mq[0], mq[1]),
                                                        __builtin_elementwise_maximum(mq[2], mq[3]))) * c_log2;
        return m_cand > m_run + RESCALE_LOG2;
    };
    auto apply_rescale = [&](bool need, float m_cand) {
        if (__any(need)) {
            const float alpha = need ? __builtin_amdgcn_exp2f(m_run - m_cand) : 1.0f;
            m_run = need ? m_cand : m_run;
            l_run *= alpha;
            l_bf *= alpha;
#pragma unroll
            for (int t = 0; t < DT; ++t)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[t][r] *= alpha;
        }
    };

    f32x16 s_a[2], s_b[2];
    score_mfma(std::integral_constant<int, 0>{}, s_a);
    {
        float mc;
        // acc and the sums are still zero: the first tile only sets the
        // running max (the rescale would multiply zeros)
        if (tile_stats(s_a, ti0, tu0, rl0, mc)) m_run = mc;
    }

    // ---- steady state --------------------------------------------------------
    // Iteration k: tile k's scores are in s_cur with its statistics applied,
    // K_k+1 and V_k are resident.
    //   phase 1: scores of tile k+1 on the matrix cores, interleaved with the
    //            exponentials of tile k and with the loads of K_k+2 (into the
    //            K buffer of tile k) and V_k+1 (into the other V buffer)
    //   phase 2: O += V_k P_k on the matrix cores, interleaved with the mask
    //            and row max of tile k+1; its (rare) rescale of O follows
    const uint32_t v_lds = lds_addr(&sm.v[0][0]);
    // One pipeline step; PAR is the buffer parity of tile k (static, so every
    // LDS read below is a lane-constant base plus an immediate offset).
    auto step = [&](auto par_c, f32x16 (&s_cur)[2], f32x16 (&s_nxt)[2]) -> bool {
        constexpr int PAR = decltype(par_c)::value;
        const bool h2 = h1 && next_own(ti2, tu2, rl2);
        // The loads of K_k+2 and V_k+1 are spread over phase 1; a tile that
        // does not exist (or a dummy) reads zeros past the end of the head
        // (no traffic).
        const uint32_t soff_k2 = tile_off(h2 && rl2, ti2, tu2);
        const uint32_t soff_v1 = tile_off(h1 && rl1, ti1, tu1);

        // phase 1: scores of tile k+1 (unused after the last tile), P of tile
        // k.  Step q issues score MFMA q, prefetches the K operand of MFMA q+KPF
        // and computes two elements of P_k (fma, exp2, sum; bf16 pack every
        // fourth step).  sched_barrier pins the order so that the vector work
        // runs in the shadow of the matrix cores.  The row sum is taken before
        // the bf16 rounding of P (so the LSE keeps fp32 accuracy).
        constexpr int NS = 2 * KS;       // score MFMAs of one tile
        constexpr int EPS = 32 / NS;     // P elements per step
        constexpr int NL = 2 * SEG_PER_WAVE;  // direct loads per wave per tile pair
        static_assert(32 % NS == 0, "P elements must split over the steps");
        // The exponentials, the bf16 packing and the DMA issue of phase 1 are
        // the longer instruction stream of the two phases: give it issue
        // priority over the other workgroup's wave on this SIMD.
        __builtin_amdgcn_s_setprio(1);
        const char* kbn = reinterpret_cast<const char*>(&sm.k[PAR ^ 1][0]);
        bf16x8 pb[4];
        float ls0 = 0.f, ls1 = 0.f;
        {
            u32x4 kop[KPF + 1];
#pragma unroll
            for (int q = 0; q < KPF; ++q)
                kop[q] = *reinterpret_cast<const u32x4*>(kbn + kofs[q >> 1] + (q & 1) * 32 * RB);
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int r = 0; r < 16; ++r) s_nxt[kt][r] = 0.f;
            f32x8 pf;
#pragma unroll
            for (int q = 0; q < NS; ++q) {
                if (q + KPF < NS)
                    kop[(q + KPF) % (KPF + 1)] = *reinterpret_cast<const u32x4*>(
                        kbn + kofs[(q + KPF) >> 1] + ((q + KPF) & 1) * 32 * RB);
                s_nxt[q & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, kop[q % (KPF + 1)]), qf[q >> 1], s_nxt[q & 1], 0, 0, 0);
#pragma unroll
                for (int e = 0; e < EPS; ++e) {
                    const int el = q * EPS + e;  // element of s_cur in P order
                    const float pv = __builtin_amdgcn_exp2f(
                        fmaf(s_cur[el >> 4][el & 15], c_log2, -m_run));
                    pf[el & 7] = pv;
                    if (e & 1) ls1 += pv; else ls0 += pv;
                }
                if (((q + 1) * EPS) % 8 == 0)
                    pb[((q + 1) * EPS) / 8 - 1] = __builtin_convertvector(pf, bf16x8);
#pragma unroll
                for (int li = (q * NL) / NS; li < ((q + 1) * NL) / NS; ++li) {
                    if (li < SEG_PER_WAVE)
                        load_lds16(k_rsrc, &sm.k[PAR][(li * NW + wave) * 64], kgo[li], soff_k2);
                    else
                        load_lds16(v_rsrc, &sm.v[PAR ^ 1][((li - SEG_PER_WAVE) * NW + wave) * 64],
                                   vgo[li - SEG_PER_WAVE], soff_v1);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        l_run += ls0 + ls1;
        {   // the bf16 weights as the PV product will see them, summed in fp32
            const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
            float lb0 = 0.f, lb1 = 0.f;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                lb0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[t][0], pb[t][1]}, ones, lb0, false);
                lb1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[t][2], pb[t][3]}, ones, lb1, false);
                lb0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[t][4], pb[t][5]}, ones, lb0, false);
                lb1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[t][6], pb[t][7]}, ones, lb1, false);
            }
            l_bf += lb0 + lb1;
        }
        __builtin_amdgcn_s_setprio(0);

        // phase 2: O^T += V^T P^T (transpose reads of V_k), interleaved with the
        // statistics of tile k+1
        bool need = false;
        float m_cand = 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const uint32_t va_base = v_lds + vofs[dt];
            u32x2 va[8];
            constexpr int VB = PAR * TILE_B;
            lds_read_tr16_x8<VB, 8 * RB>(va_base, va);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const u32x4 w = {va[2 * t][0], va[2 * t][1], va[2 * t + 1][0], va[2 * t + 1][1]};
                acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w),
                                                                  pb[t], acc[dt], 0, 0, 0);
            }
            if (dt == 0 && h1) need = tile_stats(s_nxt, ti1, tu1, rl1, m_cand);
        }
        if (h1) apply_rescale(need, m_cand);

        __builtin_amdgcn_s_waitcnt(VMCNT0);  // this wave's loads have landed
        __syncthreads();                      // ... and every other wave's
        if (!h1) return false;
        ti0 = ti1;
        tu0 = tu1;
        rl0 = rl1;
        ti1 = ti2;
        tu1 = tu2;
        rl1 = rl2;
        h1 = h2;
        return true;
    };
    while (step(std::integral_constant<int, 0>{}, s_a, s_b) &&
           step(std::integral_constant<int, 1>{}, s_b, s_a)) {
    }

    // ---- epilogue: O = acc / l_bf, LSE = (m + log2 l) ln 2 ------------------
    // O is normalised by the sum of the weights exactly as the PV product used
    // them (bf16), so the weights it applies sum to one: a row dominated by
    // one key reproduces that key's value row without the rounding error of
    // its weight (which, with the output's own bf16 rounding, could exceed
    // 2e-2 for |V| near 5).  The LSE keeps the fp32 sum, whose relative error
    // stays near 1e-7 where the bf16 sum's can reach 2^-9.
    // O goes through LDS so that the global stores are whole rows: the
    // accumulator holds, per lane, 8-byte pieces of one query row; each wave
    // writes its 32 x D tile into its own slice of the (now idle) K buffers,
    // [row][16-byte chunk ^ (row % 16)], then reads back 16 consecutive bytes
    // per lane, 16 lanes per row, and stores 4 consecutive rows per
    // instruction.  The last step's barrier ordered every LDS read of the
    // tiles before this; no other wave touches this slice.  The stores are
    // non-temporal: O is not read again here, and streaming it through L2
    // evicted K/V tiles that other workgroups were still reusing.
    if (KSPLIT > 1) {
        // Group 1 hands (m, l, l_bf, acc) of its lanes to group 0 through its
        // own (now idle) tiles and group 0's V tiles; wave w of group 1 holds
        // the same query rows, lane for lane, as wave w of group 0.  The last
        // step's barrier ordered every tile read before this.
        float* accx = reinterpret_cast<float*>(&smem[KSPLIT - 1]) + wave * (DT * 16 * 64);
        float* stx = reinterpret_cast<float*>(&smem[0].v[0][0]) + wave * (3 * 64);
        if (grp == 1) {
#pragma unroll
            for (int t = 0; t < DT; ++t)
#pragma unroll
                for (int r4 = 0; r4 < 4; ++r4) {
                    const f32x4 v4 = {acc[t][4 * r4], acc[t][4 * r4 + 1], acc[t][4 * r4 + 2],
                                      acc[t][4 * r4 + 3]};
                    *reinterpret_cast<f32x4*>(accx + ((t * 4 + r4) * 64 + lane) * 4) = v4;
                }
            stx[lane] = m_run;
            stx[64 + lane] = l_run;
            stx[128 + lane] = l_bf;
        }
        __syncthreads();
        if (grp == 1) return;
        const float m1 = stx[lane], l1 = stx[64 + lane], lb1 = stx[128 + lane];
        const float m = __builtin_elementwise_maximum(m_run, m1);
        const float a0 = __builtin_amdgcn_exp2f(m_run - m), a1 = __builtin_amdgcn_exp2f(m1 - m);
#pragma unroll
        for (int t = 0; t < DT; ++t)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const f32x4 v4 = *reinterpret_cast<const f32x4*>(accx + ((t * 4 + r4) * 64 + lane) * 4);
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[t][4 * r4 + c] = fmaf(acc[t][4 * r4 + c], a0, v4[c] * a1);
            }
        l_run = fmaf(l_run, a0, l1 * a1);
        l_bf = fmaf(l_bf, a0, lb1 * a1);
        m_run = m;
    }
    const float l_tot = pair_sum(l_run);
    const float inv = 1.f / pair_sum(l_bf);
    constexpr int OCH = D / 8;                 // 16-byte chunks per row
    char* oslice = reinterpret_cast<char*>(&sm.k[0][0]) + wave * 32 * RB;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int gq4 = 0; gq4 < 4; ++gq4) {
            f32x4 v4;
#pragma unroll
            for (int c = 0; c < 4; ++c) v4[c] = acc[dt][4 * gq4 + c] * inv;
            const int ch = (4 * dt + gq4) ^ (col % OCH);
            *reinterpret_cast<bf16x4*>(oslice + col * RB + ch * 16 + half * 8) =
                __builtin_convertvector(v4, bf16x4);
        }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's O tile is in LDS
    {
        const int32_t row0 = j * BW + p0;  // first query of this wave
        __bf16* Obase = O + (((int64_t)beta * Hq + head) * (int64_t)n + row0) * D;
        constexpr int RPI = 64 / OCH;      // rows per store instruction
#pragma unroll
        for (int it = 0; it < 32 / RPI; ++it) {
            const int r = it * RPI + lane / OCH, c = lane % OCH;
            const u32x4 w = *reinterpret_cast<const u32x4*>(oslice + r * RB + ((c ^ (r % OCH)) * 16));
            if (row0 + r < n) __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(Obase + (int64_t)r * D + c * 8));
        }
    }
    if (LSE != nullptr && half == 0 && qvalid)
        LSE[((int64_t)beta * Hq + head) * (int64_t)n + qpos] = (m_run + log2f(l_tot)) * LN2;
}

// Two key groups per workgroup: never (mode 1), always (mode 2), or (mode 0,
// automatic) when the launch has at most one work item per compute unit and
// its routes average at least 8 key tiles per item.  Measured on MI355X: the
// dense comparator gains 4-11% at 1K-4K tokens, while BF1 routes at those
// lengths (3-7 tiles per item) lose 0-11%, their time being set by fixed
// per-item latencies rather than by the chain of tiles.
bool use_key_split(int mode, int64_t items, int64_t tiles) {
    if (mode == 1) return false;
    if (mode == 2) return true;
    if (tiles < 8 * items) return false;
    static std::mutex mu;
    static std::map<int, int> cus;  // device -> compute units
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return false;
    int cu = 0;
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = cus.find(dev);
        if (it == cus.end()) {
            if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) cu = 0;
            cus.emplace(dev, cu);
        } else {
            cu = it->second;
        }
    }
    return cu > 0 && items <= cu;
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
    // key tiles the launch walks (the dense route {0..j} has NB (NB + 1) / 2
    // blocks per kv-head; a caller table is taken at its size)
    const int64_t blocks = DENSE ? (int64_t)NB * (NB + 1) / 2 : a.nnz;
    const int64_t tiles = blocks * (BW / KT) * a.batch * a.Hkv * NCHUNK;
    if (use_key_split(a.key_split, items, tiles)) {
        hipLaunchKernelGGL((attn_fwd_kernel<D, G, BW, NW, DENSE, 2>), dim3((unsigned)items),
                           dim3(2 * NW * 64), 0, stream, (const __bf16*)a.Q, (const __bf16*)a.K,
                           (const __bf16*)a.V, (__bf16*)a.O, a.LSE, a.row_ptr, a.col_idx, a.nnz,
                           (int32_t)a.n, NB, a.batch * a.Hkv, a.Hkv, c_log2);
    } else {
        hipLaunchKernelGGL((attn_fwd_kernel<D, G, BW, NW, DENSE, 1>), dim3((unsigned)items),
                           dim3(NW * 64), 0, stream, (const __bf16*)a.Q, (const __bf16*)a.K,
                           (const __bf16*)a.V, (__bf16*)a.O, a.LSE, a.row_ptr, a.col_idx, a.nnz,
                           (int32_t)a.n, NB, a.batch * a.Hkv, a.Hkv, c_log2);
    }
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

// ---------------------------------------------------------------------------
// Fixed scratch of the forward that allocates nothing
// ---------------------------------------------------------------------------
// The route table of bf1_attn_fwd_noalloc (row_ptr, then col_idx right after
// it) lives in this array; each device holds its own copy for the life of the
// process.  In host code the name is a stand-in for the symbol, never a
// device address: the address of a device's copy comes from
// hipGetSymbolAddress, taken once per device with that device current, and
// only that address is handed to kernels.
static __device__ __align__(256) int32_t scratch[kNoallocInts];

}  // namespace

hipError_t noalloc_scratch(int32_t** ptr) {
    static std::mutex mu;
    static std::map<int, int32_t*> addr;  // device -> address of its copy
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(mu);
    auto it = addr.find(dev);
    if (it == addr.end()) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        it = addr.emplace(dev, static_cast<int32_t*>(p)).first;
    }
    *ptr = it->second;
    return hipSuccess;
}

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
