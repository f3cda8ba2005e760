// BF1 causal dyadic block-sparse attention: backward kernels for gfx950
// (head_dim 64 and 128).  Gradients of O = softmax_mask(c Q K^T) V with respect to Q,
// K and V for an upstream gradient dO, on the route of the paper's §3.1
// (Eq. 1), with P recomputed from the forward's log-sum-exp:
//     P = exp(c S - LSE),  D = rowsum(dO * O),  dP = dO V^T,  dS = P * (dP - D),
//     dQ = c dS K,  dK = c dS^T Q,  dV = P^T dO   (summed over a GQA group).
//
// Kernels, in launch order:
//  * bwd_delta_kernel -- D and LSE log2 e of every query row.
//  * bwd_dkdv_kernel -- one workgroup per (batch, kv-head, 64-key tile,
//    segment of the tile's query-block list), walking the TRANSPOSED route
//    (the query blocks that select the key block); two waves accumulate dV
//    and two dK in registers, and the dS it forms is written to the workspace
//    for dQ.  Key block 0 is selected by every query block, so long lists
//    are cut into segments whose partial sums go to a workspace.
//  * bwd_reduce_kernel -- sums the segment partials of such tiles in a fixed
//    order (deterministic) into dK and dV.
//  * bwd_dq_kernel   -- one workgroup per (batch, kv-head, query block, row
//    chunk), walking the forward route like the forward kernel: dQ from the
//    stored dS and the K tiles (no score is recomputed).
//
// Tiles in LDS keep the natural [row][d] order in 16-byte chunks; chunk c of
// row r sits at c ^ bswz(r) (for d = 128, bswz(r) = 4 (r mod 4) + (r/4 mod 4);
// d = 64 has its own, below).  This one layout is conflict-free for both ways the backward reads a tile: 16 bytes
// of one row per lane (an MFMA operand with k along d) and the LDS transpose
// load (an operand with k along the rows).  Matrix-core layouts follow the
// forward (v_mfma_f32_32x32x16_bf16; accumulator lane l, register r holds
// row 8(r/4) + 4(l/32) + r%4, column l%32).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bf1_device.h"
#include "bf1_kernels.h"
#include "bf1_route.h"

namespace bf1 {
namespace {

// head_dim D of a backward instance: bytes per bf16 row, per 64-row tile,
// MFMA k-steps along d, 32-wide d tiles, 16-byte chunks per row
#define BWD_GEOMETRY(D)                                                     \
    constexpr int BD = (D), BRB = 2 * (D), BTILE = KT * BRB, BKS = (D) / 16, \
                  BDT = (D) / 32;                                           \
    (void)BD; (void)BRB; (void)BTILE; (void)BKS; (void)BDT

// Physical chunk swizzle of row `row`: chunk c of the row sits at c ^ bswz.
// Chosen (by simulating the 64 banks) so that both reads of a tile are
// conflict-free: 16 lanes reading 16 bytes of 16 consecutive rows (the
// row-wise operand), and 32 lanes of the transpose load reading 8 bytes each.
template <int D>
__device__ __forceinline__ int bswz(int row) {
    if constexpr (D == 128) return 4 * (row & 3) + ((row >> 2) & 3);
    else return (((row >> 1) & 1) << 2) | (((row >> 3) & 1) << 1) | ((row >> 2) & 1);
}

// Byte offset, inside a tile, of the 16 bytes lane `lane` moves in the direct
// load of 1 KB segment `seg` (1024 / (2 D) rows, lane order = physical).
template <int D>
__device__ __forceinline__ uint32_t seg_off(int seg, int lane) {
    constexpr int CH = D / 8;
    const int row = seg * (64 / CH) + lane / CH, pc = lane % CH;
    return (uint32_t)(row * 2 * D + ((pc ^ bswz<D>(row)) << 4));
}
// Row-wise operand read: 16 bytes of `row`, logical chunk c.
template <int D>
__device__ __forceinline__ int rw_off(int row, int c) { return row * 2 * D + ((c ^ bswz<D>(row)) << 4); }
// Transpose-read base of lane `lane` for d-tile dt, second read of a pair h2
// (rows +8); a 16-row group g adds 16 g rows (bswz is unchanged by it).
template <int D>
__device__ __forceinline__ int tr_off(int lane, int dt, int h2) {
    const int gq = lane >> 4, kk = lane & 15;
    const int row = 4 * (gq >> 1) + (kk >> 2) + 8 * h2;
    const int lb = 32 * (2 * dt + (gq & 1)) + 8 * (kk & 3);
    return row * 2 * D + (((lb >> 4) ^ bswz<D>(row)) << 4) + (lb & 15);
}

__device__ __forceinline__ float dot_bf16x8(u32x4 a, u32x4 b) {
    const bf16x8 x = __builtin_bit_cast(bf16x8, a), y = __builtin_bit_cast(bf16x8, b);
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) s = fmaf((float)x[e], (float)y[e], s);
    return s;
}

// ---------------------------------------------------------------------------
// dS units
// ---------------------------------------------------------------------------
// The dK/dV kernel forms dS = P (dP - D) of every selected (64-row query tile,
// 64-key tile, q-head) and writes it, bf16, to the workspace for the dQ
// kernel: one 8 KB unit per triple, unit index
//   (((batch x kv-head, transposed-route entry), query sub-tile), key sub-tile), head in group.
// A unit is stored in the dQ kernel's MFMA operand order: 16-byte piece
// (rh, t, lane) at ((4 rh + t) 64 + lane) 16 holds, for query 32 rh + lane % 32,
// the keys 16 t + 4 h + {0..3} and 16 t + 8 + 4 h + {0..3} (h = lane / 32):
// the B operand of k-step t of dQ^T += K^T dS^T, loaded straight into registers.
constexpr int DS_UNIT = KT * KT * 2;  // bytes per unit
typedef __attribute__((address_space(3))) u32x2 lds_u32x2;

// ---------------------------------------------------------------------------
// D and LSE log2 e
// ---------------------------------------------------------------------------
// D = rowsum(dO * O) of every query row (fp32, summed over the row's D / 8
// lanes by butterfly shuffles) and LSE * log2 e beside it, for the dK/dV
// kernel.  One lane per 16 bytes of a row.
template <int D>
__global__ __launch_bounds__(256) void bwd_delta_kernel(const __bf16* __restrict__ O, const __bf16* __restrict__ dO,
                                                        const float* __restrict__ LSE, float* __restrict__ Delta,
                                                        float* __restrict__ Lse2, int64_t rows) {
    constexpr int LPR = D / 8;  // lanes per row
    constexpr int RPB = 256 / LPR;
    const int64_t row = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
    const int c = threadIdx.x % LPR;
    float s = 0.f;
    if (row < rows) {
        // read once here (the dK/dV kernel re-reads dO tiles much later)
        const u32x4 wo = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(O + row * D) + c);
        const u32x4 wd = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(dO + row * D) + c);
        s = dot_bf16x8(wd, wo);
    }
#pragma unroll
    for (int m = LPR / 2; m > 0; m >>= 1) s += __shfl_xor(s, m);
    if (row < rows && c == 0) {
        Delta[row] = s;
        Lse2[row] = LSE[row] * LOG2E;
    }
}

// ---------------------------------------------------------------------------
// dQ
// ---------------------------------------------------------------------------
// Workgroup = 4 waves x 32 stacked query rows (like the forward), walking the
// forward route.  dS comes from the dK/dV kernel's units, so nothing is
// recomputed: per 64-key tile the workgroup stages the K tile in LDS
// (buffer->LDS DMA, double-buffered, one barrier per tile), each wave loads
// its rows' dS^T operands from the unit straight into registers, and
// accumulates dQ^T += K^T dS^T (A: transpose reads of the K tile).  Both loads
// of tile k+1 are issued before the MFMAs of tile k.  32 KB of LDS and ~120
// registers give four workgroups per CU, which together keep enough loads in
// flight to cover the HBM latency of the dS units (each is read once).
template <int D, int G, int BW>
__global__ __launch_bounds__(256, 4) void bwd_dq_kernel(
    const __bf16* __restrict__ K, const __bf16* __restrict__ dS, float* __restrict__ dQ,
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx, int64_t nnz,
    const int32_t* __restrict__ uoffs, int64_t nusers, int32_t n, int32_t NB, int32_t L,
    int32_t batch_hkv, int32_t Hkv, float scale) {
    BWD_GEOMETRY(D);
    constexpr int NW = 4, ROWS = 128;
    constexpr int NCHUNK = (G * BW) / ROWS;
    constexpr int NSUB = BW / KT;
    constexpr int SPW = (BTILE / 1024) / NW;  // K segments per wave per tile
    static_assert(NCHUNK * ROWS == G * BW, "rows must tile the stacked group");
    // K tiles (two buffers); the epilogue reuses the space as four 8 KB slices
    constexpr int LDS_BYTES = 2 * BTILE > 32768 ? 2 * BTILE : 32768;
    __shared__ u32x4 lds[LDS_BYTES / 16];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 31;
    const int half = lane >> 5;

    const int32_t x = blockIdx.x;
    const int chunk = x % NCHUNK;
    const int32_t y = x / NCHUNK;
    const int32_t bh = y % batch_hkv;
    const int32_t j = NB - 1 - y / batch_hkv;
    const int32_t beta = bh / Hkv;
    const int32_t g = bh % Hkv;
    const int Hq = Hkv * G;

    const int srow = chunk * ROWS + wave * 32;
    const int head = g * G + srow / BW;
    const int qin = srow % BW + col;  // query position inside block j
    const int32_t qpos = j * BW + qin;
    const int64_t qrow = ((int64_t)beta * Hq + head) * (int64_t)n + qpos;
    // dS unit of this wave's rows: head in the group, query sub-tile; the
    // wave's 32 rows are half rh_w of the unit
    const int rh_w = (srow % KT) / 32;
    const int u_hh = srow / BW, u_qs = (srow % BW) / KT;

    // ---- route walk (as in the forward) -------------------------------------------
    int64_t e0 = row_ptr[j], e1 = row_ptr[j + 1];
    e0 = e0 < 0 ? 0 : (e0 > nnz ? nnz : e0);
    e1 = e1 < e0 ? e0 : (e1 > nnz ? nnz : e1);
    int32_t cur_p = (int32_t)e0;
    const int32_t pos_end = (int32_t)e1;
    int cur_u = 0;
    auto next_tile = [&](int32_t& ti, int& tu) -> bool {
        while (cur_p < pos_end) {
            const int32_t i = col_idx[cur_p];
            if (i >= 0 && i <= j) {
                for (; cur_u < NSUB; ++cur_u)
                    if (i * BW + cur_u * KT < n) {
                        ti = i;
                        tu = cur_u++;
                        if (cur_u >= NSUB) {
                            ++cur_p;
                            cur_u = 0;
                        }
                        return true;
                    }
            }
            ++cur_p;
            cur_u = 0;
        }
        return false;
    };

    const __amdgpu_buffer_rsrc_t k_rsrc =
        head_rsrc(K + ((int64_t)beta * Hkv + g) * (int64_t)n * BD, (uint32_t)n * BRB);
    // dS operands of tile (ti, tu) into registers, then its K tile into LDS
    auto stage = [&](int buf, int32_t ti, int tu, u32x4 (&dsr)[4]) {
        const int32_t tiu = __builtin_amdgcn_readfirstlane(ti), tuu = __builtin_amdgcn_readfirstlane(tu);
        const int64_t et = (int64_t)__builtin_amdgcn_readfirstlane(uoffs[tiu]) + route_user_rank(L, tiu, j);
        const int64_t ui = ((((int64_t)bh * nusers + et) * NSUB + u_qs) * NSUB + tuu) * G + u_hh;
        const u32x4* src = reinterpret_cast<const u32x4*>(dS + ui * (DS_UNIT / 2)) + 4 * 64 * rh_w + lane;
#pragma unroll
        for (int t = 0; t < 4; ++t) dsr[t] = __builtin_nontemporal_load(src + 64 * t);
        const uint32_t soff = (uint32_t)(tiu * BW + tuu * KT) * BRB;
#pragma unroll
        for (int it = 0; it < SPW; ++it) {
            const int seg = it * NW + wave;
            load_lds_async<16>(k_rsrc, &lds[buf * (BTILE / 16) + seg * 64], seg_off<D>(seg, lane), soff);
        }
    };

    f32x16 acc[BDT];
#pragma unroll
    for (int t = 0; t < BDT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;

    int32_t ti = 0, tn = 0;
    int tu = 0, tnu = 0;
    u32x4 dcur[4], dnext[4];
    bool have = next_tile(ti, tu);
    if (have) stage(0, ti, tu, dcur);
    __builtin_amdgcn_s_waitcnt(VMCNT0);
    __syncthreads();
    int buf = 0;
    while (have) {
        const bool hn = next_tile(tn, tnu);
        if (hn) stage(buf ^ 1, tn, tnu, dnext);

        const uint32_t kl = lds_addr(&lds[0]) + buf * BTILE;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const bf16x8 db = __builtin_bit_cast(bf16x8, dcur[t]);
#pragma unroll
            for (int dt = 0; dt < BDT; ++dt) {
                const u32x2 alo = lds_read_tr16(kl + tr_off<D>(lane, dt, 0) + 16 * t * BRB);
                const u32x2 ahi = lds_read_tr16(kl + tr_off<D>(lane, dt, 1) + 16 * t * BRB);
                const u32x4 w = {alo[0], alo[1], ahi[0], ahi[1]};
                acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, w), db, acc[dt], 0, 0, 0);
            }
        }
        __builtin_amdgcn_s_waitcnt(VMCNT0);  // this wave's loads of the next tile have landed
        __syncthreads();                      // ... and every other wave's; this tile is free
#pragma unroll
        for (int t = 0; t < 4; ++t) dcur[t] = dnext[t];
        ti = tn;
        tu = tnu;
        have = hn;
        buf ^= 1;
    }
    __builtin_amdgcn_s_waitcnt(VMCNT0);

    // ---- dQ = c dS K, staged through an 8 KB LDS slice per wave, 64 columns at a
    // time, into half-row (256-byte) stores; rows past n skipped ----
    {
        char* slice = reinterpret_cast<char*>(&lds[0]) + wave * 8192;
        const int64_t row0 = qrow - col;  // first row of this wave
#pragma unroll
        for (int rd = 0; rd < BDT / 2; ++rd) {
#pragma unroll
            for (int dd = 0; dd < 2; ++dd)
#pragma unroll
                for (int gq4 = 0; gq4 < 4; ++gq4) {
                    f32x4 v4;
#pragma unroll
                    for (int c = 0; c < 4; ++c) v4[c] = acc[2 * rd + dd][4 * gq4 + c] * scale;
                    const int ch = (8 * dd + 2 * gq4 + half) ^ (col & 15);
                    *reinterpret_cast<f32x4*>(slice + col * 256 + ch * 16) = v4;
                }
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): these 64 columns are in LDS
#pragma unroll
            for (int it = 0; it < 8; ++it) {
                const int r = it * 4 + lane / 16, c = lane % 16;
                const f32x4 w = *reinterpret_cast<const f32x4*>(slice + r * 256 + ((c ^ (r & 15)) * 16));
                if (qpos - col + r < n)
                    __builtin_nontemporal_store(w, reinterpret_cast<f32x4*>(dQ + (row0 + r) * BD + 64 * rd + c * 4));
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);  // read back before the next columns overwrite it
        }
    }
}

// ---------------------------------------------------------------------------
// dK, dV
// ---------------------------------------------------------------------------
// Workgroup = 4 waves over one 64-key tile (block i, sub-tile u).  Waves 0
// and 1 ("P waves") own keys 0..31 and 32..63 for S, P and dV and hold their
// K^T as MFMA B operands in registers; waves 2 and 3 ("dS waves") own the same
// keys for dP, dS and dK and hold their V^T.  The workgroup walks query tiles
// (64 rows of one q-head of a query block j that selects block i), staged in
// LDS: Q and dO rows, LSE log2 e and D.  Per 32-row half of a query tile:
//   phase 1: S = Q K^T (P waves) or dP = dO V^T (dS waves)  (A: row-wise reads)
//            P waves: P = exp2(c log2e S - log2e LSE), to LDS (fp32)
//   phase 2: dS waves read P; dS = P (dP - D)                (lane = key column)
//   phase 3: dV += P^T dO (P waves) or dK += dS^T Q (dS waves)
//            (A: P / dS packed from the lane's own registers; B: transpose reads)
// The dS waves also write each half's dS (bf16, the values their dK MFMAs
// use) to the tile's dS unit, transposed through a 2 KB LDS scratch per wave
// into the dQ kernel's operand order.
// Splitting the roles halves each wave's registers (no accumulator leaves the
// VGPRs) and gives two workgroups, two waves per SIMD, per CU.  Two barriers
// per half order the exchange of P.  A segment descriptor (int32 x 8): key
// block, sub-tile, first entry of its query-block list in the transposed
// table, entry count, partial slot (-1: write dK/dV directly).
template <int D, int G, int BW>
__global__ __launch_bounds__(256, 2) void bwd_dkdv_kernel(
    const __bf16* __restrict__ Q, const __bf16* __restrict__ K, const __bf16* __restrict__ V,
    const __bf16* __restrict__ dO, const float* __restrict__ Lse2, const float* __restrict__ Delta,
    float* __restrict__ dK, float* __restrict__ dV, float* __restrict__ part, __bf16* __restrict__ dSw,
    const int32_t* __restrict__ segs, const int32_t* __restrict__ users, int32_t nslots, int64_t nusers,
    int32_t n, int32_t batch_hkv, int32_t Hkv, float c_log2, float scale) {
    BWD_GEOMETRY(D);
    constexpr int NW = 4;
    constexpr int NSUB = BW / KT;
    constexpr int SPW = (BTILE / 1024) / NW;  // Q (or dO) segments per wave per tile
    static_assert(SPW * NW * 1024 == BTILE, "segments must split over the waves");

    __shared__ u32x4 q_s[2][BTILE / 16];
    __shared__ u32x4 o_s[2][BTILE / 16];
    __shared__ float lse_s[2][KT];
    __shared__ float del_s[2][KT];
    __shared__ f32x4 p_x[2][4][64];  // P of the current half: [key half][row group][lane]
    __shared__ u32x2 dsx[2][32 * 8];  // dS transpose scratch of the dS waves: [key half][key][8-byte chunk]

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kw = wave & 1;   // key half of the tile
    const bool pw = wave < 2;  // P wave (S, P, dV) or dS wave (dP, dS, dK)
    const int col = lane & 31;
    const int half = lane >> 5;

    const int32_t x = blockIdx.x;
    const int32_t bh = x % batch_hkv;
    const int32_t* sd = segs + 8 * (x / batch_hkv);
    const int32_t i = sd[0];
    const int u = sd[1];
    const int32_t uoff = sd[2];
    const int32_t ucnt = sd[3];
    const int32_t slot = sd[4];
    const int32_t beta = bh / Hkv;
    const int32_t g = bh % Hkv;
    const int Hq = Hkv * G;

    const int kin = u * KT + 32 * kw + col;  // key position inside block i of this lane's column
    // transpose-read offsets in the dS scratch: for 16-key step tp, lane (gq, l16)
    // reads the 8-byte run of queries 16 (gq & 1) + 4 (l16 & 3) of key
    // 16 tp + 4 (gq >> 1) + l16 / 4 (+8 for the second read)
    int xoff[2][2];
    {
        const int gq = lane >> 4, l16 = lane & 15;
        const int c8 = 4 * (gq & 1) + (l16 & 3);
#pragma unroll
        for (int tp = 0; tp < 2; ++tp)
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                const int key = 16 * tp + 4 * (gq >> 1) + (l16 >> 2) + 8 * h2;
                xoff[tp][h2] = key * 64 + ((c8 ^ (key >> 2)) & 7) * 8;
            }
    }
    const int32_t kpos = i * BW + kin;
    const int64_t kvrow0 = ((int64_t)beta * Hkv + g) * (int64_t)n;

    // ---- K^T (P waves) or V^T (dS waves) of this wave's 32 keys, zero past n -------
    bf16x8 bop[BKS];
    {
        const u32x4* src = reinterpret_cast<const u32x4*>((pw ? K : V) + (kvrow0 + kpos) * BD);
#pragma unroll
        for (int s = 0; s < BKS; ++s) {
            u32x4 w = {0u, 0u, 0u, 0u};
            if (kpos < n) w = src[2 * s + half];
            bop[s] = __builtin_bit_cast(bf16x8, w);
        }
    }

    // Query tile t of this segment: entry t / (G NSUB) of the list, q-head
    // t / NSUB % G of the group, sub-tile t % NSUB of the query block.
    const int32_t ntiles = ucnt * G * NSUB;
    auto stage = [&](int buf, int32_t t) {
        const int32_t jq = users[uoff + t / (G * NSUB)];
        const int h = g * G + (t / NSUB) % G;
        const int32_t row0 = jq * BW + (t % NSUB) * KT;
        const int64_t qr0 = ((int64_t)beta * Hq + h) * (int64_t)n;
        const __amdgpu_buffer_rsrc_t qr = head_rsrc(Q + qr0 * BD, (uint32_t)n * BRB);
        const __amdgpu_buffer_rsrc_t orr = head_rsrc(dO + qr0 * BD, (uint32_t)n * BRB);
        const uint32_t soff = (uint32_t)row0 * BRB;
#pragma unroll
        for (int it = 0; it < SPW; ++it) {
            const int seg = it * NW + wave;
            load_lds_async<16>(qr, &q_s[buf][seg * 64], seg_off<D>(seg, lane), soff);
            load_lds_async<16>(orr, &o_s[buf][seg * 64], seg_off<D>(seg, lane), soff);
        }
        // 64 rows of LSE log2 e (wave 0) or D (wave 1), 4 bytes per lane
        if (wave < 2) {
            const float* src = (wave == 0 ? Lse2 : Delta) + qr0;
            float* dst = wave == 0 ? &lse_s[buf][0] : &del_s[buf][0];
            load_lds_async<4>(head_rsrc(src, (uint32_t)n * 4), dst, (uint32_t)lane * 4, (uint32_t)row0 * 4);
        }
    };
    auto tile_query_block = [&](int32_t t) -> int32_t { return users[uoff + t / (G * NSUB)]; };

    f32x16 acc[BDT];  // dV (P waves) or dK / scale (dS waves)
#pragma unroll
    for (int t = 0; t < BDT; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[t][r] = 0.f;

    if (ntiles > 0) stage(0, 0);
    __builtin_amdgcn_s_waitcnt(VMCNT0);
    __syncthreads();
    const f32x16 zero = {};
    for (int32_t t = 0, buf = 0; t < ntiles; ++t, buf ^= 1) {
        if (t + 1 < ntiles) stage(buf ^ 1, t + 1);
        const int32_t jq = tile_query_block(t);
        const bool self = jq == i;
        const int qsub = (t % NSUB) * KT;  // query position of tile row 0 inside block jq
        // this tile's dS unit (dS waves write it for the dQ kernel)
        char* dsu = reinterpret_cast<char*>(dSw) +
                    (((((int64_t)bh * nusers + uoff + t / (G * NSUB)) * NSUB + t % NSUB) * NSUB + u) * G +
                     (t / NSUB) % G) * DS_UNIT;
        // phase-1 rows (Q for S, dO for dP); phase-3 transposed tile (dO for dV, Q for dK)
        const char* ab = reinterpret_cast<const char*>(pw ? &q_s[buf][0] : &o_s[buf][0]);
        const uint32_t tl = lds_addr(pw ? &o_s[buf][0] : &q_s[buf][0]);
        const float* rvs = pw ? &lse_s[buf][0] : &del_s[buf][0];
#pragma unroll
        for (int rh = 0; rh < 2; ++rh) {
            // ---- phase 1: operand rows of this half issued as one group ahead of
            // the MFMAs (left to itself the compiler serialises read, wait, MFMA)
            u32x4 opa[BKS];
#pragma unroll
            for (int ks = 0; ks < BKS; ++ks)
                opa[ks] = *reinterpret_cast<const u32x4*>(ab + rw_off<D>(32 * rh + col, 2 * ks + half));
            f32x4 rv[4];  // LSE log2 e (P waves) or D (dS waves) of the lane's rows
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4)
                rv[g4] = *reinterpret_cast<const f32x4*>(rvs + 32 * rh + 8 * g4 + 4 * half);
            __builtin_amdgcn_sched_barrier(0);
            f32x16 sc;
#pragma unroll
            for (int ks = 0; ks < BKS; ++ks)
                sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, opa[ks]), bop[ks],
                                                             ks == 0 ? zero : sc, 0, 0, 0);
            // rows of this lane: 32 rh + 8 g4 + 4 half + c
            bf16x8 pk2[2];
            if (pw) {
                float pr[16];
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4)
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        pr[4 * g4 + c] = __builtin_amdgcn_exp2f(fmaf(sc[4 * g4 + c], c_log2, -rv[g4][c]));
                if (self) {  // the key-block-diagonal tile: token-level causal mask
#pragma unroll
                    for (int g4 = 0; g4 < 4; ++g4)
#pragma unroll
                        for (int c = 0; c < 4; ++c)
                            if (kin > qsub + 32 * rh + 8 * g4 + 4 * half + c) pr[4 * g4 + c] = 0.f;
                }
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4)
                    p_x[kw][g4][lane] = f32x4{pr[4 * g4], pr[4 * g4 + 1], pr[4 * g4 + 2], pr[4 * g4 + 3]};
#pragma unroll
                for (int r = 0; r < 16; ++r) pk2[r >> 3][r & 7] = (__bf16)pr[r];
            }
            __syncthreads();  // P of this half is in LDS
            // ---- phase 2: the dS waves take P
            f32x4 pp[4];
            if (!pw) {
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4) pp[g4] = p_x[kw][g4][lane];
            }
            __syncthreads();  // ... and has been read: the exchange buffer is free again
            if (!pw) {
#pragma unroll
                for (int g4 = 0; g4 < 4; ++g4)
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const int r = 4 * g4 + c;
                        pk2[r >> 3][r & 7] = (__bf16)(pp[g4][c] * (sc[r] - rv[g4][c]));
                    }
                // dS of this half to the workspace in the dQ kernel's operand order:
                // transposed (key rows -> query lanes) through the wave's 2 KB
                // scratch, 8-byte chunk c8 of row k at c8 ^ (k / 4) (conflict-free)
                const uint32_t xb = lds_addr(&dsx[0][0]) + kw * 2048;
#pragma unroll
                for (int m = 0; m < 2; ++m) {
                    const u32x4 w = __builtin_bit_cast(u32x4, pk2[m]);
#pragma unroll
                    for (int sec = 0; sec < 2; ++sec) {
                        const int c8 = 4 * m + 2 * sec + half;  // queries 16 m + 8 sec + 4 half + 0..3
                        *reinterpret_cast<lds_u32x2*>(static_cast<uintptr_t>(xb + col * 64 + ((c8 ^ (col >> 2)) & 7) * 8)) =
                            u32x2{w[2 * sec], w[2 * sec + 1]};
                    }
                }
                __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
#pragma unroll
                for (int tp = 0; tp < 2; ++tp) {
                    const u32x2 lo = lds_read_tr16(xb + xoff[tp][0]);
                    const u32x2 hi = lds_read_tr16(xb + xoff[tp][1]);
                    __builtin_nontemporal_store(u32x4{lo[0], lo[1], hi[0], hi[1]},
                                                reinterpret_cast<u32x4*>(dsu + ((4 * rh + 2 * kw + tp) * 64 + lane) * 16));
                }
            }
            // ---- phase 3: transpose reads of dO (P waves) or Q (dS waves), as one group
            u32x4 wt[BDT][2];
#pragma unroll
            for (int dt = 0; dt < BDT; ++dt)
#pragma unroll
                for (int m = 0; m < 2; ++m) {
                    const int go = 16 * (2 * rh + m) * BRB;
                    const u32x2 lo = lds_read_tr16(tl + tr_off<D>(lane, dt, 0) + go);
                    const u32x2 hi = lds_read_tr16(tl + tr_off<D>(lane, dt, 1) + go);
                    wt[dt][m] = u32x4{lo[0], lo[1], hi[0], hi[1]};
                }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int dt = 0; dt < BDT; ++dt)
                    acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pk2[m], __builtin_bit_cast(bf16x8, wt[dt][m]),
                                                                      acc[dt], 0, 0, 0);
        }
        __builtin_amdgcn_s_waitcnt(VMCNT0);  // this wave's loads of the next tile have landed
        __syncthreads();                      // ... and the other waves'; this tile is free
    }
    __builtin_amdgcn_s_waitcnt(VMCNT0);

    // ---- store: lane holds d column 32 dt + col, keys 8(r/4) + 4 half + r%4 ---------
    // dV (P waves) or dK (dS waves) directly (keys past n skipped), staged through
    // the idle query-tile buffers into whole-row non-temporal stores, or into the
    // segment's partial slot.
    const float osc = pw ? 1.f : scale;
    if (slot < 0) {
        constexpr int QCH = BD / 4;  // 16-byte chunks per fp32 row
        char* st = reinterpret_cast<char*>(wave < 2 ? &q_s[wave][0] : &o_s[wave - 2][0]);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int kl = 8 * (r >> 2) + 4 * half + (r & 3);  // key inside the wave's 32
#pragma unroll
            for (int dt = 0; dt < BDT; ++dt) {
                const int off = kl * (BD * 4) + (((8 * dt + (col >> 2)) ^ (kl & 15)) * 16) + (col & 3) * 4;
                *reinterpret_cast<float*>(st + off) = acc[dt][r] * osc;
            }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's tile is in LDS
        float* out = pw ? dV : dK;
        constexpr int RPI = 64 / QCH;         // rows per store instruction
#pragma unroll
        for (int it = 0; it < 32 / RPI; ++it) {
            const int r = it * RPI + lane / QCH, c = lane % QCH;
            const f32x4 w = *reinterpret_cast<const f32x4*>(st + r * (BD * 4) + ((c ^ (r & 15)) * 16));
            const int32_t kp = i * BW + u * KT + 32 * kw + r;
            if (kp < n) __builtin_nontemporal_store(w, reinterpret_cast<f32x4*>(out + (kvrow0 + kp) * BD + c * 4));
        }
        return;
    }
    float* dst = part + (((int64_t)bh * nslots + slot) * 2 + (pw ? 1 : 0)) * (KT * BD);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int key = 32 * kw + 8 * (r >> 2) + 4 * half + (r & 3);  // inside the 64-key tile
#pragma unroll
        for (int dt = 0; dt < BDT; ++dt) dst[key * BD + 32 * dt + col] = acc[dt][r] * osc;
    }
}

// Sum of the partial slots of split key tiles: reduce descriptor (int32 x 4) =
// key block, sub-tile, first slot, slot count.  Fixed summation order.  One
// workgroup per (descriptor, batch x kv-head, 256-element chunk of the 64 x D
// tile); each thread sums one element of dK and of dV over the slots.
constexpr int RED_CHUNK = 256;
template <int D, int BW>
__global__ __launch_bounds__(256) void bwd_reduce_kernel(
    float* __restrict__ dK, float* __restrict__ dV, const float* __restrict__ part,
    const int32_t* __restrict__ reds, int32_t nslots, int32_t n, int32_t batch_hkv) {
    BWD_GEOMETRY(D);
    constexpr int NCH = KT * BD / RED_CHUNK;
    constexpr int64_t SLOT = 2 * KT * BD;  // floats per slot (dK tile, then dV tile)
    const int32_t x = blockIdx.x;
    const int ch = x % NCH;
    const int32_t bh = (x / NCH) % batch_hkv;
    const int32_t* rd = reds + 4 * (x / NCH / batch_hkv);
    const int32_t i = rd[0], u = rd[1], s0 = rd[2], ns = rd[3];
    const int64_t kvrow0 = (int64_t)bh * n;
    const int e = ch * RED_CHUNK + threadIdx.x;  // element of the 64 x D tile
    const int key = e / BD, d = e % BD;
    const int32_t kp = i * BW + u * KT + key;
    const float* pk = part + ((int64_t)bh * nslots + s0) * SLOT + e;
    // slots summed in order; eight slots' loads are issued before their sums
    float sk = 0.f, sv = 0.f;
    int32_t s = 0;
    for (; s + 8 <= ns; s += 8) {
        float kk[8], vv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            kk[q] = pk[(s + q) * SLOT];
            vv[q] = pk[(s + q) * SLOT + KT * BD];
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            sk += kk[q];
            sv += vv[q];
        }
    }
    for (; s < ns; ++s) {
        sk += pk[s * SLOT];
        sv += pk[s * SLOT + KT * BD];
    }
    if (kp < n) {
        dK[(kvrow0 + kp) * BD + d] = sk;
        dV[(kvrow0 + kp) * BD + d] = sv;
    }
}

template <int D, int G, int BW>
hipError_t launch_bwd_g(const BwdArgs& a, hipStream_t stream) {
    BWD_GEOMETRY(D);
    constexpr int NCHUNK = (G * BW) / 128;
    const int32_t NB = (int32_t)((a.n + BW - 1) / BW);
    const int32_t bhk = a.batch * a.Hkv;
    const int64_t items = (int64_t)NB * bhk * NCHUNK;
    const int64_t rows = (int64_t)a.batch * a.Hq * a.n;
    const int64_t dgrid = (rows + 256 / (D / 8) - 1) / (256 / (D / 8));
    if (items > 0x7fffffff || dgrid > 0x7fffffff || (int64_t)a.nseg * bhk > 0x7fffffff ||
        (int64_t)a.nred * bhk > 0x7fffffff)
        return hipErrorInvalidValue;
    const float scale = 1.0f / sqrtf((float)BD);
    const float c_log2 = scale * LOG2E;
    // D and LSE log2 e, then dK/dV (which also writes dS), the partial sums, dQ
    hipLaunchKernelGGL((bwd_delta_kernel<D>), dim3((unsigned)dgrid), dim3(256), 0, stream,
                       (const __bf16*)a.O, (const __bf16*)a.dO, a.LSE, a.delta, a.lse2, rows);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.nseg > 0) {
        hipLaunchKernelGGL((bwd_dkdv_kernel<D, G, BW>), dim3((unsigned)(a.nseg * bhk)), dim3(256), 0,
                           stream, (const __bf16*)a.Q, (const __bf16*)a.K, (const __bf16*)a.V,
                           (const __bf16*)a.dO, a.lse2, a.delta, a.dK, a.dV, a.part, (__bf16*)a.ds,
                           a.segs, a.users, a.nslots, a.nusers, (int32_t)a.n, bhk, a.Hkv, c_log2, scale);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (a.nred > 0) {
        const int64_t grid = (int64_t)a.nred * bhk * (KT * BD / RED_CHUNK);
        if (grid > 0x7fffffff) return hipErrorInvalidValue;
        hipLaunchKernelGGL((bwd_reduce_kernel<D, BW>), dim3((unsigned)grid), dim3(256), 0,
                           stream, a.dK, a.dV, a.part, a.reds, a.nslots, (int32_t)a.n, bhk);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL((bwd_dq_kernel<D, G, BW>), dim3((unsigned)items), dim3(256), 0, stream,
                       (const __bf16*)a.K, (const __bf16*)a.ds, a.dQ, a.row_ptr, a.col_idx, a.nnz,
                       a.uoffs, a.nusers, (int32_t)a.n, NB, a.L, bhk, a.Hkv, scale);
    return hipGetLastError();
}

template <int D, int BW>
hipError_t launch_bwd_b(const BwdArgs& a, hipStream_t s) {
    switch (a.Hq / a.Hkv) {
        case 1:
            if constexpr (BW >= 128) return launch_bwd_g<D, 1, BW>(a, s);
            return hipErrorInvalidValue;  // G * B < 128: rejected by the interface
        case 2: return launch_bwd_g<D, 2, BW>(a, s);
        case 4: return launch_bwd_g<D, 4, BW>(a, s);
        default: return launch_bwd_g<D, 8, BW>(a, s);
    }
}

template <int D>
hipError_t launch_bwd_d(const BwdArgs& a, hipStream_t s) {
    return a.B == 64 ? launch_bwd_b<D, 64>(a, s) : launch_bwd_b<D, 128>(a, s);
}

}  // namespace

hipError_t launch_backward(const BwdArgs& a, hipStream_t stream) {
    return a.head_dim == 64 ? launch_bwd_d<64>(a, stream) : launch_bwd_d<128>(a, stream);
}

}  // namespace bf1
