/*
 * bf1.h -- C interface of libbf1.so: BF1 causal dyadic block-sparse
 * attention, prefill forward, for AMD Instinct MI355X (gfx950).
 *
 * The operation (paper §3.1, Eq. 1).  A sequence of n tokens is cut into
 * NB = ceil(n / B) blocks of B tokens (B is the block WIDTH here; the paper
 * writes b for the width and B for the count).  Query block j attends to the
 * key blocks
 *     P(j) = {j} ∪ {j-1, ..., j-L} ∪ {0} ∪ {j - 2^r : r >= 2},
 * restricted to [0, j] with duplicates removed (L = 2 is the paper's
 * configuration: two local blocks, the global first block, dyadic offsets
 * starting at four blocks).  Inside the self block j a token-level causal
 * triangle applies (key s visible to query t iff s <= t); every other selected
 * block is strictly earlier and fully visible.  Attention is softmax with
 * scale 1/sqrt(head_dim) and no bias (§3.1).  The result is exact softmax
 * attention restricted to that token mask (O(n log n) pairs, §3.2 Prop. 1).
 *
 * Conventions shared by every entry point:
 *  - All functions have C linkage, never abort or exit, and are thread-safe.
 *  - Device work is enqueued asynchronously on `stream` (a hipStream_t; NULL
 *    is the default stream of the current device).  Errors raised by the
 *    device surface at the caller's next synchronisation.
 *  - Argument errors are returned before anything is enqueued; no output is
 *    written in that case.
 *  - All tensors are caller-owned device memory on the current device.  The
 *    library never frees caller memory; it owns only its plan cache.
 *  - Graph capture: bf1_attn_fwd and bf1_attn_bwd build the route plan of a
 *    new (device, n, B, L) on first use (device allocation, a planner kernel
 *    on a private stream and a host wait, so a cached plan is complete and
 *    later calls add no stream dependency).  That first call cannot be
 *    captured: made while `stream` is being captured it returns
 *    BF1_ERR_CAPTURE and enqueues nothing.  Once the plan exists, calls can be
 *    captured; a captured graph keeps pointing at the plan's memory, so
 *    bf1_release_plans must not run while such a graph may still replay.
 *  - Layouts (row-major, contiguous):
 *        Q, O : [batch, Hq,  n, head_dim] bf16
 *        K, V : [batch, Hkv, n, head_dim] bf16
 *        LSE  : [batch, Hq,  n]           fp32, natural log of the softmax
 *                                           denominator including the max
 *    Q, K, V, O must be 16-byte aligned; LSE 4-byte aligned.
 *    q-head h reads kv-head h / (Hq / Hkv) (contiguous GQA groups).
 *  - Supported by the attention kernels: head_dim in {64, 128},
 *    B in {64, 128}, Hq / Hkv in {1, 2, 4, 8}, L >= 0, 0 <= n < 2^24,
 *    batch >= 0.
 *    Other values return BF1_ERR_UNSUPPORTED.  n == 0 or batch == 0 is a
 *    no-op returning BF1_OK.
 */
#ifndef BF1_H
#define BF1_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BF1_OK = 0,
    BF1_ERR_INVALID_ARG = -1,      /* null pointer, misalignment, bad size */
    BF1_ERR_UNSUPPORTED = -2,      /* valid but not built: head_dim, B, group */
    BF1_ERR_BUFFER_TOO_SMALL = -3, /* col_capacity below the route size */
    BF1_ERR_HIP = -4,              /* a HIP runtime call or launch failed */
    BF1_ERR_NOMEM = -5,            /* device allocation for the plan cache failed */
    BF1_ERR_CAPTURE = -6           /* a plan would have to be built during graph capture */
} bf1_status;

/*
 * Route sizes in closed form (host only, no device work).  §3.1 Eq. 1 for
 * the route and §3.2 Prop. 1 for the O(n log n) pair law.
 *   n >= 0, B >= 1, L >= 0.
 *   num_blocks <- NB = ceil(n / B)
 *   nnz        <- total entries of the CSR table (sum over j of |P(j)|)
 *   pairs      <- selected (query, key) token pairs per (batch, head),
 *                 counting the self-block triangle with its diagonal and a
 *                 partial last block of n - (NB-1)*B tokens.
 * Any output pointer may be NULL.  Returns BF1_ERR_INVALID_ARG on bad sizes
 * or if nnz would not fit in int32 indices.
 */
int bf1_plan_size(int64_t n, int32_t B, int32_t L,
                  int32_t* num_blocks, int64_t* nnz, int64_t* pairs);

/*
 * Route planner (§3.1, Eq. 1): writes the selected key-block table as CSR.
 *   row_ptr : device int32[NB + 1]; row_ptr[0] = 0, row_ptr[NB] = nnz.
 *   col_idx : device int32[col_capacity]; row j holds P(j) in ascending
 *             order (the self block j last), entries row_ptr[j]..row_ptr[j+1].
 * One integer HIP kernel, asynchronous on `stream`.  Returns
 * BF1_ERR_BUFFER_TOO_SMALL (nothing enqueued) if col_capacity < nnz.
 * n >= 0, B >= 1, L >= 0; n == 0 writes row_ptr[0] = 0 only.
 */
int bf1_plan(int64_t n, int32_t B, int32_t L,
             int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity,
             void* stream);

/*
 * BF1 prefill forward (§3.1): O and LSE for every (batch, q-head, token).
 * The route is built by the planner on first use for (device, n, B, L) and
 * kept in a library-owned cache (see bf1_release_plans); the attention
 * kernel then walks only the selected key blocks of each query block.
 * LSE may be NULL (not written).
 */
int bf1_attn_fwd(const void* Q, const void* K, const void* V, void* O, float* LSE,
                 int32_t batch, int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim,
                 int32_t B, int32_t L, void* stream);

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the BF1
 * prefill forward of bf1_attn_fwd, same arguments, same kernels and bitwise
 * the same results, with no allocation and no plan cache.  Each call runs the
 * route planner into a fixed scratch array owned by the library (one
 * 4 MiB __device__ array of int32, 2^20 entries, per device, held until the
 * process ends) and then the attention kernel over that table, both on
 * `stream`.  The table must fit: NB + 1 + nnz <= 2^20 (bf1_plan_size gives
 * NB and nnz; at B = 64, L = 2 this allows n up to about 2M tokens), else
 * BF1_ERR_BUFFER_TOO_SMALL is returned before anything is enqueued.  No
 * scratch content needs clearing: the planner rewrites every entry the
 * kernel reads.  All calls on one device share its array, so calls that
 * overlap in time on one device (on different streams, or from several
 * threads without ordering) race and may read each other's tables; calls
 * ordered on one stream do not.  The first call on a device looks the
 * array's address up (no allocation).
 */
int bf1_attn_fwd_noalloc(const void* Q, const void* K, const void* V, void* O, float* LSE,
                         int32_t batch, int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim,
                         int32_t B, int32_t L, void* stream);

/*
 * The same kernel with a caller-supplied route table: any causal block route
 * in the CSR form written by bf1_plan.  The paper times BF1 against other
 * routes of the same selected-pair count through one kernel (§4.3, §5.1:
 * matched local sliding and a static random graph; bf1_plan_variant builds
 * them), so the kernel takes the table as data.
 *   row_ptr : device int32[ceil(n/B) + 1], non-decreasing.
 *   col_idx : device int32[nnz]; entries of row j name key blocks.
 *   nnz     : the number of entries col_idx holds.  This argument is not in
 *             bf1_attn_fwd's interface: a table the caller wrote is not
 *             trusted, so the kernel clamps every row range to [0, nnz] and
 *             can never read past the end of col_idx, whatever row_ptr says.
 * Entries outside [0, j] are ignored (the route is causal: the self block j
 * gets the token-level triangle, earlier blocks are fully visible).  Each
 * block should appear at most once per row; a row that names no block at
 * all gets O = 0 and LSE = -inf.  All memory stays caller-owned.
 */
int bf1_attn_fwd_csr(const void* Q, const void* K, const void* V, void* O, float* LSE,
                     int32_t batch, int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim,
                     int32_t B, const int32_t* row_ptr, const int32_t* col_idx, int64_t nnz,
                     void* stream);

/*
 * Dense causal attention (every key s <= t), built from the same kernel with
 * the implicit route {0, ..., j} over 64-token blocks: the in-run comparator
 * for the BF1 operator (the paper compares against dense attention, §4.3).
 * Same layouts and support set as bf1_attn_fwd (no B, L).
 */
int bf1_dense_causal_fwd(const void* Q, const void* K, const void* V, void* O, float* LSE,
                         int32_t batch, int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim,
                         void* stream);

/*
 * Transposed route (host only, no device work): for every key block i the
 * ascending query blocks j whose route P(j) (§3.1, Eq. 1) contains i -- all
 * blocks for i = 0 (the global block), otherwise i, its L local successors
 * and the blocks i + 2^r (r >= 2) below NB.  This is the iteration space of
 * the dK/dV pass of the backward.
 *   row_ptr : HOST int32[NB + 1]; col_idx : HOST int32[col_capacity], the
 *             same nnz as the forward table (bf1_plan_size).
 * Returns BF1_ERR_BUFFER_TOO_SMALL if col_capacity < nnz.
 */
int bf1_plan_transposed(int64_t n, int32_t B, int32_t L,
                        int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity);

/*
 * BF1 backward: gradients of O = softmax(mask(Q K^T / sqrt(d))) V with the
 * §3.1 mask, for an upstream gradient dO, recomputing the weights from the
 * forward's LSE:
 *     P = exp(Q K^T / sqrt(d) - LSE),  D = rowsum(dO * O),  dS = P * (dO V^T - D),
 *     dQ = dS K / sqrt(d),  dK = dS^T Q / sqrt(d),  dV = P^T dO,
 * dK and dV summed over the q-heads of each GQA group.
 *   Q, O, dO : [batch, Hq, n, head_dim] bf16 (O and LSE as written by bf1_attn_fwd)
 *   K, V     : [batch, Hkv, n, head_dim] bf16
 *   LSE      : [batch, Hq, n] fp32, natural log
 *   dQ       : [batch, Hq, n, head_dim] fp32 (caller-owned, overwritten)
 *   dK, dV   : [batch, Hkv, n, head_dim] fp32 (caller-owned, overwritten)
 *   workspace: caller-owned device scratch of at least
 *              bf1_attn_bwd_workspace_size() bytes, 256-byte aligned; its
 *              contents on entry are irrelevant and are clobbered.
 * Supported: head_dim in {64, 128}, B in {64, 128}, G = Hq/Hkv in {1, 2, 4, 8}
 * with G * B >= 128 (so G = 1 needs B = 128); others return BF1_ERR_UNSUPPORTED.
 * Four kernels on `stream`: D and LSE log2 e per query row (to the
 * workspace); dK/dV over the transposed route (cut into segments of at most
 * 16 query blocks; the segments of long lists -- block 0 -- leave partial
 * sums in the workspace), which also writes dS (bf16, one 8 KB unit per
 * selected block pair, q-head and pair of 64-row sub-tiles) to the workspace;
 * a fixed-order sum of the partials; and dQ = dS K / sqrt(d) from the stored
 * dS along the forward route.  The workspace therefore grows with the number
 * of selected pairs (670 MB at n = 32768 with 16 q-heads, b = 64).  The route and its
 * transpose are cached per (device, n, B, L) like bf1_attn_fwd's.  The result
 * is deterministic.
 */
int bf1_attn_bwd_workspace_size(int32_t batch, int64_t n, int32_t Hq, int32_t Hkv,
                                int32_t head_dim, int32_t B, int32_t L, int64_t* bytes);
int bf1_attn_bwd(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const float* LSE, float* dQ, float* dK, float* dV,
                 int32_t batch, int64_t n, int32_t Hq, int32_t Hkv, int32_t head_dim,
                 int32_t B, int32_t L, void* workspace, int64_t workspace_bytes, void* stream);

/*
 * Route variants at BF1's selected-pair budget (host only, no device work):
 * the topology controls the paper times against BF1 (§4.3, §5.1) and
 * compares by communication depth (§5.2, Table 1).  Every variant keeps
 * |P(j)| blocks in row j (self block included, rows ascending), so its CSR
 * size and its selected pairs equal BF1's (bf1_plan_size) and its tables run
 * unchanged through bf1_attn_fwd_csr.
 *   BF1_ROUTE_BF1           Eq. 1 itself (the table bf1_plan writes).
 *   BF1_ROUTE_SLIDING       matched local sliding: blocks j-|P(j)|+1 .. j.
 *   BF1_ROUTE_STATIC_RANDOM static random nonlocal graph: the self block and
 *       the L local predecessors of Eq. 1 stay; BF1's other blocks (global
 *       and dyadic, all before j-L) are replaced by as many distinct blocks
 *       drawn uniformly from 0 .. j-L-1 with Floyd's sampling; draw t of row j
 *       is SplitMix64 output number j*2^20 + t of the generator seeded with
 *       `seed` (the paper's graph uses seed 17), mapped to [0, r] as
 *       (high 32 bits * (r+1)) >> 32.  `seed` is ignored by the other kinds.
 *   row_ptr : HOST int32[NB + 1]; col_idx : HOST int32[col_capacity].
 * Returns BF1_ERR_INVALID_ARG for an unknown kind or bad sizes,
 * BF1_ERR_BUFFER_TOO_SMALL if col_capacity < nnz.
 */
typedef enum {
    BF1_ROUTE_BF1 = 0,
    BF1_ROUTE_SLIDING = 1,
    BF1_ROUTE_STATIC_RANDOM = 2
} bf1_route_kind;

int bf1_plan_variant(int32_t kind, int64_t n, int32_t B, int32_t L, uint64_t seed,
                     int32_t* row_ptr, int32_t* col_idx, int64_t col_capacity);

/*
 * Communication depth of a causal block route (host only; §3.3 Prop. 2 and
 * §5.2): the largest, over pairs of blocks i < j, of the fewest hops from i
 * to j along edges i -> j' for every earlier block i in row j' of the table.
 *   row_ptr : HOST int32[num_blocks + 1], row_ptr[0] = 0, non-decreasing;
 *   col_idx : HOST int32[row_ptr[num_blocks]], every entry of row j in [0, j].
 *   max_depth <- the depth, or -1 if some later block is unreachable.
 * Breadth-first search from every block: O(num_blocks * (num_blocks + nnz))
 * time, num_blocks <= 16384.  Returns BF1_ERR_INVALID_ARG on a malformed or
 * non-causal table.
 */
int bf1_route_depth(const int32_t* row_ptr, const int32_t* col_idx, int32_t num_blocks,
                    int32_t* max_depth);

/*
 * One-token decode over a paged key/value cache (§3.2: a decoded token reads
 * O(log NB) blocks; §4.2 "cached one-token decode"; §5.4 selected-page
 * decode with a plan that persists across the route epoch).
 *
 * The newest token of sequence b sits at t = seq_lens[b] - 1 in query block
 * j = t / B and attends to row t of the prefill mask: all keys of the earlier
 * blocks of P(j) (Eq. 1) and keys j*B .. t of block j.  Its K and V must
 * already be in the cache.  A cache page holds one block (B tokens):
 *   K_pages, V_pages : [num_pages, Hkv, B, head_dim] bf16 (16-byte aligned)
 *   page_table       : [batch, max_pages_per_seq] int32, logical block i of
 *                      sequence b lives in page page_table[b, i]
 *   seq_lens         : [batch] int32, >= 1
 *   Q, O             : [batch, Hq, head_dim] bf16; LSE [batch, Hq] fp32
 *                      (natural log, may be NULL)
 * all device memory, caller-owned.
 *
 * Plan (built once per route epoch: it stays valid while every sequence's
 * newest token remains in the block it was built for, i.e. for up to B
 * steps):  int32 [batch, plan_stride] device memory, row b =
 *   [j, c, the c physical pages of the earlier selected blocks (ascending
 *    logical block), the page of block j, padding]
 * The page table is read only by the planner: a step reads its sequence
 * length and its plan row.  Pages must not move while a plan is in use.
 * bf1_decode_plan_stride gives the stride for sequences of up to
 * max_seq_len tokens; `dense` = 1 plans every earlier block instead of P(j)
 * (the dense decode comparator).  bf1_decode_plan is one kernel on `stream`;
 * a sequence whose length is < 1, whose block is past max_pages_per_seq, or
 * whose pages (earlier or self) fall outside [0, num_pages) is marked
 * unplannable (j = -1).
 *
 * bf1_decode_attn: two kernels on `stream` (a split kernel over the pages and
 * a merge of the split results, in a fixed order: deterministic).  A sequence
 * whose plan row was made for another block (stale) or is unplannable gets
 * NaN in its O rows and LSE; a plan row that bf1_decode_plan did not write
 * gives undefined values, never a read outside the plan row and the cache.
 * Keys past t in the self page are masked exactly, whatever the page holds.
 * workspace: device scratch of at least bf1_decode_workspace_size() bytes,
 * 16-byte aligned, contents irrelevant.  Supported: head_dim in {64, 128},
 * B in {64, 128}, Hq / Hkv in {1, 2, 4, 8}, L <= 32.
 */
int bf1_decode_plan_stride(int64_t max_seq_len, int32_t B, int32_t L, int32_t dense,
                           int32_t* plan_stride);
int bf1_decode_plan(int32_t batch, const int32_t* seq_lens, const int32_t* page_table,
                    int32_t max_pages_per_seq, int32_t num_pages, int32_t B, int32_t L, int32_t dense,
                    int32_t* plan, int32_t plan_stride, void* stream);
int bf1_decode_workspace_size(int32_t batch, int32_t Hq, int32_t Hkv, int32_t head_dim,
                              int32_t plan_stride, int64_t* bytes);
int bf1_decode_attn(const void* Q, const void* K_pages, const void* V_pages, const int32_t* seq_lens,
                    int32_t num_pages, const int32_t* plan, int32_t plan_stride, void* O, float* LSE,
                    int32_t batch, int32_t Hq, int32_t Hkv, int32_t head_dim, int32_t B,
                    void* workspace, int64_t workspace_bytes, void* stream);

/*
 * Key split of the forward kernels (bf1_attn_fwd, bf1_attn_fwd_noalloc,
 * bf1_attn_fwd_csr, bf1_dense_causal_fwd), process-wide:
 *   0  automatic (the default): when a launch has at most one work item (one
 *      query block of one kv-head, all its q-heads) per compute unit and its
 *      routes average at least 8 key tiles of 64 keys per item, each
 *      workgroup runs two groups of waves that take alternate key tiles of
 *      the route and merge their partial softmax states at the end, halving
 *      the chain of tiles per workgroup (in practice: the dense comparator
 *      below ~4K tokens; BF1 routes are too short to gain).  The result is the
 *      same attention (§3.1) up to the order of the fp32 sums.
 *   1  never split;   2  always split.
 * Each setting is deterministic; the two paths agree within the parity
 * bars, not bitwise.  Intended for tuning and tests; calls in flight are not
 * affected.  Returns BF1_ERR_INVALID_ARG for any other mode.
 */
int bf1_set_forward_key_split(int32_t mode);

/* Frees every cached plan (device memory owned by the library).  Must not
 * race with in-flight bf1_attn_fwd / bf1_attn_bwd calls that use those plans. */
void bf1_release_plans(void);

/* Static, human-readable name of a status code. */
const char* bf1_status_string(int status);

/* Interface version (major * 10000 + minor * 100 + patch). */
int bf1_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BF1_H */
