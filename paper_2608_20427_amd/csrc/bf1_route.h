// Closed forms of the BF1 block route (paper §3.1, Eq. 1; §3.2, Prop. 1),
// usable from host and device code.
//
// Route of query block j with local width L:
//   P(j) = {j} ∪ {j-1..j-L} ∪ {0} ∪ {j - 2^r : r >= 2}, clipped to [0, j].
// Its earlier blocks (j excluded) number
//   c(j) = min(j, L) + |D(j)| + [j > L and j not in D(j)],
//   D(j) = {2^r : r >= 2, L < 2^r <= j}      (dyadic offsets not already local),
// because a dyadic offset 2^r <= L lands on a local block, and block 0 is new
// only when it is neither local (j > L) nor dyadic (j not a power of two in D).
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define BF1_HD __host__ __device__ __forceinline__
#else
#define BF1_HD inline
#endif

namespace bf1 {

// Number of r >= 2 with L < 2^r < lim  (strict) -- helper for prefix sums.
BF1_HD int64_t dyadic_count_below(int64_t lim, int64_t L) {
    int64_t c = 0;
    for (int r = 2; r < 62 && (int64_t(1) << r) < lim; ++r)
        if ((int64_t(1) << r) > L) ++c;
    return c;
}

// Earlier selected blocks of query block j.
BF1_HD int64_t route_pred_count(int64_t j, int64_t L) {
    int64_t c = j < L ? j : L;
    bool pow_in_D = false;
    for (int r = 2; r < 62 && (int64_t(1) << r) <= j; ++r) {
        int64_t off = int64_t(1) << r;
        if (off > L) {
            ++c;
            if (off == j) pow_in_D = true;
        }
    }
    if (j > L && !pow_in_D) ++c;
    return c;
}

// Row start of block j in the CSR table: sum over i < j of (1 + c(i)),
// summed term by term:
//   self blocks               j
//   locals    sum min(i, L) = j(j-1)/2                    (j <= L)
//                           = L(L-1)/2 + L(j-L)           (j > L)
//   dyadics   sum |D(i)|    = sum over L < 2^r < j of (j - 2^r)
//   global                  = max(0, j-L-1) - #{r >= 2 : L < 2^r < j}
BF1_HD int64_t route_row_start(int64_t j, int64_t L) {
    int64_t s = j;
    s += (j <= L) ? j * (j - 1) / 2 : L * (L - 1) / 2 + L * (j - L);
    for (int r = 2; r < 62 && (int64_t(1) << r) < j; ++r) {
        int64_t off = int64_t(1) << r;
        if (off > L) s += j - off;
    }
    int64_t g = j - L - 1;
    s += (g > 0 ? g : 0) - dyadic_count_below(j, L);
    return s;
}

// Selected token pairs per (batch, head) for n tokens in blocks of width b:
// earlier blocks give full rectangles, the self block a triangle with its
// diagonal; only the last block (m = n - (NB-1) b tokens) can be partial.
inline int64_t route_selected_pairs(int64_t n, int64_t b, int64_t L) {
    if (n <= 0) return 0;
    int64_t NB = (n + b - 1) / b;
    int64_t m = n - (NB - 1) * b;
    int64_t full = 0;
    for (int64_t j = 0; j + 1 < NB; ++j) full += route_pred_count(j, L);
    return b * b * full + (NB - 1) * (b * (b + 1) / 2) + m * b * route_pred_count(NB - 1, L) +
           m * (m + 1) / 2;
}


// Query blocks that select key block i (the route transposed), ascending,
// written to out (may be null); returns their number.  Key block 0 is the
// global block of every query block; any other block i is selected by itself,
// its L local successors i+1..i+L and the blocks i + 2^r with r >= 2 and
// 2^r > L (smaller dyadic offsets land on the local successors), all clipped
// to [0, NB).  Locals precede dyadics, so the list comes out sorted.
inline int64_t route_users(int64_t NB, int64_t L, int64_t i, int32_t* out) {
    int64_t c = 0;
    if (i == 0) {
        for (int64_t jq = 0; jq < NB; ++jq)
            if (out) out[c++] = (int32_t)jq; else ++c;
        return c;
    }
    for (int64_t jq = i; jq <= i + L && jq < NB; ++jq)
        if (out) out[c++] = (int32_t)jq; else ++c;
    for (int64_t r = 2; r < 62; ++r) {
        const int64_t off = int64_t(1) << r;
        if (i + off >= NB) break;
        if (off > L) {
            if (out) out[c++] = (int32_t)(i + off); else ++c;
        }
    }
    return c;
}

// Position of query block j in the list route_users writes for key block i,
// for a pair (j selects i) of the route: block 0's list is every query block
// in order; any other list is i itself, its locals at distances 1..L, then the
// dyadic users at distances 2^r > L in increasing r.  Entries before j are all
// below j, so the clipping to [0, NB) never changes the position.
BF1_HD int64_t route_user_rank(int64_t L, int64_t i, int64_t j) {
    if (i == 0) return j;
    const int64_t d = j - i;
    return d <= L ? d : L + 1 + dyadic_count_below(d, L);
}

// ---- Route variants at BF1's selected-pair budget (§4.3, §5.1, Table 1) ----
// Both keep |P(j)| blocks in every row, so every query token sees exactly as
// many keys as under Eq. 1 and the totals (pairs, CSR size) are BF1's.

// Output number c (from 0) of SplitMix64 seeded with `seed` (Steele, Lea and
// Flood, OOPSLA 2014): the state after c + 1 steps of adding the golden-ratio
// increment, put through the generator's 64-bit finaliser.
inline uint64_t splitmix64_at(uint64_t seed, uint64_t c) {
    uint64_t z = seed + (c + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Contiguous local sliding route: the |P(j)| most recent blocks up to j.
inline int64_t route_sliding_row(int64_t j, int64_t L, int32_t* out) {
    const int64_t size = 1 + route_pred_count(j, L);
    for (int64_t t = 0; t < size; ++t) out[t] = (int32_t)(j - size + 1 + t);
    return size;
}

// Static random nonlocal route: the self block and its L local predecessors
// stay; the remaining k = |P(j)| - (locals + 1) entries are distinct blocks
// drawn uniformly from 0 .. j-L-1 by Floyd's k-of-m sampling (Bentley and
// Floyd, CACM 1987): for t < k, with r = m - k + t, draw x in [0, r] and
// keep r if x is already chosen, else x.  Draw t of row j uses SplitMix64
// output j * 2^20 + t, mapped to [0, r] by (high 32 bits * (r + 1)) >> 32.
// Row written ascending; returns its length.
inline int64_t route_static_random_row(int64_t j, int64_t L, uint64_t seed, int32_t* out) {
    const int64_t lo = j - L > 0 ? j - L : 0;
    const int64_t size = 1 + route_pred_count(j, L);
    const int64_t k = size - (j - lo + 1);
    const int64_t m = j - L;
    int64_t c = 0;
    for (int64_t t = 0; t < k; ++t) {
        const uint64_t r = (uint64_t)(m - k + t);
        const uint64_t x = ((splitmix64_at(seed, ((uint64_t)j << 20) + (uint64_t)t) >> 32) * (r + 1)) >> 32;
        bool seen = false;
        for (int64_t a = 0; a < c; ++a) seen |= (uint64_t)out[a] == x;
        out[c++] = (int32_t)(seen ? r : x);
    }
    // insertion sort of the k drawn blocks (k < 64)
    for (int64_t a = 1; a < c; ++a) {
        const int32_t v = out[a];
        int64_t b = a;
        for (; b > 0 && out[b - 1] > v; --b) out[b] = out[b - 1];
        out[b] = v;
    }
    for (int64_t i = lo; i <= j; ++i) out[c++] = (int32_t)i;
    return c;
}

}  // namespace bf1
