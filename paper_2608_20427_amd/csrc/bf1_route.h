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

}  // namespace bf1
