// Shard planning and design-space shrinking, host only (no device calls):
// Eq. (1) dichotomy widths and the balanced slicing plan (§6.2), the die-aware
// workgroup rank, the Eq. (2) limiters, WIScore Eq. (4), OScore Eq. (5), the
// top-fraction cut (§6.3) and the head of the shaded binary tree (§7).
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "internal.h"

extern "C" {

int miriam_plan_dichotomy(int64_t M, int64_t *widths, int cap) {
    if (M < 1 || !widths) {
        miriam::set_error("dichotomy: M must be >= 1");
        return MIRIAM_EINVAL;
    }
    const int n = __builtin_ctzll((unsigned long long)M);  // largest i with 2^i | M
    if (n + 1 > cap) {
        miriam::set_error("dichotomy: output too small");
        return MIRIAM_ERANGE;
    }
    for (int j = 0; j <= n; ++j) widths[j] = M >> (n - j);
    return n + 1;
}

int miriam_plan_split(int64_t T, int64_t n, int64_t *begin, int64_t *len) {
    if (T < 1 || n < 1 || n > T || !begin || !len) {
        miriam::set_error("split: need 1 <= n <= T");
        return MIRIAM_EINVAL;
    }
    // shard j = [floor(j*T/n), floor((j+1)*T/n)); computed with quotient/remainder to avoid overflow
    const int64_t q = T / n, r = T % n;
    for (int64_t j = 0; j < n; ++j) {
        const int64_t bj = j * q + (j * r) / n;
        const int64_t ej = (j + 1) * q + ((j + 1) * r) / n;
        begin[j] = bj;
        len[j] = ej - bj;
    }
    return MIRIAM_OK;
}

int64_t miriam_plan_wg_rank(int64_t g, int64_t G, int64_t n_xcd) {
    if (G < 1 || n_xcd < 1 || g < 0 || g >= G) return -1;
    const int64_t die = g % n_xcd, slot = g / n_xcd;
    const int64_t base = G / n_xcd, extra = G % n_xcd;  // dies [0, extra) hold one more workgroup
    return die * base + std::min(die, extra) + slot;
}

int64_t miriam_plan_eq2_grid_limit(int64_t n_sm, int64_t n_blk_rt) {
    if (n_sm < 1 || n_blk_rt < 0) return -1;
    return n_sm - (n_blk_rt % n_sm);
}

int64_t miriam_plan_eq2_block_limit(int64_t l_threads, int64_t s_blk_rt) {
    if (l_threads < 1 || s_blk_rt < 0) return -1;
    return l_threads - s_blk_rt;
}

double miriam_plan_wiscore(int64_t n_sm, int64_t l_threads, int64_t n_blk_rt, int64_t s_blk_rt,
                           int64_t n_blk_be, int64_t s_blk_be) {
    if (n_sm < 1 || l_threads < 1) return -1.0;
    const double inter = double(n_blk_rt % n_sm + n_blk_be) / double(n_sm);
    const double intra = double(s_blk_rt + s_blk_be) / double(l_threads);
    return inter * intra;
}

int miriam_plan_oscore(int64_t n, const double *lo_blk, const double *lo_pt, double max_blk, double max_pt) {
    if (n < 0 || (n > 0 && (!lo_blk || !lo_pt))) return MIRIAM_EINVAL;
    const double sb = std::accumulate(lo_blk, lo_blk + n, 0.0);
    const double sp = std::accumulate(lo_pt, lo_pt + n, 0.0);
    return (sb < max_blk && sp < max_pt) ? 1 : 0;
}

int miriam_plan_top_fraction(int n, const double *score, const int64_t *grid, const int64_t *block, double frac,
                             int *keep) {
    if (n < 0 || (n > 0 && (!score || !grid || !block || !keep))) return MIRIAM_EINVAL;
    if (n == 0) return 0;
    std::vector<int> idx(n);
    std::iota(idx.begin(), idx.end(), 0);
    std::stable_sort(idx.begin(), idx.end(), [&](int a, int b) {
        if (score[a] != score[b]) return score[a] > score[b];
        if (grid[a] != grid[b]) return grid[a] > grid[b];
        return block[a] > block[b];
    });
    int k = (int)std::ceil(frac * n - 1e-12);
    k = std::max(1, std::min(k, n));
    std::copy(idx.begin(), idx.begin() + k, keep);
    return k;
}

int64_t miriam_plan_tree_head(int64_t T, int64_t cursor, int64_t max_len, int *depth) {
    if (T < 1 || cursor < 0 || cursor >= T || max_len < 1) return MIRIAM_EINVAL;
    // walk down the chain of nodes that contain `cursor`
    int64_t b = 0, e = T;
    int d = 0;
    while (!(b == cursor && e - b <= max_len)) {
        const int64_t mid = b + (e - b) / 2;
        if (cursor < mid) e = mid;
        else b = mid;
        ++d;
    }
    if (depth) *depth = d;
    return e - b;
}

}  // extern "C"
