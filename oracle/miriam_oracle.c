/*
 * Miriam CPU oracle — TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously-correct double-precision implementation of what the
 * elastic-kernel hot path computes.  Only the test suite, the smoke check and
 * the CPU baseline leg of the benchmark may load this library; the product
 * path never does.  It shares no code, header, table or helper with the HIP
 * library: every formula below is written out from its definition.
 *
 * Paper: "Miriam: Exploiting Elastic Kernels for Real-time Multi-DNN
 * Inference on Edge GPU" (Zhao, Ling, Guan, Xing; arXiv 2307.04339).
 *
 * Conventions
 *   - Activations are NHWC, convolution weights are [Cout][KH][KW][Cin/groups],
 *     GEMM is Y[m][n] = sum_k X[m][k] * W[n][k].
 *   - Every value is a double; callers widen fp32/fp16/bf16 inputs exactly.
 *   - Functions return 0 on success and a negative number on bad arguments.
 *   - The convolution and the matrix products may spread their output elements over
 *     host threads (OpenMP, or_set_threads); each element is still computed by one
 *     thread with the loop order written below, so results do not depend on the count.
 *
 * Pins: every function here is checked by tests against closed forms, brute
 * force on tiny inputs, worked values, invariants, or an independent library
 * routine.  The one exception is noted at or_oscore (its constants are not
 * fixed by the paper; the predicate itself is pinned by hand cases).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Part 1: the elastic grid — slicing plans and the tile/owner map.          */
/* ------------------------------------------------------------------------ */

/*
 * Eq. (1), §6.2: the dichotomy slicing plan of a kernel with M thread blocks
 * lists the slice widths M/2^n, M/2^(n-1), ..., M where n is the largest i
 * with M divisible by 2^i (the 2-adic valuation of M).
 * Writes n+1 widths into out (smallest first) and returns n+1; returns -1 for
 * M < 1 and -2 if cap is too small.
 */
int or_dichotomy(int64_t M, int64_t *out, int cap)
{
    if (M < 1) return -1;
    int n = 0;
    int64_t m = M;
    while (m % 2 == 0) { m /= 2; n++; }
    if (n + 1 > cap) return -2;
    for (int j = 0; j <= n; j++) {
        int64_t p = 1;
        for (int q = 0; q < n - j; q++) p *= 2;
        out[j] = M / p;
    }
    return n + 1;
}

/*
 * Slicing plan P(K) = [s0 .. s_{n-1}] at thread-block granularity (§6.2).
 * Reading for any shard count n (the paper's dichotomy only yields powers of
 * two of an even M): shard j covers tiles [floor(j*T/n), floor((j+1)*T/n)).
 * When 2^k divides T and n = 2^k every shard has width T/2^k, i.e. Eq. (1).
 */
int or_balanced_split(int64_t T, int64_t n, int64_t *begin, int64_t *len)
{
    if (T < 1 || n < 1 || n > T) return -1;
    for (int64_t j = 0; j < n; j++) {
        int64_t b = (j * T) / n;
        int64_t e = ((j + 1) * T) / n;
        begin[j] = b;
        len[j] = e - b;
    }
    return 0;
}

/*
 * Physical-to-logical workgroup order inside one launch.  Workgroups of a
 * launch are handed round-robin to the chip's X dies; to keep tiles that share
 * operands on one die, physical workgroup g (die x = g mod X, slot g div X) is
 * given logical rank  x*floor(G/X) + min(x, G mod X) + g div X.
 * This is a bijection of [0, G).
 */
int64_t or_wg_rank(int64_t g, int64_t G, int64_t X)
{
    int64_t q = G / X, r = G % X;
    int64_t x = g % X;
    int64_t s = g / X;
    return x * q + (x < r ? x : r) + s;
}

/*
 * Elastic grid + persistent threads (§6.1, §6.2): a shard [b, b+l) launched
 * with G physical workgroups.  Workgroup g with logical rank r (or_wg_rank)
 * executes tiles  t_i = b + r + i*G  for i = 0, 1, ... while t_i < b + l.
 *
 * Given a plan of n shards, fill for each tile t in [0,T):
 *   owner_shard[t], owner_wg[t], owner_iter[t]   (last writer)
 *   count[t]                                      (number of executions)
 * Each shard j has its own grid G[j].  Returns 0, or -1 on bad input.
 */
int or_owner_map(int64_t T, int64_t n, const int64_t *begin, const int64_t *len,
                 const int64_t *G, int64_t X,
                 int32_t *owner_shard, int32_t *owner_wg, int32_t *owner_iter,
                 int32_t *count)
{
    if (T < 0 || n < 0 || X < 1) return -1;
    for (int64_t t = 0; t < T; t++) {
        owner_shard[t] = -1; owner_wg[t] = -1; owner_iter[t] = -1; count[t] = 0;
    }
    for (int64_t j = 0; j < n; j++) {
        if (begin[j] < 0 || len[j] < 1 || begin[j] + len[j] > T || G[j] < 1) return -1;
        for (int64_t g = 0; g < G[j]; g++) {
            int64_t r = or_wg_rank(g, G[j], X);
            for (int64_t i = 0;; i++) {
                int64_t t = begin[j] + r + i * G[j];
                if (t >= begin[j] + len[j]) break;
                owner_shard[t] = (int32_t)j;
                owner_wg[t] = (int32_t)g;
                owner_iter[t] = (int32_t)i;
                count[t] += 1;
            }
        }
    }
    return 0;
}

/*
 * Elastic block (§6.1): the logical block of L logical waves is run by a
 * physical block of P waves with the N:1 map  logical wave lambda ->
 * physical wave (lambda mod P), round floor(lambda / P).
 */
int or_wave_map(int L, int P, int lambda, int *phys_wave, int *round)
{
    if (P < 1 || L < 1 || L % P != 0 || lambda < 0 || lambda >= L) return -1;
    *phys_wave = lambda % P;
    *round = lambda / P;
    return 0;
}

/*
 * Tile id -> (batch, mt, nt) for a contraction whose output is a batch of
 * M x N matrices cut into TM x TN tiles; the N index runs fastest.
 */
int or_tile_coords(int64_t t, int64_t M, int64_t N, int64_t TM, int64_t TN,
                   int64_t *bi, int64_t *mt, int64_t *nt)
{
    if (TM < 1 || TN < 1 || M < 1 || N < 1 || t < 0) return -1;
    int64_t mT = (M + TM - 1) / TM, nT = (N + TN - 1) / TN;
    *bi = t / (mT * nT);
    int64_t r = t % (mT * nT);
    *mt = r / nT;
    *nt = r % nT;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Part 2: design-space shrinking (§6.3, Table 1, Eq. (2), (4), (5)).        */
/* ------------------------------------------------------------------------ */

/* Eq. (2), first line: N_blk_be <= N_SM - (N_blk_rt mod N_SM). */
int64_t or_eq2_grid_limit(int64_t n_sm, int64_t n_blk_rt)
{
    return n_sm - (n_blk_rt % n_sm);
}

/* Eq. (2), second line: S_blk_be <= L_threads - S_blk_rt. */
int64_t or_eq2_block_limit(int64_t l_threads, int64_t s_blk_rt)
{
    return l_threads - s_blk_rt;
}

/* 1 if the candidate (N_blk_be, S_blk_be) satisfies both lines of Eq. (2). */
int or_eq2_feasible(int64_t n_sm, int64_t l_threads, int64_t n_blk_rt, int64_t s_blk_rt,
                    int64_t n_blk_be, int64_t s_blk_be)
{
    return n_blk_be <= or_eq2_grid_limit(n_sm, n_blk_rt) &&
           s_blk_be <= or_eq2_block_limit(l_threads, s_blk_rt);
}

/*
 * Eq. (4) WIScore.  The printed second factor adds S_blk_be to itself; the
 * reading taken here is (S_blk_rt + S_blk_be) / L_threads, the share of the
 * per-SM thread limit used by both kernels, which with Eq. (2) keeps the
 * score in [0, 1] as the paper states.
 */
double or_wiscore(int64_t n_sm, int64_t l_threads, int64_t n_blk_rt, int64_t s_blk_rt,
                  int64_t n_blk_be, int64_t s_blk_be)
{
    double inter = (double)((n_blk_rt % n_sm) + n_blk_be) / (double)n_sm;
    double intra = (double)(s_blk_rt + s_blk_be) / (double)l_threads;
    return inter * intra;
}

/*
 * Eq. (5) OScore: 1 when the summed block-launch overhead and the summed
 * persistent-thread overhead of the n shards both stay under their bars,
 * else 0.  The bars are constants the paper does not give; callers pass them.
 */
int or_oscore(int64_t n, const double *lo_blk, const double *lo_pt,
              double max_blk, double max_pt)
{
    double sb = 0.0, sp = 0.0;
    for (int64_t i = 0; i < n; i++) { sb += lo_blk[i]; sp += lo_pt[i]; }
    return (sb < max_blk && sp < max_pt) ? 1 : 0;
}

/*
 * §6.3 "top 20%": rank candidates by score (ties: larger grid first, then
 * larger block first) and keep ceil(frac * n) of them, at least one.
 * Writes the kept candidate indices (best first) to keep[] and returns the
 * count.  Selection by repeated scan of the remaining candidates, O(n^2).
 */
int or_top_fraction(int n, const double *score, const int64_t *grid, const int64_t *block,
                    double frac, int *keep)
{
    if (n < 1) return 0;
    int k = (int)ceil(frac * (double)n - 1e-12);
    if (k < 1) k = 1;
    if (k > n) k = n;
    char *used = (char *)calloc((size_t)n, 1);
    for (int s = 0; s < k; s++) {
        int best = -1;
        for (int i = 0; i < n; i++) {
            if (used[i]) continue;
            if (best < 0) { best = i; continue; }
            int better = 0;
            if (score[i] > score[best]) better = 1;
            else if (score[i] == score[best]) {
                if (grid[i] > grid[best]) better = 1;
                else if (grid[i] == grid[best] && block[i] > block[best]) better = 1;
            }
            if (better) best = i;
        }
        used[best] = 1;
        keep[s] = best;
    }
    free(used);
    return k;
}

/* ------------------------------------------------------------------------ */
/* Part 3: the shaded binary tree of §7.                                     */
/* ------------------------------------------------------------------------ */

/*
 * The tree's root is the whole tile range [0, T); a node [b, e) with e-b >= 2
 * has the children [b, floor((b+e)/2)) and [floor((b+e)/2), e).  Shards are
 * taken from the head of the tree: with everything before `cursor` already
 * dispatched, the next shard is the shallowest node that starts at `cursor`
 * and holds at most `max_len` tiles.  Found by listing, depth by depth, every
 * node of the tree (breadth-first) and returning the first match.
 * Returns the node's length (its end is cursor + length) and its depth.
 */
int64_t or_tree_head(int64_t T, int64_t cursor, int64_t max_len, int *depth_out)
{
    if (T < 1 || cursor < 0 || cursor >= T || max_len < 1) return -1;
    /* level-by-level list of nodes; at most T leaves so 2T nodes per level is ample */
    int64_t *lb = (int64_t *)malloc(sizeof(int64_t) * 2 * (size_t)T);
    int64_t *le = (int64_t *)malloc(sizeof(int64_t) * 2 * (size_t)T);
    int64_t *nb = (int64_t *)malloc(sizeof(int64_t) * 2 * (size_t)T);
    int64_t *ne = (int64_t *)malloc(sizeof(int64_t) * 2 * (size_t)T);
    int64_t cnt = 1;
    lb[0] = 0; le[0] = T;
    int64_t found = -1;
    for (int depth = 0; cnt > 0; depth++) {
        for (int64_t i = 0; i < cnt; i++) {
            if (lb[i] == cursor && le[i] - lb[i] <= max_len) {
                found = le[i] - lb[i];
                *depth_out = depth;
                break;
            }
        }
        if (found >= 0) break;
        int64_t nc = 0;
        for (int64_t i = 0; i < cnt; i++) {
            if (le[i] - lb[i] >= 2) {
                int64_t mid = (lb[i] + le[i]) / 2;
                nb[nc] = lb[i]; ne[nc] = mid; nc++;
                nb[nc] = mid; ne[nc] = le[i]; nc++;
            }
        }
        memcpy(lb, nb, sizeof(int64_t) * (size_t)nc);
        memcpy(le, ne, sizeof(int64_t) * (size_t)nc);
        cnt = nc;
    }
    free(lb); free(le); free(nb); free(ne);
    return found;
}

/* ------------------------------------------------------------------------ */
/* Part 4: the DNN operators an elastic kernel must reproduce exactly.       */
/* (The elastic transformation preserves the original computation, §6.4.)    */
/* ------------------------------------------------------------------------ */

/*
 * 2-D convolution (cross-correlation, as in DNN frameworks), zero padding:
 *   Ho = floor((H + 2*pad - KH) / stride) + 1, likewise Wo;
 *   y[n,p,q,co] = sum_{ci in group, r, u} x[n, p*stride - pad + r, q*stride - pad + u, ci]
 *                                        * w[co, r, u, ci - group_base]
 * x: N x H x W x C (NHWC), w: K x KH x KW x (C/groups), y: N x Ho x Wo x K.
 * groups == C gives depthwise convolution.
 */
int or_conv2d(const double *x, int64_t N, int64_t H, int64_t W, int64_t C,
              const double *w, int64_t K, int64_t KH, int64_t KW,
              int64_t stride, int64_t pad, int64_t groups, double *y)
{
    if (groups < 1 || C % groups != 0 || K % groups != 0 || stride < 1 || pad < 0) return -1;
    int64_t Ho = (H + 2 * pad - KH) / stride + 1;
    int64_t Wo = (W + 2 * pad - KW) / stride + 1;
    if (Ho < 1 || Wo < 1) return -1;
    int64_t cg = C / groups, kg = K / groups;
#pragma omp parallel for collapse(3) schedule(static)
    for (int64_t n = 0; n < N; n++)
        for (int64_t p = 0; p < Ho; p++)
            for (int64_t q = 0; q < Wo; q++)
                for (int64_t co = 0; co < K; co++) {
                    int64_t g = co / kg;
                    double s = 0.0;
                    for (int64_t r = 0; r < KH; r++) {
                        int64_t h = p * stride - pad + r;
                        if (h < 0 || h >= H) continue;
                        for (int64_t u = 0; u < KW; u++) {
                            int64_t ww = q * stride - pad + u;
                            if (ww < 0 || ww >= W) continue;
                            for (int64_t c = 0; c < cg; c++) {
                                double xv = x[((n * H + h) * W + ww) * C + g * cg + c];
                                double wv = w[((co * KH + r) * KW + u) * cg + c];
                                s += xv * wv;
                            }
                        }
                    }
                    y[((n * Ho + p) * Wo + q) * K + co] = s;
                }
    return 0;
}

/* Fully connected layer / matrix product: Y[m][n] = sum_k X[m][k] * W[n][k]. */
int or_gemm_nt(const double *X, const double *Wt, int64_t M, int64_t N, int64_t K, double *Y)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t m = 0; m < M; m++)
        for (int64_t n = 0; n < N; n++) {
            double s = 0.0;
            for (int64_t k = 0; k < K; k++) s += X[m * K + k] * Wt[n * K + k];
            Y[m * N + n] = s;
        }
    return 0;
}

/* Matrix product with the right operand stored K x N: Y[m][n] = sum_k X[m][k] * B[k][n]. */
int or_gemm_nn(const double *X, const double *B, int64_t M, int64_t N, int64_t K, double *Y)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t m = 0; m < M; m++)
        for (int64_t n = 0; n < N; n++) {
            double s = 0.0;
            for (int64_t k = 0; k < K; k++) s += X[m * K + k] * B[k * N + n];
            Y[m * N + n] = s;
        }
    return 0;
}

/* Activation codes shared with the Python wrapper of this oracle. */
enum { OR_ACT_NONE = 0, OR_ACT_RELU = 1, OR_ACT_RELU6 = 2, OR_ACT_GELU = 3 };

static double or_act(double v, int act)
{
    switch (act) {
    case OR_ACT_RELU: return v > 0.0 ? v : 0.0;
    case OR_ACT_RELU6: return v < 0.0 ? 0.0 : (v > 6.0 ? 6.0 : v);
    case OR_ACT_GELU: return 0.5 * v * (1.0 + erf(v / sqrt(2.0)));
    default: return v;
    }
}

/*
 * Per-channel epilogue over rows x C values (channel index fastest), in order:
 *   v = y + bias[c]                                  (if bias)
 *   v = (v - mean[c]) / sqrt(var[c] + eps) * gamma[c] + beta[c]   (inference BN, if bn)
 *   v = v + residual                                  (if residual)
 *   v = act(v)
 * bn points at 4*C doubles: gamma, beta, mean, var.
 */
int or_epilogue(double *y, int64_t rows, int64_t C, const double *bias, const double *bn,
                double eps, const double *residual, int act)
{
    for (int64_t i = 0; i < rows; i++)
        for (int64_t c = 0; c < C; c++) {
            double v = y[i * C + c];
            if (bias) v += bias[c];
            if (bn) v = (v - bn[2 * C + c]) / sqrt(bn[3 * C + c] + eps) * bn[c] + bn[C + c];
            if (residual) v += residual[i * C + c];
            y[i * C + c] = or_act(v, act);
        }
    return 0;
}

/*
 * Max pooling over NHWC with zero-sized (ignored) padding: taps outside the
 * input do not take part in the maximum.
 */
int or_maxpool(const double *x, int64_t N, int64_t H, int64_t W, int64_t C,
               int64_t KH, int64_t KW, int64_t stride, int64_t pad, double *y)
{
    int64_t Ho = (H + 2 * pad - KH) / stride + 1;
    int64_t Wo = (W + 2 * pad - KW) / stride + 1;
    if (Ho < 1 || Wo < 1) return -1;
    for (int64_t n = 0; n < N; n++)
        for (int64_t p = 0; p < Ho; p++)
            for (int64_t q = 0; q < Wo; q++)
                for (int64_t c = 0; c < C; c++) {
                    double m = -INFINITY;
                    for (int64_t r = 0; r < KH; r++)
                        for (int64_t u = 0; u < KW; u++) {
                            int64_t h = p * stride - pad + r, w = q * stride - pad + u;
                            if (h < 0 || h >= H || w < 0 || w >= W) continue;
                            double v = x[((n * H + h) * W + w) * C + c];
                            if (v > m) m = v;
                        }
                    y[((n * Ho + p) * Wo + q) * C + c] = m;
                }
    return 0;
}

/* Average pooling over NHWC; the sum of the in-bounds taps is divided by KH*KW. */
int or_avgpool(const double *x, int64_t N, int64_t H, int64_t W, int64_t C,
               int64_t KH, int64_t KW, int64_t stride, int64_t pad, double *y)
{
    int64_t Ho = (H + 2 * pad - KH) / stride + 1;
    int64_t Wo = (W + 2 * pad - KW) / stride + 1;
    if (Ho < 1 || Wo < 1) return -1;
    for (int64_t n = 0; n < N; n++)
        for (int64_t p = 0; p < Ho; p++)
            for (int64_t q = 0; q < Wo; q++)
                for (int64_t c = 0; c < C; c++) {
                    double s = 0.0;
                    for (int64_t r = 0; r < KH; r++)
                        for (int64_t u = 0; u < KW; u++) {
                            int64_t h = p * stride - pad + r, w = q * stride - pad + u;
                            if (h < 0 || h >= H || w < 0 || w >= W) continue;
                            s += x[((n * H + h) * W + w) * C + c];
                        }
                    y[((n * Ho + p) * Wo + q) * C + c] = s / (double)(KH * KW);
                }
    return 0;
}

/* Row softmax: y[i][j] = exp(x[i][j] - max_j x[i]) / sum_j exp(x[i][j] - max_j x[i]). */
int or_softmax_rows(const double *x, int64_t rows, int64_t n, double scale, double *y)
{
    for (int64_t i = 0; i < rows; i++) {
        double m = -INFINITY;
        for (int64_t j = 0; j < n; j++) if (scale * x[i * n + j] > m) m = scale * x[i * n + j];
        double s = 0.0;
        for (int64_t j = 0; j < n; j++) s += exp(scale * x[i * n + j] - m);
        for (int64_t j = 0; j < n; j++) y[i * n + j] = exp(scale * x[i * n + j] - m) / s;
    }
    return 0;
}

/*
 * Layer normalisation of each row (biased variance), optionally after adding
 * a residual row:  v = x (+ r);  y = (v - mean(v)) / sqrt(var(v) + eps) * gamma + beta.
 */
int or_layernorm_rows(const double *x, const double *res, int64_t rows, int64_t n,
                      const double *gamma, const double *beta, double eps, double *y)
{
    double *v = (double *)malloc(sizeof(double) * (size_t)n);
    for (int64_t i = 0; i < rows; i++) {
        double mu = 0.0;
        for (int64_t j = 0; j < n; j++) {
            v[j] = x[i * n + j] + (res ? res[i * n + j] : 0.0);
            mu += v[j];
        }
        mu /= (double)n;
        double var = 0.0;
        for (int64_t j = 0; j < n; j++) var += (v[j] - mu) * (v[j] - mu);
        var /= (double)n;
        double inv = 1.0 / sqrt(var + eps);
        for (int64_t j = 0; j < n; j++) y[i * n + j] = (v[j] - mu) * inv * gamma[j] + beta[j];
    }
    free(v);
    return 0;
}

/* Host threads for the convolution and the matrix products (n >= 1); returns the count now in
 * force.  n = 0 only reports it. */
int or_set_threads(int n)
{
    if (n > 0) omp_set_num_threads(n);
    return omp_get_max_threads();
}
