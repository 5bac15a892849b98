/*
 * pcomoe_oracle.c -- plain, slow CPU oracle of the path-compositional MoE layer
 * (PCoMoE, arXiv 2609.01024).
 *
 * TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
 * baseline leg may load this library. The GPU library never calls it, and the two
 * share no source, header, table or helper.
 *
 * Everything is evaluated in double precision from the same float32 / bfloat16
 * inputs the GPU receives (bfloat16 values are widened exactly). Nothing is blocked,
 * fused or reordered beyond what the definitions state:
 *
 *   top-k routing and weights  (Section 2, vanilla MoE equation y = sum_e alpha_e F_e(h))
 *   SwiGLU expert              (Section 2, F_e(h) = W_down (SiLU(W_gate h) * (W_up h)))
 *   expansion / projection     (Section 4.1, U_e(h) and D_e(z) = W_down z)
 *   compositional path         (Section 4.1, P_ij(h) = D_j(U_i(h)))
 *   path-level aggregation     (Section 4.1, y = sum over Pi(h) of beta_ij P_ij(h))
 *   active mask with m_ii = 1  (Section 4.2, last two paragraphs; Section 4.3)
 *   source-grouped form        (Section 4.3, y = sum_{i in S} sum_{j in T_i} beta_ij D_j(U_i))
 *
 * Readings taken where the paper is silent (each is listed in the design notes):
 *   - the token's candidate paths are the ordered pairs (a, b) of its top-k slots
 *     whose experts (e_a, e_b) the mask allows; the diagonal is always allowed;
 *   - top-k is ordered by logit descending, ties to the lower expert id, selected on
 *     the float32 logits;
 *   - alpha (router weights) are the softmax over the k selected logits, i.e. the
 *     full softmax renormalised over the top-k;
 *   - beta is "source conditional" by default: beta_ab = p_a p_b / sum_{b' in T_a} p_b'.
 *     With a diagonal-only mask this gives beta_aa = p_a (the vanilla layer, as
 *     Section 4.1 requires); with every pair allowed it is the product p_a p_b.
 *     The product and globally normalised products are kept as alternatives.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F32 = 0, ORC_BF16 = 1 };
enum { ORC_BETA_SRC_COND = 0, ORC_BETA_PRODUCT = 1, ORC_BETA_GLOBAL = 2 };
enum { ORC_OK = 0, ORC_BAD_ARG = 1, ORC_NO_MEM = 2 };

#define ORC_MAX_K 8

/* One element of a float32 or bfloat16 array, widened to double. A bfloat16 is
 * the upper 16 bits of a float32, so widening is exact. */
static double elem(const void* base, int dtype, int64_t i) {
    if (dtype == ORC_F32) return (double)((const float*)base)[i];
    uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

int pcmo_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void pcmo_set_num_threads(int nt) {
#ifdef _OPENMP
    if (nt > 0) omp_set_num_threads(nt);
#else
    (void)nt;
#endif
}

/* Top-k expert selection of one token (the selected set E(h) of the vanilla layer,
 * Section 2) and the routing weights alpha_e renormalised over the selected set.
 * Slot a holds the a-th largest logit; equal logits go to the lower expert id
 * (only a strictly larger logit displaces the current best). */
static void topk_one(const float* l, int n, int k, int32_t* ids, double* p) {
    unsigned char* taken = (unsigned char*)calloc((size_t)n, 1);
    for (int a = 0; a < k; ++a) {
        int best = -1;
        for (int e = 0; e < n; ++e) {
            if (taken[e]) continue;
            if (best < 0 || l[e] > l[best]) best = e;
        }
        ids[a] = best;
        taken[best] = 1;
    }
    free(taken);
    /* softmax over the k selected logits, shifted by the largest for range safety */
    double top = (double)l[ids[0]], s = 0.0;
    for (int a = 0; a < k; ++a) s += exp((double)l[ids[a]] - top);
    for (int a = 0; a < k; ++a) p[a] = exp((double)l[ids[a]] - top) / s;
}

/* Active paths of one token and their weights.
 * Pi(h) = {(a, b) : a == b or mask[e_a][e_b] == 1}: the mask restricted to the token's
 * selected experts, with m_ii = 1 hard-coded (Section 4.2) so every diagonal path
 * survives (Section 4.3's fallback). Bit a*k + b of *bits marks (a, b).
 * beta has k*k entries, row a = source slot, column b = target slot, 0 off-path. */
static void paths_one(const int32_t* ids, const double* p, const uint8_t* mask, int n, int k,
                      int mode, uint64_t* bits, double* beta) {
    uint64_t b64 = 0;
    for (int a = 0; a < k; ++a)
        for (int b = 0; b < k; ++b)
            if (a == b || mask[(int64_t)ids[a] * n + ids[b]]) b64 |= (uint64_t)1 << (a * k + b);
    *bits = b64;
    for (int i = 0; i < k * k; ++i) beta[i] = 0.0;
    double global = 0.0;
    for (int a = 0; a < k; ++a)
        for (int b = 0; b < k; ++b)
            if (b64 >> (a * k + b) & 1) global += p[a] * p[b];
    for (int a = 0; a < k; ++a) {
        double src = 0.0; /* sum of p over the targets T_a of source a */
        for (int b = 0; b < k; ++b)
            if (b64 >> (a * k + b) & 1) src += p[b];
        for (int b = 0; b < k; ++b) {
            if (!(b64 >> (a * k + b) & 1)) continue;
            double prod = p[a] * p[b];
            if (mode == ORC_BETA_SRC_COND) beta[a * k + b] = prod / src;
            else if (mode == ORC_BETA_PRODUCT) beta[a * k + b] = prod;
            else beta[a * k + b] = prod / global;
        }
    }
}

static int check_common(int64_t T, int n, int k) {
    if (T < 0 || n < 1 || k < 1 || k > n || k > ORC_MAX_K) return ORC_BAD_ARG;
    return ORC_OK;
}

/* Routing for T tokens: topk_ids[T,k], topk_w[T,k] (double). */
int pcmo_route(const float* logits, int64_t T, int n, int k, int32_t* topk_ids, double* topk_w) {
    int st = check_common(T, n, k);
    if (st) return st;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) topk_one(logits + t * n, n, k, topk_ids + t * k, topk_w + t * k);
    return ORC_OK;
}

/* Path bits [T] and beta [T,k,k] from routing outputs and the [n,n] mask. */
int pcmo_paths(const int32_t* topk_ids, const double* topk_w, const uint8_t* mask, int64_t T, int n,
               int k, int beta_mode, uint64_t* path_bits, double* beta) {
    int st = check_common(T, n, k);
    if (st) return st;
    if (beta_mode < 0 || beta_mode > 2) return ORC_BAD_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t)
        paths_one(topk_ids + t * k, topk_w + t * k, mask, n, k, beta_mode, path_bits + t,
                  beta + t * k * k);
    return ORC_OK;
}

/* Grouped dispatch layout (Section 2: tokens grouped by expert for batched execution;
 * Section 4.3: the expansion of source i runs once per (token, source)).
 * Rows are the (token, slot) pairs in order of (expert ascending, token ascending):
 * a counting sort that walks tokens in ascending order, so it is stable.
 * expert_offsets[n+1]: first row of each expert; row_token[R], row_slot[R]: the pair
 * held by each row; row_of[T*k]: the row of each pair. */
int pcmo_permute(const int32_t* topk_ids, int64_t T, int n, int k, int32_t* expert_offsets,
                 int32_t* row_token, int32_t* row_slot, int32_t* row_of) {
    int st = check_common(T, n, k);
    if (st) return st;
    int64_t* cursor = (int64_t*)calloc((size_t)n + 1, sizeof(int64_t));
    if (!cursor) return ORC_NO_MEM;
    for (int64_t i = 0; i < T * k; ++i) {
        int e = topk_ids[i];
        if (e < 0 || e >= n) { free(cursor); return ORC_BAD_ARG; }
        cursor[e + 1] += 1;
    }
    for (int e = 0; e < n; ++e) cursor[e + 1] += cursor[e];
    for (int e = 0; e <= n; ++e) expert_offsets[e] = (int32_t)cursor[e];
    for (int64_t t = 0; t < T; ++t)
        for (int a = 0; a < k; ++a) {
            int64_t r = cursor[topk_ids[t * k + a]]++;
            row_token[r] = (int32_t)t;
            row_slot[r] = a;
            row_of[t * k + a] = (int32_t)r;
        }
    free(cursor);
    return ORC_OK;
}

static double silu(double v) { return v / (1.0 + exp(-v)); }

/* Expansion side of one expert for one token (Section 4.1):
 * U[f] = SiLU(sum_h Wg[f][h] x[h]) * (sum_h Wu[f][h] x[h]), Wg/Wu are [F,H] row-major. */
static void expansion(int dtype, const void* x, int64_t x_off, const void* wg, const void* wu,
                      int64_t w_off, int H, int F, double* U) {
    for (int f = 0; f < F; ++f) {
        double g = 0.0, u = 0.0;
        int64_t row = w_off + (int64_t)f * H;
        for (int h = 0; h < H; ++h) {
            double xv = elem(x, dtype, x_off + h);
            g += elem(wg, dtype, row + h) * xv;
            u += elem(wu, dtype, row + h) * xv;
        }
        U[f] = silu(g) * u;
    }
}

/* Projection side of one expert (Section 4.1): out[m] = sum_f Wd[m][f] z[f], Wd is [H,F]. */
static void projection(int dtype, const void* wd, int64_t w_off, int H, int F, const double* z,
                       double* out) {
    for (int m = 0; m < H; ++m) {
        double s = 0.0;
        int64_t row = w_off + (int64_t)m * F;
        for (int f = 0; f < F; ++f) s += elem(wd, dtype, row + f) * z[f];
        out[m] = s;
    }
}

/* The layer output of selected tokens, y = sum_{(a,b) in Pi} beta_ab D_{e_b}(U_{e_a}(x_t)),
 * paths visited in lexicographic (a, b) order (Section 4.1's aggregation, grouped by
 * source as in Section 4.3).
 *   reuse = 0: U_{e_a} is re-evaluated for every path (per-path execution);
 *   reuse = 1: U_{e_a} is evaluated once per source and reused (Section 4.3).
 * Both use the same arithmetic, so their results are bit-identical.
 * tokens[ntok] lists the tokens to evaluate; y_out is [ntok, H] double.
 * x [T,H], logits [T,n], w_gate/w_up [n,F,H], w_down [n,H,F], mask [n,n]. */
int pcmo_layer_tokens(int dtype, const void* x, const float* logits, const void* w_gate,
                      const void* w_up, const void* w_down, const uint8_t* mask, int64_t T, int H,
                      int F, int n, int k, int beta_mode, int reuse, const int64_t* tokens,
                      int64_t ntok, double* y_out) {
    int st = check_common(T, n, k);
    if (st) return st;
    if (H < 1 || F < 1 || (dtype != ORC_F32 && dtype != ORC_BF16) || beta_mode < 0 || beta_mode > 2)
        return ORC_BAD_ARG;
    for (int64_t i = 0; i < ntok; ++i)
        if (tokens[i] < 0 || tokens[i] >= T) return ORC_BAD_ARG;
    int failed = 0;
#pragma omp parallel
    {
        double* U = (double*)malloc(sizeof(double) * (size_t)F * (reuse ? k : 1));
        double* P = (double*)malloc(sizeof(double) * (size_t)H);
        if (!U || !P) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t i = 0; i < ntok; ++i) {
                int64_t t = tokens[i];
                int32_t ids[ORC_MAX_K];
                double p[ORC_MAX_K], beta[ORC_MAX_K * ORC_MAX_K];
                uint64_t bits;
                topk_one(logits + t * n, n, k, ids, p);
                paths_one(ids, p, mask, n, k, beta_mode, &bits, beta);
                double* y = y_out + i * H;
                for (int m = 0; m < H; ++m) y[m] = 0.0;
                if (reuse)
                    for (int a = 0; a < k; ++a)
                        expansion(dtype, x, t * H, w_gate, w_up, (int64_t)ids[a] * F * H, H, F,
                                  U + (int64_t)a * F);
                for (int a = 0; a < k; ++a) {
                    for (int b = 0; b < k; ++b) {
                        if (!(bits >> (a * k + b) & 1)) continue;
                        const double* Ua = U + (reuse ? (int64_t)a * F : 0);
                        if (!reuse)
                            expansion(dtype, x, t * H, w_gate, w_up, (int64_t)ids[a] * F * H, H,
                                      F, U);
                        projection(dtype, w_down, (int64_t)ids[b] * H * F, H, F, Ua, P);
                        for (int m = 0; m < H; ++m) y[m] += beta[a * k + b] * P[m];
                    }
                }
            }
        }
        free(U);
        free(P);
    }
    return failed ? ORC_NO_MEM : ORC_OK;
}

/* Expansion rows for stage checks: U_out[i,:] = U_{experts[i]}(x_{tokens[i]}), [nrows, F]. */
int pcmo_expansion_rows(int dtype, const void* x, const void* w_gate, const void* w_up, int64_t T,
                        int H, int F, int n, const int64_t* tokens, const int32_t* experts,
                        int64_t nrows, double* U_out) {
    if (T < 0 || H < 1 || F < 1 || n < 1) return ORC_BAD_ARG;
    for (int64_t i = 0; i < nrows; ++i)
        if (tokens[i] < 0 || tokens[i] >= T || experts[i] < 0 || experts[i] >= n) return ORC_BAD_ARG;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < nrows; ++i)
        expansion(dtype, x, tokens[i] * H, w_gate, w_up, (int64_t)experts[i] * F * H, H, F,
                  U_out + i * F);
    return ORC_OK;
}

/* The always-on shared expert, a plain SwiGLU FFN (Section 2's F_e with its own weights)
 * with weight 1: y_out[i,:] = W_down (SiLU(W_gate x) * (W_up x)) for x = x[tokens[i]].
 * wg/wu are [Fs,H], wd is [H,Fs]. */
int pcmo_dense_swiglu_tokens(int dtype, const void* x, const void* wg, const void* wu,
                             const void* wd, int64_t T, int H, int Fs, const int64_t* tokens,
                             int64_t ntok, double* y_out) {
    if (T < 0 || H < 1 || Fs < 1 || (dtype != ORC_F32 && dtype != ORC_BF16)) return ORC_BAD_ARG;
    for (int64_t i = 0; i < ntok; ++i)
        if (tokens[i] < 0 || tokens[i] >= T) return ORC_BAD_ARG;
    int failed = 0;
#pragma omp parallel
    {
        double* U = (double*)malloc(sizeof(double) * (size_t)Fs);
        if (!U) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t i = 0; i < ntok; ++i) {
                expansion(dtype, x, tokens[i] * H, wg, wu, 0, H, Fs, U);
                projection(dtype, wd, 0, H, Fs, U, y_out + i * H);
            }
        }
        free(U);
    }
    return failed ? ORC_NO_MEM : ORC_OK;
}

/* ---------------------------------------------------------------------------------
 * Scored compositional routing: the router the paper runs at inference.
 *
 *   s_ij = g_base_i + b_ij + lambda g_tgt_j                (Section 4.2, path score)
 *   Pi   = the K highest s_ij over A = {(i, j) : m_ij = 1}, with m_ii = 1
 *                                                          (Section 4.3, TopK over A)
 *   S    = {i : (i, j) in Pi},  T_i = {j : (i, j) in Pi}  (Section 4.3)
 *   y    = sum_{i in S} sum_{j in T_i} beta_ij D_j(U_i(h)) (Section 4.3)
 *
 * Readings where the paper is silent (listed in the design notes):
 *   - the score is formed in float32 as fmaf(lambda, g_tgt_j, g_base_i + b_ij), so that
 *     every implementation takes the selection on identical values;
 *   - equal scores go to the lower flattened index i*n + j;
 *   - beta is the softmax of the K selected scores;
 *   - K <= n, which keeps K <= |A| because every diagonal pair is active.
 * --------------------------------------------------------------------------------- */

static float path_score(const float* gb, const float* gt, const float* bias, float lambda, int n,
                        int i, int j) {
    return fmaf(lambda, gt[j], gb[i] + bias[(int64_t)i * n + j]);
}

/* One token: src[K], tgt[K] and score[K] of the selected paths in selection order
 * (score descending, ties to the lower i*n + j), beta[K] their softmax weights. */
static int route_scored_one(const float* gb, const float* gt, float lambda, const float* bias,
                            const uint8_t* mask, int n, int K, int32_t* src, int32_t* tgt,
                            float* score, double* beta) {
    unsigned char* taken = (unsigned char*)calloc((size_t)n * n, 1);
    if (!taken) return ORC_NO_MEM;
    for (int r = 0; r < K; ++r) {
        int bi = -1, bj = -1;
        float bs = 0.0f;
        for (int i = 0; i < n; ++i)
            for (int j = 0; j < n; ++j) {
                if (i != j && !mask[(int64_t)i * n + j]) continue;   /* outside A */
                if (taken[(int64_t)i * n + j]) continue;
                float s = path_score(gb, gt, bias, lambda, n, i, j);
                if (bi < 0 || s > bs) { bi = i; bj = j; bs = s; }    /* first of equals wins */
            }
        src[r] = bi;
        tgt[r] = bj;
        score[r] = bs;
        taken[(int64_t)bi * n + bj] = 1;
    }
    free(taken);
    double top = (double)score[0], sum = 0.0;
    for (int r = 0; r < K; ++r) sum += exp((double)score[r] - top);
    for (int r = 0; r < K; ++r) beta[r] = exp((double)score[r] - top) / sum;
    return ORC_OK;
}

static int check_scored(int64_t T, int n, int K) {
    if (T < 0 || n < 1 || K < 1 || K > n || K > ORC_MAX_K) return ORC_BAD_ARG;
    return ORC_OK;
}

/* Routing of T tokens: sel_src[T,K], sel_tgt[T,K], sel_score[T,K] (float), beta[T,K].
 * g_base, g_tgt [T,n]; bias [n,n]; mask [n,n] (row = source i, column = target j). */
int pcmo_route_scored(const float* g_base, const float* g_tgt, float lambda, const float* bias,
                      const uint8_t* mask, int64_t T, int n, int K, int32_t* sel_src,
                      int32_t* sel_tgt, float* sel_score, double* beta) {
    int st = check_scored(T, n, K);
    if (st) return st;
    int failed = 0;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t)
        if (route_scored_one(g_base + t * n, g_tgt + t * n, lambda, bias, mask, n, K,
                             sel_src + t * K, sel_tgt + t * K, sel_score + t * K, beta + t * K))
#pragma omp atomic write
            failed = 1;
    return failed ? ORC_NO_MEM : ORC_OK;
}

/* Source and target groups of each token's selected paths (Section 4.3): the sources S
 * and the targets, each in ascending expert order (n_src[t], srcs[t, 0..n_src), and
 * n_tgt[t], tgts[t, 0..n_tgt)); bit a*K + b of bits[t] marks the path (srcs[a], tgts[b])
 * and beta_g[t, a, b] is its weight (0 off-path). */
int pcmo_group_scored(const int32_t* sel_src, const int32_t* sel_tgt, const double* beta, int64_t T,
                      int K, int32_t* n_src, int32_t* srcs, int32_t* n_tgt, int32_t* tgts,
                      uint64_t* bits, double* beta_g) {
    if (T < 0 || K < 1 || K > ORC_MAX_K) return ORC_BAD_ARG;
    for (int64_t t = 0; t < T; ++t) {
        const int32_t* ps = sel_src + t * K;
        const int32_t* pt = sel_tgt + t * K;
        int32_t* S = srcs + t * K;
        int32_t* G = tgts + t * K;
        int ns = 0, ng = 0;
        for (int r = 0; r < K; ++r) {         /* distinct values, kept sorted ascending */
            int v = ps[r], pos = 0, dup = 0;
            for (int q = 0; q < ns; ++q) { if (S[q] == v) dup = 1; if (S[q] < v) pos = q + 1; }
            if (!dup) { for (int q = ns; q > pos; --q) S[q] = S[q - 1]; S[pos] = v; ++ns; }
            v = pt[r]; pos = 0; dup = 0;
            for (int q = 0; q < ng; ++q) { if (G[q] == v) dup = 1; if (G[q] < v) pos = q + 1; }
            if (!dup) { for (int q = ng; q > pos; --q) G[q] = G[q - 1]; G[pos] = v; ++ng; }
        }
        for (int q = ns; q < K; ++q) S[q] = -1;
        for (int q = ng; q < K; ++q) G[q] = -1;
        n_src[t] = ns;
        n_tgt[t] = ng;
        uint64_t b64 = 0;
        double* bg = beta_g + t * K * K;
        for (int q = 0; q < K * K; ++q) bg[q] = 0.0;
        for (int r = 0; r < K; ++r) {
            int a = 0, b = 0;
            while (S[a] != ps[r]) ++a;
            while (G[b] != pt[r]) ++b;
            b64 |= (uint64_t)1 << (a * K + b);
            bg[a * K + b] = beta[t * K + r];
        }
        bits[t] = b64;
    }
    return ORC_OK;
}

/* Grouped dispatch with a variable number of entries per token: token t contributes
 * counts[t] <= K entries ids[t, 0..counts[t]) (distinct experts). Rows are ordered by
 * (expert ascending, token ascending); row_of[t, a] = -1 for a >= counts[t]. */
int pcmo_permute_var(const int32_t* ids, const int32_t* counts, int64_t T, int n, int K,
                     int32_t* expert_offsets, int32_t* row_token, int32_t* row_slot,
                     int32_t* row_of) {
    if (T < 0 || n < 1 || K < 1) return ORC_BAD_ARG;
    int64_t* cursor = (int64_t*)calloc((size_t)n + 1, sizeof(int64_t));
    if (!cursor) return ORC_NO_MEM;
    for (int64_t t = 0; t < T; ++t) {
        if (counts[t] < 0 || counts[t] > K) { free(cursor); return ORC_BAD_ARG; }
        for (int a = 0; a < counts[t]; ++a) {
            int e = ids[t * K + a];
            if (e < 0 || e >= n) { free(cursor); return ORC_BAD_ARG; }
            cursor[e + 1]++;
        }
    }
    for (int e = 0; e < n; ++e) cursor[e + 1] += cursor[e];
    for (int e = 0; e <= n; ++e) expert_offsets[e] = (int32_t)cursor[e];
    for (int64_t t = 0; t < T; ++t)
        for (int a = 0; a < K; ++a) {
            if (a >= counts[t]) { row_of[t * K + a] = -1; continue; }
            int64_t r = cursor[ids[t * K + a]]++;
            row_token[r] = (int32_t)t;
            row_slot[r] = (int32_t)a;
            row_of[t * K + a] = (int32_t)r;
        }
    free(cursor);
    return ORC_OK;
}

/* Layer output of selected tokens under scored routing:
 * y = sum over the selected paths r of beta_r D_{tgt_r}(U_{src_r}(x_t)), visited in
 * selection order.
 *   reuse = 0: U is re-evaluated for every path;
 *   reuse = 1: U is evaluated once per distinct source and reused (Section 4.3).
 * Both use the same arithmetic, so their results are bit-identical. */
int pcmo_layer_scored_tokens(int dtype, const void* x, const float* g_base, const float* g_tgt,
                             float lambda, const float* bias, const uint8_t* mask,
                             const void* w_gate, const void* w_up, const void* w_down, int64_t T,
                             int H, int F, int n, int K, int reuse, const int64_t* tokens,
                             int64_t ntok, double* y_out) {
    int st = check_scored(T, n, K);
    if (st) return st;
    if (H < 1 || F < 1 || (dtype != ORC_F32 && dtype != ORC_BF16)) return ORC_BAD_ARG;
    for (int64_t i = 0; i < ntok; ++i)
        if (tokens[i] < 0 || tokens[i] >= T) return ORC_BAD_ARG;
    int failed = 0;
#pragma omp parallel
    {
        double* U = (double*)malloc(sizeof(double) * (size_t)F * K);
        double* P = (double*)malloc(sizeof(double) * (size_t)H);
        if (!U || !P) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t i = 0; i < ntok; ++i) {
                int64_t t = tokens[i];
                int32_t src[ORC_MAX_K], tgt[ORC_MAX_K], have[ORC_MAX_K];
                float score[ORC_MAX_K];
                double beta[ORC_MAX_K];
                if (route_scored_one(g_base + t * n, g_tgt + t * n, lambda, bias, mask, n, K, src,
                                     tgt, score, beta)) {
#pragma omp atomic write
                    failed = 1;
                    continue;
                }
                double* y = y_out + i * H;
                for (int m = 0; m < H; ++m) y[m] = 0.0;
                int nhave = 0;
                for (int r = 0; r < K; ++r) {
                    const double* Ui = U;
                    if (reuse) {
                        int slot = -1;
                        for (int q = 0; q < nhave; ++q) if (have[q] == src[r]) slot = q;
                        if (slot < 0) {
                            slot = nhave++;
                            have[slot] = src[r];
                            expansion(dtype, x, t * H, w_gate, w_up, (int64_t)src[r] * F * H, H, F,
                                      U + (int64_t)slot * F);
                        }
                        Ui = U + (int64_t)slot * F;
                    } else {
                        expansion(dtype, x, t * H, w_gate, w_up, (int64_t)src[r] * F * H, H, F, U);
                    }
                    projection(dtype, w_down, (int64_t)tgt[r] * H * F, H, F, Ui, P);
                    for (int m = 0; m < H; ++m) y[m] += beta[r] * P[m];
                }
            }
        }
        free(U);
        free(P);
    }
    return failed ? ORC_NO_MEM : ORC_OK;
}

/* Router scores (Section 2: the router scores each expert from the hidden state h):
 * logits[t][e] = sum_h x[t][h] W_r[e][h], double precision, h ascending.
 * x [T,H] and w_router [n,H] float32 or bfloat16 (widened exactly). */
int pcmo_router_logits(int dtype, const void* x, const void* w_router, int64_t T, int H, int n,
                       double* logits) {
    if (T < 0 || H < 1 || n < 1 || (dtype != ORC_F32 && dtype != ORC_BF16)) return ORC_BAD_ARG;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t)
        for (int e = 0; e < n; ++e) {
            double s = 0.0;
            for (int h = 0; h < H; ++h)
                s += elem(x, dtype, t * H + h) * elem(w_router, dtype, (int64_t)e * H + h);
            logits[t * n + e] = s;
        }
    return ORC_OK;
}
