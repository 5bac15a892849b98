// Scored compositional routing (Section 4.2's path score, Section 4.3's TopK over the
// active path set and source-grouped dispatch).
//
//   s_ij = g_base_i + b_ij + lambda g_tgt_j, over the active set A = {(i,j) : m_ij = 1},
//   m_ii = 1; the K best paths, ties to the lower i*n + j; beta = softmax of their scores.
//
// The active set is materialised once per layer (layout_kernel: the (i, j) of every
// active pair in ascending i*n + j, with its bias b_ij), so that the per-token router
// only walks the active pairs. The score is formed as fmaf(lambda, g_tgt_j,
// g_base_i + b_ij) in float32.
//
// route_scored_kernel: W waves per token. Each lane keeps the 8 best keys of the pairs it
// visits; K rounds of a wave-wide maximum give each wave's winners, and the token's first
// wave merges the waves' winners the same way. A key
// is (orderable score) << 32 | (~(i*n + j)), so a larger key is a larger score or, for an
// equal score, a lower flattened index. The token's distinct sources and targets
// (ascending expert order), the path bits over (source slot, target slot) and the
// grouped weights follow from the K winners.
#include "internal.h"

namespace pcm {
namespace {


// float -> unsigned key with the same order (inputs finite; -0 is folded into +0 first)
__device__ inline uint32_t orderable(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ inline float from_orderable(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Active pairs of the [n,n] mask (diagonal always active) in ascending i*n + j, one row
// per step of a single 256-thread workgroup (one thread per column).
__global__ __launch_bounds__(256) void layout_kernel(const uint8_t* __restrict__ mask,
                                                     const float* __restrict__ bias, int n,
                                                     int32_t* __restrict__ count,
                                                     uint32_t* __restrict__ pair,
                                                     float* __restrict__ pair_bias) {
    __shared__ int wave_tot[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int base = 0;
    for (int i = 0; i < n; ++i) {
        const int j = tid;
        const bool act = j < n && (j == i || mask[(int64_t)i * n + j] != 0);
        const uint64_t bal = __ballot(act);
        if (lane == 0) wave_tot[wave] = __popcll(bal);
        __syncthreads();
        int off = base, total = 0;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            if (w < wave) off += wave_tot[w];
            total += wave_tot[w];
        }
        if (act) {
            const int pos = off + __popcll(bal & ((1ull << lane) - 1ull));
            pair[pos] = ((uint32_t)i << 16) | (uint32_t)j;
            pair_bias[pos] = bias[(int64_t)i * n + j];
        }
        base += total;
        __syncthreads();
    }
    if (tid == 0) *count = base;
}

// Insert key into a descending list of N keys (static indices only).
template <int N>
__device__ inline void insert_key(uint64_t (&best)[N], uint64_t key) {
    if (key > best[N - 1]) {
        best[N - 1] = key;
#pragma unroll
        for (int q = N - 1; q > 0; --q)
            if (best[q] > best[q - 1]) {
                const uint64_t tmp = best[q];
                best[q] = best[q - 1];
                best[q - 1] = tmp;
            }
    }
}

// K rounds of a wave-wide maximum over the lanes' descending lists; the lane holding the
// winner pops it. Returns the winners in out[0..K) (the same on every lane).
template <int N>
__device__ inline void wave_topk(uint64_t (&best)[N], int K, uint64_t (&out)[kMaxK]) {
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) {
        out[r] = 0;
        if (r >= K) continue;
        const uint64_t m = wave_max_u64(best[0]);
        if (best[0] == m) {
#pragma unroll
            for (int q = 0; q < N - 1; ++q) best[q] = best[q + 1];
            best[N - 1] = 0;
        }
        out[r] = m;
    }
}

// TPB tokens per workgroup, W waves per token: the waves of a token split its active
// pairs, each keeps its K best, and the token's first wave merges the W*K candidates and
// writes the token's outputs.
template <int W, int TPB>
__global__ __launch_bounds__(W * TPB * 64) void route_scored_kernel(
    const float* __restrict__ g_base, const float* __restrict__ g_tgt, float lambda,
    const int32_t* __restrict__ count_p, const uint32_t* __restrict__ pair,
    const float* __restrict__ pair_bias, int64_t T, int n, int K, int32_t* __restrict__ sel_pair,
    float* __restrict__ sel_score, int32_t* __restrict__ n_src_out, int32_t* __restrict__ src_out,
    int32_t* __restrict__ n_tgt_out, int32_t* __restrict__ tgt_out, uint64_t* __restrict__ bits_out,
    float* __restrict__ beta_out) {
    __shared__ float gb_s[TPB][kMaxN], gt_s[TPB][kMaxN];
    __shared__ uint64_t cand[TPB][W * kMaxK];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int slot = wave / W, wt = wave % W, tt = wt * 64 + lane;  // token slot, thread in token
    const int64_t t = (int64_t)blockIdx.x * TPB + slot;
    const bool active = t < T;
    for (int x = tt; x < n; x += W * 64) {
        gb_s[slot][x] = active ? g_base[t * n + x] : 0.0f;
        gt_s[slot][x] = active ? g_tgt[t * n + x] : 0.0f;
    }
    __syncthreads();

    // this lane's 8 best keys over its share of the active pairs, descending
    uint64_t best[kMaxK];
#pragma unroll
    for (int q = 0; q < kMaxK; ++q) best[q] = 0;  // below every real key
    const int count = active ? *count_p : 0;
    for (int p = tt; p < count; p += W * 64) {
        const uint32_t pr = pair[p];
        const int i = (int)(pr >> 16), j = (int)(pr & 0xFFFFu);
        float s = __builtin_fmaf(lambda, gt_s[slot][j], gb_s[slot][i] + pair_bias[p]);
        s = (s == 0.0f) ? 0.0f : s;
        insert_key(best, ((uint64_t)orderable(s) << 32) |
                             (uint32_t)(0xFFFFFFFFu - (uint32_t)(i * n + j)));
    }
    uint64_t win[kMaxK];
    wave_topk(best, K, win);
    if (W > 1) {
#pragma unroll
        for (int r = 0; r < kMaxK; ++r)
            if (lane == r) cand[slot][wt * kMaxK + r] = win[r];
        __syncthreads();
        if (wt != 0) return;  // no barrier follows
        // the token's first wave merges the W*8 candidates, (W*8 + 63) / 64 per lane
        constexpr int PER = (W * kMaxK + 63) / 64;
        uint64_t c[PER];
#pragma unroll
        for (int q = 0; q < PER; ++q) {
            const int idx = lane + 64 * q;
            c[q] = idx < W * kMaxK ? cand[slot][idx] : 0;
        }
#pragma unroll
        for (int q = 1; q < PER; ++q)   // keep each lane's list descending
#pragma unroll
            for (int v = q; v > 0; --v)
                if (c[v] > c[v - 1]) {
                    const uint64_t tmp = c[v];
                    c[v] = c[v - 1];
                    c[v - 1] = tmp;
                }
        wave_topk(c, K, win);
    }
    if (!active) return;
    int src[kMaxK], tgt[kMaxK];
    float score[kMaxK];
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) {
        const uint32_t flat = 0xFFFFFFFFu - (uint32_t)win[r];
        src[r] = r < K ? (int)(flat / (uint32_t)n) : 0;
        tgt[r] = r < K ? (int)(flat % (uint32_t)n) : 0;
        score[r] = r < K ? from_orderable((uint32_t)(win[r] >> 32)) : 0.0f;
    }

    // weights: softmax of the selected scores (the first is the largest)
    float w[kMaxK], sum = 0.0f;
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) {
        w[r] = r < K ? expf(score[r] - score[0]) : 0.0f;
        sum += w[r];
    }
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) w[r] = w[r] / sum;

    // distinct sources / targets in ascending expert order: the slot of path r is the
    // number of distinct values below its own
    int sslot[kMaxK], tslot[kMaxK], ns = 0, nt = 0;
    bool sfirst[kMaxK], tfirst[kMaxK];
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) {
        sfirst[r] = r < K;
        tfirst[r] = r < K;
#pragma unroll
        for (int q = 0; q < kMaxK; ++q)
            if (q < r) {
                if (src[q] == src[r]) sfirst[r] = false;
                if (tgt[q] == tgt[r]) tfirst[r] = false;
            }
        ns += sfirst[r] ? 1 : 0;
        nt += tfirst[r] ? 1 : 0;
    }
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) {
        int a = 0, b = 0;
#pragma unroll
        for (int q = 0; q < kMaxK; ++q) {
            a += (sfirst[q] && src[q] < src[r]) ? 1 : 0;
            b += (tfirst[q] && tgt[q] < tgt[r]) ? 1 : 0;
        }
        sslot[r] = a;
        tslot[r] = b;
    }
    uint64_t bits = 0;
#pragma unroll
    for (int r = 0; r < kMaxK; ++r)
        if (r < K) bits |= 1ull << (sslot[r] * K + tslot[r]);

    // lane l writes entry l of each per-token array
    int e_src = -1, e_tgt = -1, pr = 0;
    float sc = 0.0f, bg = 0.0f;
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) {
        if (r >= K) continue;
        if (sfirst[r] && sslot[r] == lane) e_src = src[r];
        if (tfirst[r] && tslot[r] == lane) e_tgt = tgt[r];
        if (r == lane) {
            pr = src[r] * n + tgt[r];
            sc = score[r];
        }
        if (sslot[r] * K + tslot[r] == lane) bg = w[r];
    }
    if (lane < K) {
        sel_pair[t * K + lane] = pr;
        sel_score[t * K + lane] = sc;
        src_out[t * K + lane] = e_src;
        tgt_out[t * K + lane] = e_tgt;
    }
    if (lane < K * K) beta_out[t * K * K + lane] = bg;
    if (lane == 0) {
        n_src_out[t] = ns;
        n_tgt_out[t] = nt;
        bits_out[t] = bits;
    }
}

}  // namespace

hipError_t launch_path_layout(const uint8_t* mask, const float* bias, int n, int32_t* count,
                              uint32_t* pair, float* pair_bias, hipStream_t s) {
    layout_kernel<<<1, 256, 0, s>>>(mask, bias, n, count, pair, pair_bias);
    return hipGetLastError();
}

hipError_t launch_route_scored(const float* g_base, const float* g_tgt, float lambda,
                               const int32_t* count, const uint32_t* pair, const float* pair_bias,
                               int64_t T, int n, int K, int32_t* sel_pair, float* sel_score,
                               int32_t* n_src, int32_t* src_expert, int32_t* n_tgt,
                               int32_t* tgt_expert, uint64_t* bits, float* beta, hipStream_t s) {
    if (T == 0) return hipSuccess;
    // few tokens: 16 waves share each token's active pairs; many: one wave per token
    if (T <= 512)
        route_scored_kernel<16, 1><<<(unsigned)T, 16 * 64, 0, s>>>(
            g_base, g_tgt, lambda, count, pair, pair_bias, T, n, K, sel_pair, sel_score, n_src,
            src_expert, n_tgt, tgt_expert, bits, beta);
    else
        route_scored_kernel<1, 4><<<(unsigned)ceil_div(T, 4), 4 * 64, 0, s>>>(
            g_base, g_tgt, lambda, count, pair, pair_bias, T, n, K, sel_pair, sel_score, n_src,
            src_expert, n_tgt, tgt_expert, bits, beta);
    return hipGetLastError();
}

}  // namespace pcm
