// Path table and grouped dispatch layout (Section 4.2: inactive paths are masked out
// before weighting, with m_ii = 1; Section 4.3: dispatch metadata grouped by expansion
// source so that each (token, source) expansion runs once).
//
// Per token (one thread each): the active paths Pi = {(a,b): a == b or m[e_a][e_b]}, their
// weights beta, and the token's k rows. Rows are ordered by (expert, token); the rank of a
// row inside its expert is found without atomics whose order matters:
//   - each wave of 64 tokens ORs its lane bit into words[wave][e] for each selected e
//     (OR is order-independent, so the words are deterministic);
//   - rows of e before token (wave, lane) = rows of e in earlier blocks (a scan over
//     block counts) + in earlier waves of this block (popcounts) + popcount(words[wave][e]
//     & lanes below this one).
// T <= 256 runs as one fused launch; larger T as count / scan / scatter launches.
#include "internal.h"

namespace pcm {

namespace {

constexpr int kWaves = kPathBlock / 64;

enum Phase { kFused = 0, kCount = 1, kScatter = 2 };

struct PathSmem {
    unsigned long long words[kWaves][kMaxN];
    int prefix[kWaves][kMaxN];
    int scan[kMaxN];
};

// Exclusive scan of smem.scan[0..n) in place; returns the total to every thread.
__device__ int block_exclusive_scan(int* scan, int n) {
    const int tid = threadIdx.x;
    int own = (tid < n) ? scan[tid] : 0;
    for (int d = 1; d < kMaxN; d <<= 1) {
        int v = (tid < kMaxN && tid >= d) ? scan[tid - d] : 0;
        __syncthreads();
        if (tid < kMaxN) scan[tid] += v;
        __syncthreads();
    }
    const int total = scan[kMaxN - 1];
    __syncthreads();
    if (tid < kMaxN) scan[tid] -= own;
    __syncthreads();
    return total;
}

template <int PH>
__global__ __launch_bounds__(kPathBlock) void paths_kernel(
    const int32_t* __restrict__ ids, const float* __restrict__ w, const uint8_t* __restrict__ mask,
    int64_t T, int n, int k, int beta_mode, uint64_t* __restrict__ bits_out,
    float* __restrict__ beta_out, int32_t* __restrict__ offsets, int32_t* __restrict__ row_token,
    int32_t* __restrict__ row_slot, int32_t* __restrict__ row_of, int32_t* __restrict__ block_counts) {
    __shared__ PathSmem sm;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    for (int i = tid; i < kWaves * kMaxN; i += kPathBlock) (&sm.words[0][0])[i] = 0ull;
    __syncthreads();

    const int64_t t = (int64_t)blockIdx.x * kPathBlock + tid;
    const bool valid = t < T;
    int e[kMaxK];
#pragma unroll
    for (int a = 0; a < kMaxK; ++a) {
        int v = (valid && a < k) ? ids[t * k + a] : 0;
        e[a] = v < 0 ? 0 : (v >= n ? n - 1 : v);
    }
    if (valid) {
        if (PH != kScatter) {
            float p[kMaxK];
#pragma unroll
            for (int a = 0; a < kMaxK; ++a) p[a] = a < k ? w[t * k + a] : 0.0f;
            // every (a, b) entry is loaded (e[] is always a valid id), so the 64 loads are
            // issued together instead of one dependent load per branch
            uint8_t mv[kMaxK][kMaxK];
#pragma unroll
            for (int a = 0; a < kMaxK; ++a)
#pragma unroll
                for (int b = 0; b < kMaxK; ++b) mv[a][b] = mask[(int64_t)e[a] * n + e[b]];
            uint64_t bits = 0;
#pragma unroll
            for (int a = 0; a < kMaxK; ++a)
#pragma unroll
                for (int b = 0; b < kMaxK; ++b)
                    if (a < k && b < k && (a == b || mv[a][b])) bits |= 1ull << (a * k + b);
            bits_out[t] = bits;
            float global = 0.0f;
#pragma unroll
            for (int a = 0; a < kMaxK; ++a)
#pragma unroll
                for (int b = 0; b < kMaxK; ++b)
                    if (a < k && b < k && ((bits >> (a * k + b)) & 1))
                        global = fmaf(p[a], p[b], global);  // explicit: one rounding per term
            float* bt = beta_out + t * k * k;
#pragma unroll
            for (int a = 0; a < kMaxK; ++a) {
                if (a >= k) break;
                float src = 0.0f;  // sum of p over the targets of source a
#pragma unroll
                for (int b = 0; b < kMaxK; ++b)
                    if (b < k && ((bits >> (a * k + b)) & 1)) src += p[b];
#pragma unroll
                for (int b = 0; b < kMaxK; ++b) {
                    if (b >= k) break;
                    float v = 0.0f;
                    if ((bits >> (a * k + b)) & 1) {
                        // p_a (p_b / src) rather than a reciprocal: stays exact (beta_aa = p_a
                        // for a source whose only target is itself) when p is subnormal
                        v = beta_mode == 0 ? p[a] * (p[b] / src)
                                           : (beta_mode == 1 ? p[a] * p[b] : p[a] * p[b] / global);
                    }
                    bt[a * k + b] = v;
                }
            }
        }
#pragma unroll
        for (int a = 0; a < kMaxK; ++a)
            if (a < k) atomicOr(&sm.words[wave][e[a]], 1ull << lane);
    }
    __syncthreads();

    // rows of each expert in the earlier waves of this block
    for (int x = tid; x < kMaxN; x += kPathBlock) {
        int run = 0;
        if (x < n) {
#pragma unroll
            for (int v = 0; v < kWaves; ++v) {
                sm.prefix[v][x] = run;
                run += __popcll(sm.words[v][x]);
            }
        }
        sm.scan[x] = run;
    }
    __syncthreads();

    if (PH == kCount) {
        for (int x = tid; x < n; x += kPathBlock) block_counts[(int64_t)blockIdx.x * n + x] = sm.scan[x];
        return;
    }
    if (PH == kFused) {
        const int total = block_exclusive_scan(sm.scan, n);
        for (int x = tid; x < n; x += kPathBlock) offsets[x] = sm.scan[x];
        if (tid == 0) offsets[n] = total;
    } else {
        for (int x = tid; x < n; x += kPathBlock) sm.scan[x] = block_counts[(int64_t)blockIdx.x * n + x];
        __syncthreads();
    }
    if (valid) {
        const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
        for (int a = 0; a < kMaxK; ++a) {
            if (a >= k) break;
            const int x = e[a];
            const int pos = sm.scan[x] + sm.prefix[wave][x] + __popcll(sm.words[wave][x] & below);
            row_token[pos] = (int32_t)t;
            row_slot[pos] = a;
            row_of[t * k + a] = pos;
        }
    }
}

// Turn per-block counts [NB][n] into per-block first rows and fill expert_offsets.
__global__ __launch_bounds__(kMaxN) void paths_scan_kernel(int32_t* __restrict__ block_counts,
                                                           int64_t NB, int n,
                                                           int32_t* __restrict__ offsets) {
    __shared__ int scan[kMaxN];
    const int x = threadIdx.x;
    int run = 0;
    if (x < n)
        for (int64_t b0 = 0; b0 < NB; b0 += 16) {  // 16 independent loads, then the running sum
            int c[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) c[j] = b0 + j < NB ? block_counts[(b0 + j) * n + x] : 0;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                if (b0 + j < NB) block_counts[(b0 + j) * n + x] = run;
                run += c[j];
            }
        }
    scan[x] = x < n ? run : 0;
    __syncthreads();
    int own = scan[x];
    for (int d = 1; d < kMaxN; d <<= 1) {
        int v = x >= d ? scan[x - d] : 0;
        __syncthreads();
        scan[x] += v;
        __syncthreads();
    }
    const int excl = scan[x] - own;
    if (x < n) {
        offsets[x] = excl;
        for (int64_t b0 = 0; b0 < NB; b0 += 16) {
            int c[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) c[j] = b0 + j < NB ? block_counts[(b0 + j) * n + x] : 0;
#pragma unroll
            for (int j = 0; j < 16; ++j)
                if (b0 + j < NB) block_counts[(b0 + j) * n + x] = c[j] + excl;
        }
    }
    if (x == kMaxN - 1) offsets[n] = scan[x];
}

// Grouped dispatch with a variable number of entries per token: token t contributes
// counts[t] <= K distinct experts ids[t, 0..counts[t]) (scored routing: the distinct
// sources, or the distinct targets, of its selected paths). Rows are ordered by
// (expert, token) with the same OR-bitset ranks as paths_kernel; row_of[t, a] = -1 for
// a >= counts[t].
template <int PH>
__global__ __launch_bounds__(kPathBlock) void dispatch_kernel(
    const int32_t* __restrict__ ids, const int32_t* __restrict__ counts, int64_t T, int n, int K,
    int32_t* __restrict__ offsets, int32_t* __restrict__ row_token, int32_t* __restrict__ row_slot,
    int32_t* __restrict__ row_of, int32_t* __restrict__ block_counts) {
    __shared__ PathSmem sm;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    for (int i = tid; i < kWaves * kMaxN; i += kPathBlock) (&sm.words[0][0])[i] = 0ull;
    __syncthreads();

    const int64_t t = (int64_t)blockIdx.x * kPathBlock + tid;
    const bool valid = t < T;
    int c = valid ? counts[t] : 0;
    c = c < 0 ? 0 : (c > K ? K : c);
    int e[kMaxK];
#pragma unroll
    for (int a = 0; a < kMaxK; ++a) {
        int v = (a < c) ? ids[t * K + a] : 0;
        e[a] = v < 0 ? 0 : (v >= n ? n - 1 : v);
    }
#pragma unroll
    for (int a = 0; a < kMaxK; ++a)
        if (a < c) atomicOr(&sm.words[wave][e[a]], 1ull << lane);
    __syncthreads();

    for (int x = tid; x < kMaxN; x += kPathBlock) {
        int run = 0;
        if (x < n) {
#pragma unroll
            for (int v = 0; v < kWaves; ++v) {
                sm.prefix[v][x] = run;
                run += __popcll(sm.words[v][x]);
            }
        }
        sm.scan[x] = run;
    }
    __syncthreads();

    if (PH == kCount) {
        for (int x = tid; x < n; x += kPathBlock) block_counts[(int64_t)blockIdx.x * n + x] = sm.scan[x];
        return;
    }
    if (PH == kFused) {
        const int total = block_exclusive_scan(sm.scan, n);
        for (int x = tid; x < n; x += kPathBlock) offsets[x] = sm.scan[x];
        if (tid == 0) offsets[n] = total;
    } else {
        for (int x = tid; x < n; x += kPathBlock) sm.scan[x] = block_counts[(int64_t)blockIdx.x * n + x];
        __syncthreads();
    }
    if (valid) {
        const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
        for (int a = 0; a < kMaxK; ++a) {
            if (a >= K) break;
            if (a >= c) {
                row_of[t * K + a] = -1;
                continue;
            }
            const int x = e[a];
            const int pos = sm.scan[x] + sm.prefix[wave][x] + __popcll(sm.words[wave][x] & below);
            row_token[pos] = (int32_t)t;
            row_slot[pos] = a;
            row_of[t * K + a] = pos;
        }
    }
}

}  // namespace

size_t build_paths_ws_bytes(int64_t T, int n) {
    const int64_t NB = ceil_div(T, kPathBlock);
    return NB <= 1 ? 0 : align_up((size_t)NB * n * sizeof(int32_t), 256);
}

hipError_t launch_build_paths(const int32_t* ids, const float* w, const uint8_t* mask, int64_t T,
                              int n, int k, int beta_mode, uint64_t* bits, float* beta,
                              int32_t* offsets, int32_t* row_token, int32_t* row_slot,
                              int32_t* row_of, int32_t* block_counts, hipStream_t s) {
    const int64_t NB = ceil_div(T, kPathBlock);
    if (NB <= 1) {
        paths_kernel<kFused><<<1, kPathBlock, 0, s>>>(ids, w, mask, T, n, k, beta_mode, bits, beta,
                                                      offsets, row_token, row_slot, row_of, nullptr);
        return hipGetLastError();
    }
    paths_kernel<kCount><<<(unsigned)NB, kPathBlock, 0, s>>>(ids, w, mask, T, n, k, beta_mode, bits,
                                                             beta, offsets, row_token, row_slot,
                                                             row_of, block_counts);
    paths_scan_kernel<<<1, kMaxN, 0, s>>>(block_counts, NB, n, offsets);
    paths_kernel<kScatter><<<(unsigned)NB, kPathBlock, 0, s>>>(ids, w, mask, T, n, k, beta_mode,
                                                               bits, beta, offsets, row_token,
                                                               row_slot, row_of, block_counts);
    return hipGetLastError();
}

}  // namespace pcm

namespace pcm {

hipError_t launch_dispatch(const int32_t* ids, const int32_t* counts, int64_t T, int n, int K,
                           int32_t* offsets, int32_t* row_token, int32_t* row_slot,
                           int32_t* row_of, int32_t* block_counts, hipStream_t s) {
    const int64_t NB = ceil_div(T, kPathBlock);
    if (NB <= 1) {
        dispatch_kernel<kFused><<<1, kPathBlock, 0, s>>>(ids, counts, T, n, K, offsets, row_token,
                                                        row_slot, row_of, nullptr);
        return hipGetLastError();
    }
    dispatch_kernel<kCount><<<(unsigned)NB, kPathBlock, 0, s>>>(ids, counts, T, n, K, offsets,
                                                               row_token, row_slot, row_of,
                                                               block_counts);
    paths_scan_kernel<<<1, kMaxN, 0, s>>>(block_counts, NB, n, offsets);
    dispatch_kernel<kScatter><<<(unsigned)NB, kPathBlock, 0, s>>>(ids, counts, T, n, K, offsets,
                                                                 row_token, row_slot, row_of,
                                                                 block_counts);
    return hipGetLastError();
}

}  // namespace pcm
