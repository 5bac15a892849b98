// Router top-k and renormalised softmax (Section 2's top-k expert selection; the first
// step of Section 4.3's fused indexing), and the router GEMM fused ahead of it. One wavefront per token: each lane holds up to
// four logits as 64-bit keys (order-preserving float bits, then the complemented expert
// id), so a wave-wide maximum picks the largest logit and, among equal logits, the lower
// id. k rounds of the maximum give the slots in order.
#include "internal.h"

namespace pcm {

__device__ inline uint32_t orderable(float v) {
    if (v == 0.0f) v = 0.0f;  // -0 and +0 are the same logit
    uint32_t u = __float_as_uint(v);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ inline float from_orderable(uint32_t o) {
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}

// Top-k of one token's n logits l[] (global or LDS) by one wavefront; lane a < k writes
// slot a of ids_t / w_t.
template <int EPL>
__device__ inline void route_token(const float* l, int n, int k, int lane, int32_t* ids_t,
                                   float* w_t) {
    uint64_t key[EPL];
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
        const int e = lane + 64 * j;
        key[j] = e < n ? ((uint64_t)orderable(l[e]) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)e)
                       : 0ull;  // every real key is > 0
    }
    uint64_t sel[kMaxK];
#pragma unroll
    for (int a = 0; a < kMaxK; ++a) {
        if (a >= k) break;
        uint64_t best = key[0];
#pragma unroll
        for (int j = 1; j < EPL; ++j) best = key[j] > best ? key[j] : best;
        best = wave_max_u64(best);
        sel[a] = best;
#pragma unroll
        for (int j = 0; j < EPL; ++j)
            if (key[j] == best) key[j] = 0ull;
    }
    // softmax over the selected logits, shifted by the largest
    const float top = from_orderable((uint32_t)(sel[0] >> 32));
    float s = 0.0f;
#pragma unroll
    for (int a = 0; a < kMaxK; ++a)
        if (a < k) s += expf(from_orderable((uint32_t)(sel[a] >> 32)) - top);
#pragma unroll
    for (int a = 0; a < kMaxK; ++a) {
        if (a < k && lane == a) {
            ids_t[a] = (int32_t)(0xFFFFFFFFu - (uint32_t)sel[a]);
            w_t[a] = expf(from_orderable((uint32_t)(sel[a] >> 32)) - top) / s;
        }
    }
}

// ------------------------------------------------------------- fused indexing
// Section 4.3's single indexing operation over the layer's packed mask: route, path filter,
// path weights and the dispatch layout. Per token, one wavefront, in compact per-lane state
// (runtime loops over the k slots keep the code small), index_token:
//   - top-k: k rounds of a wave maximum over 64-bit keys as in route_token (with one logit
//     per lane, over the 32-bit logit keys, the lowest lane holding the maximum winning);
//     lane a keeps slot a's key, then lanes a < k take their exponentials and the softmax
//     denominator is summed in slot order, as route_token sums it;
//   - paths: lane a*k + b < k^2 tests (a, b) against the mask (diagonal set); one ballot
//     gives the token's bits; the same lane forms beta_ab in the path build's order of
//     operations (slot weights broadcast by readlane), so both give the same bits.
// The dispatch layout orders rows by (expert, token): a token's bit in a per-expert LDS
// bitset, popcounts for counts, and the popcount of the bits below a token for its rank, so
// no order-dependent atomic decides an index. Two launch shapes:
//   - T <= 64: one token per wave, 4 waves per workgroup; after its tokens each workgroup
//     takes a ticket, and the last one reads every token's experts back and builds the
//     whole layout (one launch);
//   - otherwise workgroups of 16 waves own kIdxCount tokens each, write their per-expert
//     counts, and route_scatter_kernel places the rows (two launches).
// Every workgroup loads its logits and the packed mask before its first store (a wave's
// loads complete in order with its stores, so a load behind a store would wait for it).
#ifndef PCM_IDX_COUNT
#define PCM_IDX_COUNT 32
#endif
constexpr int kIdxCount = PCM_IDX_COUNT;    // tokens per counting block
constexpr int kIdxSmall = 64;    // largest T of the single-launch case
constexpr int kIdxScatter = 128; // tokens per placing block (whole counting blocks)
constexpr int kIdxWaves = 16;
constexpr int kIdxThreads = 64 * kIdxWaves;
constexpr int kIdxSmallWaves = 4;
static_assert(kIdxScatter % kIdxCount == 0 && kIdxScatter * kMaxK == kIdxThreads, "layout");

__device__ inline float readlane_f32(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Exclusive scan of v over threads 0..kMaxN-1 of the workgroup (its first four waves; every
// thread of the workgroup must call it): wave scans by DPP, then the wave totals.
// Returns the exclusive prefix to threads < kMaxN and the total in *total for all threads.
__device__ inline int scan_columns(int v, int* wave_tot, int* total) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int incl = wave_incl_scan_i32(v);
    if (tid < kMaxN && lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int base = 0, all = 0;
#pragma unroll
    for (int q = 0; q < kMaxN / 64; ++q) {
        const int c = wave_tot[q];
        base += q < wave ? c : 0;
        all += c;
    }
    *total = all;
    return base + incl - v;
}

// Logits of token t (zeros past T) as this lane's EPL values.
template <int EPL>
__device__ inline void load_logits(const float* logits, int64_t t, int64_t T, int n, int lane,
                                   float (&lv)[EPL]) {
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
        const int x = lane + 64 * q;
        lv[q] = (t < T && x < n) ? logits[t * n + x] : 0.0f;
    }
}

// Per-lane constants of index_token, formed once per wave: the lane's path (a, b) =
// (lane / k, lane % k) and the byte addresses (for ds_bpermute) of the lanes it reads: slot a,
// slot b, and the last lane of path row a, which ends that row's running sum. Lanes at or past
// k * k read in-range lanes whose values they do not use.
struct PathLane {
    int pa, pb, at_a, at_b, at_row_end;
};
__device__ inline PathLane path_lane(int lane, int k) {
    PathLane q;
    q.pa = lane / k;
    q.pb = lane - q.pa * k;
    q.at_a = (q.pa & 63) << 2;
    q.at_b = q.pb << 2;
    q.at_row_end = ((q.pa * k + k - 1) & 63) << 2;
    // kept in registers: otherwise the compiler recomputes the division for every token
    asm volatile("" : "+v"(q.pa), "+v"(q.pb), "+v"(q.at_a), "+v"(q.at_b), "+v"(q.at_row_end));
    return q;
}
__device__ inline int bperm_i32(int at, int v) { return __builtin_amdgcn_ds_bpermute(at, v); }
__device__ inline float bperm_f32(int at, float v) {
    return __int_as_float(__builtin_amdgcn_ds_bpermute(at, __float_as_int(v)));
}

// One token by one wavefront (all 64 lanes active): writes its top-k ids and weights, path
// bits and beta; returns its slot expert to lanes < k (0 elsewhere). mask_s: the packed mask
// in LDS, ceil(n / 64) = EPL words per row; pl from path_lane(lane, k).
template <int EPL>
__device__ inline int index_token(const float (&lv)[EPL], const uint64_t* mask_s, int n,
                                  int k, int beta_mode, int64_t t, int lane, const PathLane& pl,
                                  int32_t* ids, float* w, uint64_t* bits_out, float* beta_out) {
    const int pa_ = pl.pa, pb_ = pl.pb;
    uint64_t key[EPL];
#pragma unroll
    for (int q = 0; q < EPL; ++q) {
        const int x = lane + 64 * q;
        key[q] = x < n ? ((uint64_t)orderable(lv[q]) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)x)
                       : 0ull;  // every real key is > 0
    }
    uint64_t mine = 0ull, first = 0ull;  // slot `lane`'s key (lanes < k), slot 0's key
    if constexpr (EPL == 1) {
        // one logit per lane and lane = expert id: the largest high word (the orderable logit),
        // and the lowest lane holding it (the first bit of a ballot) is the lower id, which is
        // the order of the 64-bit keys. The round's winner, slot a's key and its removal are
        // single-lane writes from scalar registers.
        uint32_t kv = (uint32_t)(key[0] >> 32), mhi = 0u, mlo = 0u, fhi = 0u;
        for (int a = 0; a < k; ++a) {
            const uint32_t m = wave_max_u32(kv);
            const int sl = __builtin_amdgcn_readfirstlane(
                __ffsll((unsigned long long)__ballot(kv == m)) - 1);
            if (a == 0) fhi = m;
            const uint32_t id_key = 0xFFFFFFFFu - (uint32_t)sl;
            // (the lane select goes through m0: a scalar value and a scalar lane select in two
            // other registers would exceed the instruction's one constant-bus read; two wait
            // states after the last write, since the next round's first DPP reads kv)
            asm volatile(
                "s_mov_b32 m0, %3\n\t"
                "v_writelane_b32 %0, 0, m0\n\t"
                "s_mov_b32 m0, %5\n\t"
                "v_writelane_b32 %1, %4, m0\n\t"
                "v_writelane_b32 %2, %6, m0\n\t"
                "s_nop 1"
                : "+v"(kv), "+v"(mhi), "+v"(mlo)
                : "s"(sl), "s"(m), "s"(a), "s"(id_key)
                : "m0");
        }
        mine = ((uint64_t)mhi << 32) | mlo;
        first = (uint64_t)fhi << 32;
    } else {
        // the lane's keys in descending order, so that each round looks at key[0] only and the
        // lane holding the round's maximum pops it
        auto order = [&](int i, int j) {
            const uint64_t hi = key[i] > key[j] ? key[i] : key[j], lo = key[i] > key[j] ? key[j] : key[i];
            key[i] = hi;
            key[j] = lo;
        };
        if constexpr (EPL == 2) order(0, 1);
        if constexpr (EPL == 3) { order(0, 1); order(1, 2); order(0, 1); }
        if constexpr (EPL == 4) { order(0, 1); order(2, 3); order(0, 2); order(1, 3); order(1, 2); }
        for (int a = 0; a < k; ++a) {
            const uint64_t best = wave_max_u64(key[0]);
            if (a == 0) first = best;
            if (lane == a) mine = best;
            if (key[0] == best) {
#pragma unroll
                for (int q = 0; q + 1 < EPL; ++q) key[q] = key[q + 1];
                key[EPL - 1] = 0ull;
            }
        }
    }
    // softmax over the selected logits, shifted by the largest, summed in slot order
    const float top = from_orderable((uint32_t)(first >> 32));
    const float ex = lane < k ? expf(from_orderable((uint32_t)(mine >> 32)) - top) : 0.0f;
    float s = 0.0f;
    for (int a = 0; a < k; ++a) s += readlane_f32(ex, a);
    const int e = lane < k ? (int)(0xFFFFFFFFu - (uint32_t)mine) : 0;
    const float p = lane < k ? ex / s : 0.0f;
    if (lane < k) {
        int32_t* const ids_t = ids + t * k;  // scalar base, lane offset
        float* const w_t = w + t * k;
        ids_t[lane] = e;
        w_t[lane] = p;
    }
    // path (a, b) of this lane: the slots' experts and weights by cross-lane reads
    const bool in = lane < k * k;
    const int ea = bperm_i32(pl.at_a, e), eb = bperm_i32(pl.at_b, e);
    const float pa = bperm_f32(pl.at_a, p), pb = bperm_f32(pl.at_b, p);
    const bool on = in && (pa_ == pb_ || ((mask_s[ea * EPL + (eb >> 6)] >> (eb & 63)) & 1ull));
    const uint64_t bits = __ballot(on);
    if (lane == 0) bits_out[t] = bits;
    float den = 1.0f;
    if (beta_mode == 0) {
        // the sum of p over the targets of this lane's source a, b ascending (the path build's
        // order of additions): a running sum along lanes a*k .. a*k+k-1, lane a*k+b holding
        // p_b where (a, b) is a path and 0 elsewhere (adding +0 to a sum of non-negative terms
        // leaves it unchanged). At step j the lanes with b >= j add their term to the value of
        // the lane before them (a DPP shift by one lane across the wave), so the lane with
        // b = j ends with ((p_0 + p_1) + ...) + p_j; the row's last lane holds the sum.
        const float v = on ? pb : 0.0f;
        float run = v;
        for (int j = 1; j < k; ++j) {
            const float prev =
                __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(run), 0x138, 0xF, 0xF, true));
            run = pb_ >= j ? prev + v : run;
        }
        den = bperm_f32(pl.at_row_end, run);
    } else if (beta_mode == 2) {
        den = 0.0f;  // sum of p_a' p_b' over the token's paths, (a', b') ascending
        for (int aa = 0; aa < k; ++aa) {
            const float paa = readlane_f32(p, aa);
            for (int bb = 0; bb < k; ++bb) {
                const float pbb = readlane_f32(p, bb);
                if ((bits >> (aa * k + bb)) & 1) den = fmaf(paa, pbb, den);
            }
        }
    }
    if (in) {
        float v = 0.0f;
        if (on) v = beta_mode == 0 ? pa * (pb / den) : (beta_mode == 1 ? pa * pb : pa * pb / den);
        float* const beta_t = beta_out + t * k * k;
        beta_t[lane] = v;
    }
    return e;
}

// T > 64: kIdxCount tokens per workgroup of 16 waves (wave w takes tokens w, w + 16, ...);
// writes the block's rows per expert to block_counts[blockIdx][n].
template <int EPL>
__global__ __launch_bounds__(kIdxThreads) void route_paths_kernel(
    const float* __restrict__ logits, const uint64_t* __restrict__ packed, int64_t T, int n, int k,
    int beta_mode, int32_t* __restrict__ ids, float* __restrict__ w, uint64_t* __restrict__ bits_out,
    float* __restrict__ beta_out, int32_t* __restrict__ block_counts) {
    constexpr int PER = kIdxCount / kIdxWaves;  // tokens per wave, one after another
    __shared__ unsigned long long words[kMaxN];
    __shared__ uint64_t mask_s[kMaxN * (kMaxN / 64)];
    // the wave index in a scalar register, so that token indices and store addresses are too
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    for (int x = tid; x < kMaxN; x += kIdxThreads) words[x] = 0ull;
    const int W = (n + 63) / 64;  // packed words per mask row
    const int64_t t0 = (int64_t)blockIdx.x * kIdxCount;
    float lv[PER][EPL];
#pragma unroll
    for (int j = 0; j < PER; ++j) load_logits<EPL>(logits, t0 + j * kIdxWaves + wave, T, n, lane, lv[j]);
    for (int x = tid; x < n * W; x += kIdxThreads) mask_s[x] = packed[x];
    __syncthreads();  // words cleared, mask staged
    const PathLane pl = path_lane(lane, k);
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int tib = j * kIdxWaves + wave;
        const int64_t t = t0 + tib;
        if (t >= T) break;  // wave-uniform
        const int e = index_token<EPL>(lv[j], mask_s, n, k, beta_mode, t, lane, pl, ids, w,
                                       bits_out, beta_out);
        if (lane < k) atomicOr(&words[e], 1ull << tib);
    }
    __syncthreads();
    for (int x = tid; x < n; x += kIdxThreads)
        block_counts[(int64_t)blockIdx.x * n + x] = __popcll(words[x]);
}

// T <= 64: one token per wave, kIdxSmallWaves waves per workgroup. Each workgroup, after its
// tokens' outputs, takes a ticket from *ticket (agent-scope acquire-release, so the last
// workgroup sees every other workgroup's top-k ids); the last one builds the layout from
// those ids and sets *ticket back to 0 for the next call.
template <int EPL>
__global__ __launch_bounds__(64 * kIdxSmallWaves) void route_paths_small_kernel(
    const float* __restrict__ logits, const uint64_t* __restrict__ packed, int64_t T, int n, int k,
    int beta_mode, int32_t* __restrict__ ids, float* __restrict__ w, uint64_t* __restrict__ bits_out,
    float* __restrict__ beta_out, int32_t* __restrict__ offsets, int32_t* __restrict__ row_token,
    int32_t* __restrict__ row_slot, int32_t* __restrict__ row_of, uint32_t* __restrict__ ticket) {
    constexpr int NT = 64 * kIdxSmallWaves;
    constexpr int RPT = kIdxSmall * kMaxK / NT;  // rows per thread of the layout
    __shared__ unsigned long long words[kMaxN];
    __shared__ uint64_t mask_s[kMaxN * (kMaxN / 64)];
    __shared__ int scan[kMaxN];
    __shared__ int wave_tot[kMaxN / 64];
    __shared__ int last;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int W = (n + 63) / 64;
    const int64_t t = (int64_t)blockIdx.x * kIdxSmallWaves + wave;
    float lv[EPL];
    load_logits<EPL>(logits, t, T, n, lane, lv);
    for (int x = tid; x < n * W; x += NT) mask_s[x] = packed[x];
    for (int x = tid; x < kMaxN; x += NT) words[x] = 0ull;
    __syncthreads();
    if (t < T)  // wave-uniform
        index_token<EPL>(lv, mask_s, n, k, beta_mode, t, lane, path_lane(lane, k), ids, w,
                         bits_out, beta_out);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");  // this wave's outputs, device-wide
    __syncthreads();
    if (tid == 0)
        last = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT) ==
               gridDim.x - 1;
    __syncthreads();
    if (!last) return;  // workgroup-uniform
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    // every token's experts, ORed into the per-expert bitsets
    int e[RPT];
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
        const int i = tid + r * NT;
        e[r] = 0;
        if (i < T * k) {
            const int v = __hip_atomic_load(ids + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            e[r] = v < 0 ? 0 : (v >= n ? n - 1 : v);
            atomicOr(&words[e[r]], 1ull << (i / k));
        }
    }
    __syncthreads();
    const int own = tid < n ? __popcll(words[tid]) : 0;
    int total;
    const int excl = scan_columns(own, wave_tot, &total);
    if (tid < kMaxN) scan[tid] = excl;
    if (tid < n) offsets[tid] = excl;
    if (tid == 0) {
        offsets[n] = total;
        __hip_atomic_store(ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
        const int i = tid + r * NT;
        if (i < T * k) {
            const int tib = i / k, a = i - (i / k) * k, x = e[r];
            const int pos = scan[x] + __popcll(words[x] & ((1ull << tib) - 1ull));
            row_token[pos] = tib;
            row_slot[pos] = a;
            row_of[i] = pos;
        }
    }
}

// Rows of kIdxScatter tokens (whole counting blocks) once every counting block has written
// its counts [NB][n]: each workgroup reduces the count table itself (column totals, and the
// column sums over the counting blocks before its own; integer sums, so the order of the
// LDS atomics does not matter), scans the totals into the expert offsets (written by
// workgroup 0), rebuilds its bitsets from the top-k ids (one 64-bit word per 64 tokens) and
// places its rows.
__global__ __launch_bounds__(kIdxThreads) void route_scatter_kernel(
    const int32_t* __restrict__ ids, int64_t T, int n, int k, const int32_t* __restrict__ block_counts,
    int64_t NB, int32_t* __restrict__ offsets, int32_t* __restrict__ row_token,
    int32_t* __restrict__ row_slot, int32_t* __restrict__ row_of) {
    constexpr int NW = kIdxScatter / 64;
    constexpr int UN = 16;  // count loads in flight per thread
    __shared__ unsigned long long words[NW][kMaxN];
    __shared__ int tot[kMaxN];
    __shared__ int before[kMaxN];
    __shared__ int first[kMaxN];
    __shared__ int wave_tot[kMaxN / 64];
    const int tid = threadIdx.x;
    const int64_t me = blockIdx.x;
    const int64_t b_me = me * (kIdxScatter / kIdxCount);  // first counting block of this one
    // this thread's row (token tib, slot a), loaded ahead of the count table
    const int tib = tid / kMaxK, a = tid - (tid / kMaxK) * kMaxK;
    const int64_t t = me * kIdxScatter + tib;
    const bool valid = a < k && t < T;
    int e = 0;
    if (valid) {
        const int v = ids[t * k + a];
        e = v < 0 ? 0 : (v >= n ? n - 1 : v);
    }
    int np = 1;
    while (np < n) np <<= 1;
    const int G = kIdxThreads / np;  // groups of counting blocks per column, >= 4
    const int x = tid % np, g = tid / np;
    // the first UN of this thread's count-table entries are loaded with the row's id, before
    // the barrier (the rest, for tables of more than UN * G blocks, after it)
    int c[UN];
#pragma unroll
    for (int u = 0; u < UN; ++u) {
        const int64_t b = g + (int64_t)u * G;
        c[u] = (x < n && b < NB) ? block_counts[b * n + x] : 0;
    }
    for (int i = tid; i < NW * kMaxN; i += kIdxThreads) (&words[0][0])[i] = 0ull;
    for (int i = tid; i < kMaxN; i += kIdxThreads) tot[i] = before[i] = 0;
    __syncthreads();
    if (valid) atomicOr(&words[tib >> 6][e], 1ull << (tib & 63));
    int st = 0, sb = 0;
    if (x < n) {
        for (int64_t b0 = g;; ) {
#pragma unroll
            for (int u = 0; u < UN; ++u) {
                st += c[u];
                sb += b0 + (int64_t)u * G < b_me ? c[u] : 0;
            }
            b0 += (int64_t)UN * G;
            if (b0 >= NB) break;
#pragma unroll
            for (int u = 0; u < UN; ++u) {
                const int64_t b = b0 + (int64_t)u * G;
                c[u] = b < NB ? block_counts[b * n + x] : 0;
            }
        }
        if (st) atomicAdd(&tot[x], st);
        if (sb) atomicAdd(&before[x], sb);
    }
    __syncthreads();
    const int own = tid < n ? tot[tid] : 0;
    int total;
    const int excl = scan_columns(own, wave_tot, &total);
    if (me == 0) {
        if (tid < n) offsets[tid] = excl;
        if (tid == 0) offsets[n] = total;
    }
    if (tid < n) first[tid] = excl + before[tid];
    __syncthreads();
    if (valid) {
        const int wd = tib >> 6;
        int pos = first[e] + __popcll(words[wd][e] & ((1ull << (tib & 63)) - 1ull));
#pragma unroll
        for (int q = 0; q < NW; ++q)
            if (q < wd) pos += __popcll(words[q][e]);
        row_token[pos] = (int32_t)t;
        row_slot[pos] = a;
        row_of[t * k + a] = pos;
    }
}

// Offline per-layer mask layout: bit j % 64 of word [i][j / 64] is set when path i -> j is
// allowed (mask[i][j] != 0, or i == j).
__global__ __launch_bounds__(256) void mask_pack_kernel(const uint8_t* __restrict__ mask, int n,
                                                        uint64_t* __restrict__ packed) {
    const int W = (n + 63) / 64;
    const int i = blockIdx.x;  // one mask row per workgroup
    for (int wd = threadIdx.x / 64; wd < W; wd += 4) {
        const int j = wd * 64 + (threadIdx.x & 63);
        const bool on = j < n && (j == i || mask[(int64_t)i * n + j] != 0);
        const uint64_t b = __ballot(on);
        if ((threadIdx.x & 63) == 0) packed[(int64_t)i * W + wd] = b;
    }
}

template <int EPL>
__global__ __launch_bounds__(256) void route_kernel(const float* __restrict__ logits, int64_t T,
                                                    int n, int k, int32_t* __restrict__ ids,
                                                    float* __restrict__ w) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;  // wave-uniform
    route_token<EPL>(logits + t * n, n, k, lane, ids + t * k, w + t * k);
}

// Router logits fused with the top-k (the router's own GEMM, Section 2: the scores the
// router computes from h): logits[t, e] = x_t . W_r[e], float32 accumulation.
// bf16, two launches:
//  * router_part_kernel: every wave computes one 16-expert x 16-token block of partial dot
//    products over one K slice on the matrix cores (v_mfma_f32_16x16x32_bf16, router rows
//    as the first operand), fragments loaded straight from global memory; part[s][t][e];
//  * router_topk_kernel: one wave per token sums the K slices in order (deterministic),
//    writes the logits if asked, and runs the top-k on them.
// The K split is chosen so that about 2048 waves share the work.
__global__ __launch_bounds__(256) void router_part_kernel(const uint16_t* __restrict__ x,
                                                          const uint16_t* __restrict__ wr,
                                                          int64_t T, int H, int n, int et,
                                                          int64_t tt, int ks, int steps,
                                                          float* __restrict__ part) {
    const int lane = threadIdx.x & 63;
    const int64_t unit = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (unit >= (int64_t)et * tt * ks) return;  // wave-uniform
    const int e_tile = (int)(unit % et);
    const int64_t t_tile = (unit / et) % tt;
    const int s = (int)(unit / ((int64_t)et * tt));
    const int r16 = lane & 15, kg = lane >> 4;
    const int64_t t0 = t_tile * 16;
    const int64_t tok = t0 + r16 < T ? t0 + r16 : T - 1;
    const int e = e_tile * 16 + r16 < n ? e_tile * 16 + r16 : n - 1;
    const int KT = H / 32, k0 = s * steps, k1 = k0 + steps < KT ? k0 + steps : KT;
    const bf16x8* xp = (const bf16x8*)(x + tok * H + kg * 8);
    const bf16x8* wp = (const bf16x8*)(wr + (int64_t)e * H + kg * 8);
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int kt = k0; kt < k1; ++kt)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wp[kt * 4], xp[kt * 4], acc, 0, 0, 0);
    // acc[r]: expert e_tile*16 + 4*kg + r of token t0 + r16
    const int npad = et * 16;
    if (t0 + r16 < T) {
        float* dst = part + ((int64_t)s * T + t0 + r16) * npad + e_tile * 16 + 4 * kg;
        *(float4*)dst = make_float4(acc[0], acc[1], acc[2], acc[3]);
    }
}

template <int EPL>
__global__ __launch_bounds__(256) void router_topk_kernel(const float* __restrict__ part,
                                                          int64_t T, int n, int npad, int ks,
                                                          int k, float* __restrict__ logits,
                                                          int32_t* __restrict__ ids,
                                                          float* __restrict__ w) {
    __shared__ float lg[4][kMaxN];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t t = (int64_t)blockIdx.x * 4 + wave;
    if (t >= T) return;  // wave-uniform; only wave-local LDS use follows
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
        const int e = lane + 64 * j;
        if (e >= n) continue;
        float v = 0.0f;
        for (int s = 0; s < ks; ++s) v += part[((int64_t)s * T + t) * npad + e];
        lg[wave][e] = v;
        if (logits) logits[t * n + e] = v;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    route_token<EPL>(lg[wave], n, k, lane, ids + t * k, w + t * k);
}

// The same for many K slices (large H, few tokens): one workgroup per token, thread e
// sums expert e's slices (independent loads, several in flight), then wave 0 runs the
// top-k. The sum over slices runs in the same order as in router_topk_kernel.
template <int EPL>
__global__ __launch_bounds__(256) void router_topk_wide_kernel(const float* __restrict__ part,
                                                               int64_t T, int n, int npad, int ks,
                                                               int k, float* __restrict__ logits,
                                                               int32_t* __restrict__ ids,
                                                               float* __restrict__ w) {
    __shared__ float lg[kMaxN];
    const int64_t t = blockIdx.x;
    for (int e = threadIdx.x; e < n; e += blockDim.x) {
        const float* p = part + t * npad + e;
        const int64_t stride = T * npad;
        float v = 0.0f;
        int s = 0;
        for (; s + 8 <= ks; s += 8) {
            float q[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) q[j] = p[(s + j) * stride];
#pragma unroll
            for (int j = 0; j < 8; ++j) v += q[j];
        }
        for (; s < ks; ++s) v += p[s * stride];
        lg[e] = v;
        if (logits) logits[t * n + e] = v;
    }
    __syncthreads();
    if (threadIdx.x < 64) route_token<EPL>(lg, n, k, threadIdx.x, ids + t * k, w + t * k);
}

// float32: one wavefront per token; lane e (+64 j) forms x_t . W_r[e] with h ascending.
__global__ __launch_bounds__(256) void router_f32_kernel(const float* __restrict__ x,
                                                         const float* __restrict__ wr, int64_t T,
                                                         int H, int n, int k,
                                                         float* __restrict__ logits,
                                                         int32_t* __restrict__ ids,
                                                         float* __restrict__ w) {
    __shared__ float lg[4][kMaxN];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t t = (int64_t)blockIdx.x * 4 + wave;
    const bool active = t < T;
    for (int e = lane; e < n; e += 64) {
        float s = 0.0f;
        if (active)
            for (int h = 0; h < H; ++h) s = fmaf(x[t * H + h], wr[(int64_t)e * H + h], s);
        lg[wave][e] = s;
        if (logits && active) logits[t * n + e] = s;
    }
    __syncthreads();
    if (!active) return;
    if (n <= 64) route_token<1>(lg[wave], n, k, lane, ids + t * k, w + t * k);
    else if (n <= 128) route_token<2>(lg[wave], n, k, lane, ids + t * k, w + t * k);
    else if (n <= 192) route_token<3>(lg[wave], n, k, lane, ids + t * k, w + t * k);
    else route_token<4>(lg[wave], n, k, lane, ids + t * k, w + t * k);
}

hipError_t launch_route(const float* logits, int64_t T, int n, int k, int32_t* ids, float* w,
                        hipStream_t s) {
    const dim3 grid((unsigned)ceil_div(T, 4)), block(256);
    const int epl = (int)ceil_div(n, 64);
    switch (epl) {
        case 1: route_kernel<1><<<grid, block, 0, s>>>(logits, T, n, k, ids, w); break;
        case 2: route_kernel<2><<<grid, block, 0, s>>>(logits, T, n, k, ids, w); break;
        case 3: route_kernel<3><<<grid, block, 0, s>>>(logits, T, n, k, ids, w); break;
        default: route_kernel<4><<<grid, block, 0, s>>>(logits, T, n, k, ids, w); break;
    }
    return hipGetLastError();
}

size_t route_paths_ws_bytes(int64_t T, int n) {
    // the single-launch ticket, then (T > 64) the counts [ceil(T / kIdxCount)][n]
    return 256 + (T <= kIdxSmall ? 0 : align_up((size_t)ceil_div(T, kIdxCount) * n * sizeof(int32_t), 256));
}

hipError_t launch_mask_pack(const uint8_t* mask, int n, uint64_t* packed, hipStream_t s) {
    mask_pack_kernel<<<(unsigned)n, 256, 0, s>>>(mask, n, packed);
    return hipGetLastError();
}

hipError_t launch_route_paths(const float* logits, const uint64_t* packed, int64_t T, int n, int k,
                              int beta_mode, int32_t* ids, float* w, uint64_t* bits, float* beta,
                              int32_t* offsets, int32_t* row_token, int32_t* row_slot,
                              int32_t* row_of, void* ws, hipStream_t s) {
    const int epl = (int)ceil_div(n, 64);
    uint32_t* ticket = (uint32_t*)ws;
    if (T <= kIdxSmall) {
        const unsigned blocks = (unsigned)ceil_div(T, kIdxSmallWaves);
        auto go = [&](auto kern) {
            kern<<<blocks, 64 * kIdxSmallWaves, 0, s>>>(logits, packed, T, n, k, beta_mode, ids, w,
                                                        bits, beta, offsets, row_token, row_slot,
                                                        row_of, ticket);
        };
        switch (epl) {
            case 1: go(route_paths_small_kernel<1>); break;
            case 2: go(route_paths_small_kernel<2>); break;
            case 3: go(route_paths_small_kernel<3>); break;
            default: go(route_paths_small_kernel<4>); break;
        }
        return hipGetLastError();
    }
    int32_t* block_counts = (int32_t*)((char*)ws + 256);
    const int64_t NB = ceil_div(T, kIdxCount);
    auto go = [&](auto kern) {
        kern<<<(unsigned)NB, kIdxThreads, 0, s>>>(logits, packed, T, n, k, beta_mode, ids, w, bits,
                                                  beta, block_counts);
    };
    switch (epl) {
        case 1: go(route_paths_kernel<1>); break;
        case 2: go(route_paths_kernel<2>); break;
        case 3: go(route_paths_kernel<3>); break;
        default: go(route_paths_kernel<4>); break;
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    route_scatter_kernel<<<(unsigned)ceil_div(T, kIdxScatter), kIdxThreads, 0, s>>>(
        ids, T, n, k, block_counts, NB, offsets, row_token, row_slot, row_of);
    return hipGetLastError();
}

// K split of the router GEMM: slices of `steps` 32-wide K steps, about 2048 waves in all.
void router_split(int64_t T, int H, int n, int* et, int64_t* tt, int* ks, int* steps) {
    *et = (int)ceil_div(n, 16);
    *tt = ceil_div(T, 16);
    const int KT = H / 32;
    int64_t want = ceil_div(2048, (int64_t)*et * *tt);
    want = want < 1 ? 1 : (want > KT ? KT : want);
    *steps = (int)ceil_div(KT, want);
    *ks = (int)ceil_div(KT, *steps);
}

size_t router_ws_bytes(int64_t T, int H, int n) {
    int et, ks, steps;
    int64_t tt;
    router_split(T, H, n, &et, &tt, &ks, &steps);
    return align_up((size_t)ks * T * et * 16 * sizeof(float), 256);
}

hipError_t launch_router(bool bf16, const void* x, const void* wr, int64_t T, int H, int n, int k,
                         float* logits, int32_t* ids, float* w, float* part, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (!bf16) {
        router_f32_kernel<<<(unsigned)ceil_div(T, 4), 256, 0, s>>>((const float*)x, (const float*)wr,
                                                                  T, H, n, k, logits, ids, w);
        return hipGetLastError();
    }
    int et, ks, steps;
    int64_t tt;
    router_split(T, H, n, &et, &tt, &ks, &steps);
    const int64_t units = (int64_t)et * tt * ks;
    router_part_kernel<<<(unsigned)ceil_div(units, 4), 256, 0, s>>>(
        (const uint16_t*)x, (const uint16_t*)wr, T, H, n, et, tt, ks, steps, part);
    const dim3 grid((unsigned)ceil_div(T, 4)), block(256);
    const int npad = et * 16;
    if (ks * ceil_div(n, 64) > 16) {   // long serial sums per lane: spread them over a workgroup
        const dim3 wgrid((unsigned)T);
        switch (ceil_div(n, 64)) {
            case 1: router_topk_wide_kernel<1><<<wgrid, block, 0, s>>>(part, T, n, npad, ks, k, logits, ids, w); break;
            case 2: router_topk_wide_kernel<2><<<wgrid, block, 0, s>>>(part, T, n, npad, ks, k, logits, ids, w); break;
            case 3: router_topk_wide_kernel<3><<<wgrid, block, 0, s>>>(part, T, n, npad, ks, k, logits, ids, w); break;
            default: router_topk_wide_kernel<4><<<wgrid, block, 0, s>>>(part, T, n, npad, ks, k, logits, ids, w); break;
        }
        return hipGetLastError();
    }
    switch (ceil_div(n, 64)) {
        case 1: router_topk_kernel<1><<<grid, block, 0, s>>>(part, T, n, npad, ks, k, logits, ids, w); break;
        case 2: router_topk_kernel<2><<<grid, block, 0, s>>>(part, T, n, npad, ks, k, logits, ids, w); break;
        case 3: router_topk_kernel<3><<<grid, block, 0, s>>>(part, T, n, npad, ks, k, logits, ids, w); break;
        default: router_topk_kernel<4><<<grid, block, 0, s>>>(part, T, n, npad, ks, k, logits, ids, w); break;
    }
    return hipGetLastError();
}

}  // namespace pcm
