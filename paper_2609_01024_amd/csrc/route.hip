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
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const uint64_t o = __shfl_xor(best, off);
            best = o > best ? o : best;
        }
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
