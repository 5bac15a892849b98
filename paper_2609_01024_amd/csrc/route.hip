// Router top-k and renormalised softmax (Section 2's top-k expert selection; the first
// step of Section 4.3's fused indexing). One wavefront per token: each lane holds up to
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

template <int EPL>
__global__ __launch_bounds__(256) void route_kernel(const float* __restrict__ logits, int64_t T,
                                                    int n, int k, int32_t* __restrict__ ids,
                                                    float* __restrict__ w) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;  // wave-uniform
    const float* l = logits + t * n;
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
            ids[t * k + a] = (int32_t)(0xFFFFFFFFu - (uint32_t)sel[a]);
            w[t * k + a] = expf(from_orderable((uint32_t)(sel[a] >> 32)) - top) / s;
        }
    }
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

}  // namespace pcm
