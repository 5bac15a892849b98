// Path mix and combine (Section 4.1's path aggregation in Section 4.3's source-grouped form).
//   mix:     z_(t,b) = sum_{a : (a,b) in Pi(t)} beta_ab u_(t,a)   (a ascending, float32 math)
//            Because the projection W_down[e_b] is linear, applying it once to z_(t,b)
//            equals summing beta_ab W_down[e_b] u_(t,a) over the paths into target b.
//            For bf16 layers z is written as split hi/lo bf16 pairs for the down GEMM.
//   combine: y_t = [y_t] + sum_{b ascending} o_(t,b)
// One workgroup per token; each thread owns 8 consecutive columns.
#include "internal.h"

namespace pcm {
namespace {

__device__ inline void load8(const float* p, float* v) {
    const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ inline uint4 pack8(const float* v) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
        w[i] = (uint32_t)f32_to_bf16_rne(v[2 * i]) | ((uint32_t)f32_to_bf16_rne(v[2 * i + 1]) << 16);
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// One token per workgroup; 8 consecutive columns per thread.
template <bool SPLIT>
__global__ __launch_bounds__(256) void mix_kernel(const float* __restrict__ u, void* __restrict__ z,
                                                  const uint64_t* __restrict__ bits,
                                                  const float* __restrict__ beta,
                                                  const int32_t* __restrict__ row_of, int k, int F,
                                                  int64_t R) {
    const int64_t t = blockIdx.x;
    const uint64_t pb = bits[t];
    int64_t rows[kMaxK];
#pragma unroll
    for (int a = 0; a < kMaxK; ++a) {
        int64_t r = a < k ? row_of[t * k + a] : 0;
        rows[a] = r < 0 ? 0 : (r >= R ? R - 1 : r);
    }
    const float* bt = beta + t * k * k;
    for (int c = threadIdx.x * 8; c < F; c += blockDim.x * 8) {
        float ua[kMaxK][8];
#pragma unroll
        for (int a = 0; a < kMaxK; ++a)
            if (a < k) load8(u + rows[a] * F + c, ua[a]);
#pragma unroll
        for (int b = 0; b < kMaxK; ++b) {
            if (b >= k) break;
            float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int a = 0; a < kMaxK; ++a) {
                if (a < k && ((pb >> (a * k + b)) & 1)) {
                    const float w = bt[a * k + b];
#pragma unroll
                    for (int i = 0; i < 8; ++i) acc[i] = fmaf(w, ua[a][i], acc[i]);
                }
            }
            if (SPLIT) {
                float lo[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) lo[i] = acc[i] - bf16_bits_to_f32(f32_to_bf16_rne(acc[i]));
                uint16_t* dst = (uint16_t*)z + rows[b] * 2 * F + (c / kSplitBlock) * 2 * kSplitBlock
                                + c % kSplitBlock;
                *(uint4*)dst = pack8(acc);
                *(uint4*)(dst + kSplitBlock) = pack8(lo);
            } else {
                float* dst = (float*)z + rows[b] * F + c;
                *(float4*)dst = make_float4(acc[0], acc[1], acc[2], acc[3]);
                *(float4*)(dst + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
            }
        }
    }
}

__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ o,
                                                      const int32_t* __restrict__ row_of, int k,
                                                      int H, int64_t R, float* __restrict__ y,
                                                      int accumulate) {
    const int64_t t = blockIdx.x;
    int64_t rows[kMaxK];
#pragma unroll
    for (int b = 0; b < kMaxK; ++b) {
        int64_t r = b < k ? row_of[t * k + b] : 0;
        rows[b] = r < 0 ? 0 : (r >= R ? R - 1 : r);
    }
    for (int c = threadIdx.x * 4; c < H; c += blockDim.x * 4) {
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int b = 0; b < kMaxK; ++b) {
            if (b >= k) break;
            const float4 v = *(const float4*)(o + rows[b] * H + c);
            s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
        }
        float4* dst = (float4*)(y + t * H + c);
        if (accumulate) {
            const float4 old = *dst;
            s.x = old.x + s.x; s.y = old.y + s.y; s.z = old.z + s.z; s.w = old.w + s.w;
        }
        *dst = s;
    }
}

}  // namespace

hipError_t launch_mix(bool split, const float* u, void* z, const uint64_t* bits, const float* beta,
                      const int32_t* row_of, int64_t T, int k, int F, hipStream_t s) {
    if (T == 0) return hipSuccess;
    const int threads = F / 8 >= 256 ? 256 : ((F / 8 + 63) / 64) * 64;
    if (split)
        mix_kernel<true><<<(unsigned)T, threads, 0, s>>>(u, z, bits, beta, row_of, k, F, T * k);
    else
        mix_kernel<false><<<(unsigned)T, threads, 0, s>>>(u, z, bits, beta, row_of, k, F, T * k);
    return hipGetLastError();
}

hipError_t launch_combine(const float* o, const int32_t* row_of, int64_t T, int k, int H,
                          float* y, int accumulate, hipStream_t s) {
    if (T == 0) return hipSuccess;
    const int threads = H / 4 >= 256 ? 256 : ((H / 4 + 63) / 64) * 64;
    combine_kernel<<<(unsigned)T, threads, 0, s>>>(o, row_of, k, H, T * k, y, accumulate);
    return hipGetLastError();
}

}  // namespace pcm
