// Path mix and combine (Section 4.1's path aggregation in Section 4.3's source-grouped form).
//   mix:     z_(t,b) = sum_{a : (a,b) in Pi(t)} beta_ab u_(t,a)   (a ascending, float32 math)
//            Because the projection W_down[e_b] is linear, applying it once to z_(t,b)
//            equals summing beta_ab W_down[e_b] u_(t,a) over the paths into target b.
//            bf16 layers store z as float16 rows scaled by a power of two (largest element
//            just below 2^14) with the inverse scale kept per row for the down GEMM.
//   combine: y_t = [y_t] + sum_{b ascending} o_(t,b)
// One workgroup per token; each thread owns 8 consecutive columns.
#include "internal.h"

namespace pcm {
namespace {

__device__ inline void load8(const float* p, float* v) {
    const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

struct TokenPaths {
    uint64_t bits;
    int64_t rows[kMaxK];
    const float* beta;
    int k;
};

__device__ inline TokenPaths token_paths(const uint64_t* bits, const float* beta,
                                         const int32_t* row_of, int64_t t, int k, int64_t R) {
    TokenPaths p;
    if (bits == nullptr) {  // identity: one row per token, weight 1
        p.bits = 1;
        p.rows[0] = t;
        p.beta = nullptr;
        p.k = 1;
        return p;
    }
    p.bits = bits[t];
#pragma unroll
    for (int a = 0; a < kMaxK; ++a) {
        int64_t r = a < k ? row_of[t * k + a] : 0;
        p.rows[a] = r < 0 ? 0 : (r >= R ? R - 1 : r);
    }
    p.beta = beta + t * k * k;
    p.k = k;
    return p;
}

// z values of 8 columns starting at c for every target b of the token
__device__ inline void mix8(const float* __restrict__ u, const TokenPaths& p, int F, int c,
                            float (&z)[kMaxK][8]) {
    float ua[kMaxK][8];
#pragma unroll
    for (int a = 0; a < kMaxK; ++a)
        if (a < p.k) load8(u + p.rows[a] * F + c, ua[a]);
#pragma unroll
    for (int b = 0; b < kMaxK; ++b) {
        if (b >= p.k) break;
#pragma unroll
        for (int i = 0; i < 8; ++i) z[b][i] = 0.f;
#pragma unroll
        for (int a = 0; a < kMaxK; ++a) {
            if (a < p.k && ((p.bits >> (a * p.k + b)) & 1)) {
                const float w = p.beta ? p.beta[a * p.k + b] : 1.0f;
#pragma unroll
                for (int i = 0; i < 8; ++i) z[b][i] = fmaf(w, ua[a][i], z[b][i]);
            }
        }
    }
}

template <bool F16>
__global__ __launch_bounds__(256) void mix_kernel(const float* __restrict__ u, void* __restrict__ z,
                                                  float* __restrict__ zscale,
                                                  const uint64_t* __restrict__ bits,
                                                  const float* __restrict__ beta,
                                                  const int32_t* __restrict__ row_of, int k, int F,
                                                  int64_t R) {
    const int64_t t = blockIdx.x;
    const TokenPaths p = token_paths(bits, beta, row_of, t, k, R);
    float scale[kMaxK];
    if (F16) {
        // pass 1: largest |z| of each target row, reduced over the workgroup
        float mx[kMaxK];
#pragma unroll
        for (int b = 0; b < kMaxK; ++b) mx[b] = 0.f;
        for (int c = threadIdx.x * 8; c < F; c += blockDim.x * 8) {
            float zz[kMaxK][8];
            mix8(u, p, F, c, zz);
#pragma unroll
            for (int b = 0; b < kMaxK; ++b)
                if (b < p.k)
#pragma unroll
                    for (int i = 0; i < 8; ++i) mx[b] = fmaxf(mx[b], fabsf(zz[b][i]));
        }
        __shared__ float red[kMaxK][4];
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
        for (int b = 0; b < kMaxK; ++b) {
            if (b >= p.k) break;
            float v = mx[b];
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
            if (lane == 0) red[b][wave] = v;
        }
        __syncthreads();
        const int nw = (blockDim.x + 63) / 64;
#pragma unroll
        for (int b = 0; b < kMaxK; ++b) {
            if (b >= p.k) break;
            float v = 0.f;
            for (int w = 0; w < nw; ++w) v = fmaxf(v, red[b][w]);
            // scale = 2^(kZScaleExp - e) with v < 2^e, so every |z * scale| < 2^kZScaleExp
            int e = 0;
            if (v > 0.f) frexpf(v, &e);
            int sh = kZScaleExp - e;
            sh = sh > 126 ? 126 : (sh < -126 ? -126 : sh);
            scale[b] = ldexpf(1.0f, sh);
            if (threadIdx.x == 0) zscale[p.rows[b]] = ldexpf(1.0f, -sh);
        }
    }
    // pass 2 (only pass for float32 layers): store z
    for (int c = threadIdx.x * 8; c < F; c += blockDim.x * 8) {
        float zz[kMaxK][8];
        mix8(u, p, F, c, zz);
#pragma unroll
        for (int b = 0; b < kMaxK; ++b) {
            if (b >= p.k) break;
            if (F16) {
                uint32_t w[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const _Float16 lo = (_Float16)(zz[b][2 * i] * scale[b]);
                    const _Float16 hi = (_Float16)(zz[b][2 * i + 1] * scale[b]);
                    w[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) |
                           ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
                }
                *(uint4*)((uint16_t*)z + p.rows[b] * F + c) = make_uint4(w[0], w[1], w[2], w[3]);
            } else {
                float* dst = (float*)z + p.rows[b] * F + c;
                *(float4*)dst = make_float4(zz[b][0], zz[b][1], zz[b][2], zz[b][3]);
                *(float4*)(dst + 4) = make_float4(zz[b][4], zz[b][5], zz[b][6], zz[b][7]);
            }
        }
    }
}

// Single-pass form of the float16 mix: each thread keeps its ITER column chunks of every
// target row in registers (KK >= k targets), so U is read once; then the row maxima are
// reduced over the workgroup and the scaled rows stored.
template <int KK, int ITER>
__global__ __launch_bounds__(1024) void mix_regs_kernel(const float* __restrict__ u,
                                                        uint16_t* __restrict__ z,
                                                        float* __restrict__ zscale,
                                                        const uint64_t* __restrict__ bits,
                                                        const float* __restrict__ beta,
                                                        const int32_t* __restrict__ row_of, int k,
                                                        int F, int64_t R) {
    const int64_t t = blockIdx.x;
    const TokenPaths p = token_paths(bits, beta, row_of, t, k, R);
    float zz[ITER][KK][8];
    float mx[KK];
#pragma unroll
    for (int b = 0; b < KK; ++b) mx[b] = 0.f;
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
#pragma unroll
        for (int b = 0; b < KK; ++b)
#pragma unroll
            for (int i = 0; i < 8; ++i) zz[it][b][i] = 0.f;
        const int c = (threadIdx.x + it * blockDim.x) * 8;
        if (c >= F) continue;
        // sources in ascending order, each row's 8 values added to every target it feeds
#pragma unroll
        for (int a = 0; a < KK; ++a) {
            if (a >= p.k) break;
            float ua[8];
            load8(u + p.rows[a] * F + c, ua);
#pragma unroll
            for (int b = 0; b < KK; ++b) {
                if (b < p.k && ((p.bits >> (a * p.k + b)) & 1)) {
                    const float w = p.beta ? p.beta[a * p.k + b] : 1.0f;
#pragma unroll
                    for (int i = 0; i < 8; ++i) zz[it][b][i] = fmaf(w, ua[i], zz[it][b][i]);
                }
            }
        }
#pragma unroll
        for (int b = 0; b < KK; ++b)
#pragma unroll
            for (int i = 0; i < 8; ++i) mx[b] = fmaxf(mx[b], fabsf(zz[it][b][i]));
    }
    __shared__ float red[KK][16];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int b = 0; b < KK; ++b) {
        float v = mx[b];
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
        if (lane == 0) red[b][wave] = v;
    }
    __syncthreads();
    const int nw = (blockDim.x + 63) / 64;
    float scale[KK];
#pragma unroll
    for (int b = 0; b < KK; ++b) {
        float v = 0.f;
        for (int w = 0; w < nw; ++w) v = fmaxf(v, red[b][w]);
        // scale = 2^(kZScaleExp - e) with v < 2^e, so every |z * scale| < 2^kZScaleExp
        int e = 0;
        if (v > 0.f) frexpf(v, &e);
        int sh = kZScaleExp - e;
        sh = sh > 126 ? 126 : (sh < -126 ? -126 : sh);
        scale[b] = ldexpf(1.0f, sh);
        if (threadIdx.x == 0 && b < p.k) zscale[p.rows[b]] = ldexpf(1.0f, -sh);
    }
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
        const int c = (threadIdx.x + it * blockDim.x) * 8;
        if (c >= F) continue;
#pragma unroll
        for (int b = 0; b < KK; ++b) {
            if (b >= p.k) break;
            uint32_t w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const _Float16 lo = (_Float16)(zz[it][b][2 * i] * scale[b]);
                const _Float16 hi = (_Float16)(zz[it][b][2 * i + 1] * scale[b]);
                w[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) |
                       ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
            }
            *(uint4*)(z + p.rows[b] * F + c) = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
}

template <int KK, int ITER>
void launch_mix_regs(unsigned blocks, int threads, const float* u, void* z, float* zscale,
                     const uint64_t* bits, const float* beta, const int32_t* row_of, int k, int F,
                     int64_t R, hipStream_t s) {
    mix_regs_kernel<KK, ITER><<<blocks, threads, 0, s>>>(u, (uint16_t*)z, zscale, bits, beta,
                                                         row_of, k, F, R);
}

__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ o, int ksplit,
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
            for (int q = 0; q < ksplit; ++q) {  // K slices of the projection, in order
                const float4 v = *(const float4*)(o + (q * R + rows[b]) * H + c);
                s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
            }
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

hipError_t launch_mix(const float* u, void* z, float* zscale, const uint64_t* bits,
                      const float* beta, const int32_t* row_of, int64_t T, int k, int F,
                      hipStream_t s) {
    if (T == 0) return hipSuccess;
    const int threads = F / 8 >= 256 ? 256 : ((F / 8 + 63) / 64) * 64;
    const int64_t R = bits ? T * k : T;
    if (zscale) {
        // single pass when a thread's share of every target row fits in 64 registers
        const int chunks = F / 8;
        const int threads_r = chunks >= 1024 ? 1024 : ((chunks + 63) / 64) * 64;
        const int iter = (chunks + threads_r - 1) / threads_r;
        const int kk = k <= 1 ? 1 : (k <= 2 ? 2 : (k <= 4 ? 4 : 8));
        const int it = iter <= 1 ? 1 : (iter <= 2 ? 2 : (iter <= 4 ? 4 : (iter <= 8 ? 8 : 16)));  // 16: two-pass
        const unsigned blocks = (unsigned)T;
        if (kk * it <= 8) {
            auto go = [&](auto fn) {
                fn(blocks, threads_r, u, z, zscale, bits, beta, row_of, k, F, R, s);
                return hipGetLastError();
            };
            switch (kk * 100 + it) {
                case 101: return go(launch_mix_regs<1, 1>);
                case 102: return go(launch_mix_regs<1, 2>);
                case 104: return go(launch_mix_regs<1, 4>);
                case 108: return go(launch_mix_regs<1, 8>);
                case 201: return go(launch_mix_regs<2, 1>);
                case 202: return go(launch_mix_regs<2, 2>);
                case 204: return go(launch_mix_regs<2, 4>);
                case 401: return go(launch_mix_regs<4, 1>);
                case 402: return go(launch_mix_regs<4, 2>);
                case 801: return go(launch_mix_regs<8, 1>);
                default: break;
            }
        }
        mix_kernel<true><<<(unsigned)T, threads, 0, s>>>(u, z, zscale, bits, beta, row_of, k, F, R);
    } else
        mix_kernel<false><<<(unsigned)T, threads, 0, s>>>(u, z, zscale, bits, beta, row_of, k, F, R);
    return hipGetLastError();
}

hipError_t launch_combine(const float* o, int ksplit, const int32_t* row_of, int64_t T, int k,
                          int H, float* y, int accumulate, hipStream_t s) {
    if (T == 0) return hipSuccess;
    const int threads = H / 4 >= 256 ? 256 : ((H / 4 + 63) / 64) * 64;
    combine_kernel<<<(unsigned)T, threads, 0, s>>>(o, ksplit, row_of, k, H, T * k, y, accumulate);
    return hipGetLastError();
}

}  // namespace pcm
