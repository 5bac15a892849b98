// Path mix and combine (Section 4.1's path aggregation in Section 4.3's source-grouped form).
//   mix:     z_(t,b) = sum_{a : (a,b) in Pi(t)} beta_ab u_(t,a)   (a ascending, float32 math)
//            Because the projection W_down[e_b] is linear, applying it once to z_(t,b)
//            equals summing beta_ab W_down[e_b] u_(t,a) over the paths into target b.
//            bf16 layers store z as float16 rows scaled by a power of two (largest element
//            just below 2^14) with the inverse scale kept per row for the down GEMM.
//   combine: y_t = [y_t] + sum_{b ascending} o_(t,b)
// The token's source slots a (U rows) and target slots b (z / o rows) are the same k
// top-k slots for the vanilla-compatible router, and the distinct sources and targets of
// the selected paths for the scored router.
// One workgroup per token; each thread owns 8 consecutive columns.
#include "internal.h"

namespace pcm {
namespace {

// U is read once, by the mix: its loads are non-temporal
__device__ inline void load8(const float* p, float* v) {
    const floatx4 a = __builtin_nontemporal_load((const floatx4*)p);
    const floatx4 b = __builtin_nontemporal_load((const floatx4*)(p + 4));
    v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3]; v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
}

struct TokenPaths {
    uint64_t bits;           // bit a*K + b: source slot a feeds target slot b
    int64_t src[kMaxK];      // U row of each source slot
    int64_t tgt[kMaxK];      // z / o row of each target slot
    const float* beta;       // [K,K] (NULL: weight 1)
    int ns, nt, K;
};

__device__ inline int64_t clamp_row(int64_t r, int64_t R) { return r < 0 ? 0 : (r >= R ? R - 1 : r); }

__device__ inline TokenPaths token_paths(const MixMap& m, int64_t t) {
    TokenPaths p;
    if (m.bits == nullptr) {  // identity: one row per token, weight 1
        p.bits = 1;
        p.src[0] = p.tgt[0] = t;
        p.beta = nullptr;
        p.ns = p.nt = p.K = 1;
        return p;
    }
    p.K = m.K;
    p.ns = m.n_src ? m.n_src[t] : m.K;
    p.nt = m.n_tgt ? m.n_tgt[t] : m.K;
    p.ns = p.ns < 0 ? 0 : (p.ns > m.K ? m.K : p.ns);
    p.nt = p.nt < 0 ? 0 : (p.nt > m.K ? m.K : p.nt);
    p.bits = m.bits[t];
#pragma unroll
    for (int a = 0; a < kMaxK; ++a) {
        p.src[a] = a < p.ns ? clamp_row(m.src_row[t * m.K + a], m.R_src) : 0;
        p.tgt[a] = a < p.nt ? clamp_row(m.tgt_row[t * m.K + a], m.R_tgt) : 0;
    }
    p.beta = m.beta + t * m.K * m.K;
    return p;
}

// z values of 8 columns starting at c for every target b of the token
__device__ inline void mix8(const float* __restrict__ u, const TokenPaths& p, int F, int c,
                            float (&z)[kMaxK][8]) {
    float ua[kMaxK][8];
#pragma unroll
    for (int a = 0; a < kMaxK; ++a)
        if (a < p.ns) load8(u + p.src[a] * F + c, ua[a]);
#pragma unroll
    for (int b = 0; b < kMaxK; ++b) {
        if (b >= p.nt) break;
#pragma unroll
        for (int i = 0; i < 8; ++i) z[b][i] = 0.f;
#pragma unroll
        for (int a = 0; a < kMaxK; ++a) {
            if (a < p.ns && ((p.bits >> (a * p.K + b)) & 1)) {
                const float w = p.beta ? p.beta[a * p.K + b] : 1.0f;
#pragma unroll
                for (int i = 0; i < 8; ++i) z[b][i] = fmaf(w, ua[a][i], z[b][i]);
            }
        }
    }
}

template <bool F16>
__global__ __launch_bounds__(256) void mix_kernel(const float* __restrict__ u, void* __restrict__ z,
                                                  float* __restrict__ zscale, MixMap m, int F) {
    const int64_t t = blockIdx.x;
    if (m.live && t >= *m.live) return;  // whole workgroup
    const TokenPaths p = token_paths(m, t);
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
                if (b < p.nt)
#pragma unroll
                    for (int i = 0; i < 8; ++i) mx[b] = fmaxf(mx[b], fabsf(zz[b][i]));
        }
        __shared__ float red[kMaxK][4];
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
        for (int b = 0; b < kMaxK; ++b) {
            if (b >= p.nt) break;
            // magnitudes are >= 0 (NaN never enters mx), so their bits order as the values
            const float v = __uint_as_float(wave_max_u32(__float_as_uint(mx[b])));
            if (lane == 0) red[b][wave] = v;
        }
        __syncthreads();
        const int nw = (blockDim.x + 63) / 64;
#pragma unroll
        for (int b = 0; b < kMaxK; ++b) {
            if (b >= p.nt) break;
            float v = 0.f;
            for (int w = 0; w < nw; ++w) v = fmaxf(v, red[b][w]);
            // scale = 2^(kZScaleExp - e) with v < 2^e, so every |z * scale| < 2^kZScaleExp
            int e = 0;
            if (v > 0.f) frexpf(v, &e);
            int sh = kZScaleExp - e;
            sh = sh > 126 ? 126 : (sh < -126 ? -126 : sh);
            scale[b] = ldexpf(1.0f, sh);
            if (threadIdx.x == 0) zscale[p.tgt[b]] = ldexpf(1.0f, -sh);
        }
    }
    // pass 2 (only pass for float32 layers): store z
    for (int c = threadIdx.x * 8; c < F; c += blockDim.x * 8) {
        float zz[kMaxK][8];
        mix8(u, p, F, c, zz);
#pragma unroll
        for (int b = 0; b < kMaxK; ++b) {
            if (b >= p.nt) break;
            if (F16) {
                uint32_t w[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const _Float16 lo = (_Float16)(zz[b][2 * i] * scale[b]);
                    const _Float16 hi = (_Float16)(zz[b][2 * i + 1] * scale[b]);
                    w[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) |
                           ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
                }
                *(uint4*)((uint16_t*)z + p.tgt[b] * F + c) = make_uint4(w[0], w[1], w[2], w[3]);
            } else {
                float* dst = (float*)z + p.tgt[b] * F + c;
                *(float4*)dst = make_float4(zz[b][0], zz[b][1], zz[b][2], zz[b][3]);
                *(float4*)(dst + 4) = make_float4(zz[b][4], zz[b][5], zz[b][6], zz[b][7]);
            }
        }
    }
}

// Single-pass form of the float16 mix: each thread keeps its ITER column chunks (CPT columns
// each) of every target row in registers (KK >= the token's target count), so U is read once;
// then the row maxima are reduced over the workgroup and the scaled rows stored. Eight target
// rows take 4-column chunks: with 8-column chunks a thread held 128 values and spilled.
template <int KK, int ITER, int CPT>
__global__ __launch_bounds__(1024) void mix_regs_kernel(const float* __restrict__ u,
                                                        uint16_t* __restrict__ z,
                                                        float* __restrict__ zscale, MixMap m,
                                                        int F) {
    const int64_t t = blockIdx.x;
    if (m.live && t >= *m.live) return;  // whole workgroup
    const TokenPaths p = token_paths(m, t);
    float zz[ITER][KK][CPT];
    float mx[KK];
#pragma unroll
    for (int b = 0; b < KK; ++b) mx[b] = 0.f;
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
#pragma unroll
        for (int b = 0; b < KK; ++b)
#pragma unroll
            for (int i = 0; i < CPT; ++i) zz[it][b][i] = 0.f;
        const int c = (threadIdx.x + it * blockDim.x) * CPT;
        if (c >= F) continue;
        // sources in ascending order, each row's 8 values added to every target it feeds;
        // the loads of all sources are issued before the first multiply-add
        float ua[KK][CPT];
#pragma unroll
        for (int a = 0; a < KK; ++a)
            if (a < p.ns) {
                if constexpr (CPT == 8) {
                    load8(u + p.src[a] * F + c, ua[a]);
                } else {
                    const floatx4 v = __builtin_nontemporal_load((const floatx4*)(u + p.src[a] * F + c));
                    ua[a][0] = v[0]; ua[a][1] = v[1]; ua[a][2] = v[2]; ua[a][3] = v[3];
                }
            }
#pragma unroll
        for (int a = 0; a < KK; ++a) {
            if (a >= p.ns) break;
#pragma unroll
            for (int b = 0; b < KK; ++b) {
                if (b < p.nt && ((p.bits >> (a * p.K + b)) & 1)) {
                    const float w = p.beta ? p.beta[a * p.K + b] : 1.0f;
#pragma unroll
                    for (int i = 0; i < CPT; ++i) zz[it][b][i] = fmaf(w, ua[a][i], zz[it][b][i]);
                }
            }
        }
#pragma unroll
        for (int b = 0; b < KK; ++b)
#pragma unroll
            for (int i = 0; i < CPT; ++i) mx[b] = fmaxf(mx[b], fabsf(zz[it][b][i]));
    }
    __shared__ float red[KK][16];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int b = 0; b < KK; ++b) {
        // magnitudes are >= 0 (NaN never enters mx), so their bits order as the values
        const float v = __uint_as_float(wave_max_u32(__float_as_uint(mx[b])));
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
        if (threadIdx.x == 0 && b < p.nt) zscale[p.tgt[b]] = ldexpf(1.0f, -sh);
    }
#pragma unroll
    for (int it = 0; it < ITER; ++it) {
        const int c = (threadIdx.x + it * blockDim.x) * CPT;
        if (c >= F) continue;
#pragma unroll
        for (int b = 0; b < KK; ++b) {
            if (b >= p.nt) break;
            uint32_t w[CPT / 2];
#pragma unroll
            for (int i = 0; i < CPT / 2; ++i) {
                const _Float16 lo = (_Float16)(zz[it][b][2 * i] * scale[b]);
                const _Float16 hi = (_Float16)(zz[it][b][2 * i + 1] * scale[b]);
                w[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) |
                       ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
            }
            if constexpr (CPT == 8) *(uint4*)(z + p.tgt[b] * F + c) = make_uint4(w[0], w[1], w[2], w[3]);
            else *(uint2*)(z + p.tgt[b] * F + c) = make_uint2(w[0], w[1]);
        }
    }
}

template <int KK, int ITER, int CPT>
void launch_mix_regs(unsigned blocks, int threads, const float* u, void* z, float* zscale,
                     const MixMap& m, int F, hipStream_t s) {
    mix_regs_kernel<KK, ITER, CPT><<<blocks, threads, 0, s>>>(u, (uint16_t*)z, zscale, m, F);
}

// y_t = [y_t] + sum over targets b (ascending) and K slices q (ascending) of o_(t,b) slice q.
// One token per workgroup; each thread takes two 4-column chunks and issues the loads of
// every row of both before the first add. The register copy is sized by the layer (KMAX >= the
// target count, KS = the K slices, 1 or 2; KS = 0: a loop for more slices): sized for the
// largest case, it held 128 values and let three waves run per SIMD. o is read once, so its
// loads are non-temporal.
template <int KMAX, int KS>
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ o, int ksplit,
                                                      MixMap m, int H, float* __restrict__ y,
                                                      int accumulate) {
    const int64_t t = blockIdx.x;
    const TokenPaths p = token_paths(m, t);
    constexpr int CU = 2;
    // column blocks of CB columns (CU chunks of 4 per thread): blockIdx.y takes every
    // gridDim.y-th block
    const int CB = blockDim.x * 4 * CU;
    for (int c0 = blockIdx.y * CB + threadIdx.x * 4; c0 < H; c0 += gridDim.y * CB) {
        float4 s[CU];
        if constexpr (KS > 0) {   // ksplit == KS, at most KMAX targets: loads held in registers
            float4 v[CU][KMAX][KS];
#pragma unroll
            for (int u = 0; u < CU; ++u) {
                const int c = c0 + u * blockDim.x * 4;
#pragma unroll
                for (int b = 0; b < KMAX; ++b)
#pragma unroll
                    for (int q = 0; q < KS; ++q)
                        if (c < H && b < p.nt) {
                            const floatx4 w = __builtin_nontemporal_load(
                                (const floatx4*)(o + (q * m.R_tgt + p.tgt[b]) * H + c));
                            v[u][b][q] = make_float4(w[0], w[1], w[2], w[3]);
                        }
            }
#pragma unroll
            for (int u = 0; u < CU; ++u) {
                s[u] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int b = 0; b < KMAX; ++b)
#pragma unroll
                    for (int q = 0; q < KS; ++q)
                        if (b < p.nt) {
                            s[u].x += v[u][b][q].x; s[u].y += v[u][b][q].y;
                            s[u].z += v[u][b][q].z; s[u].w += v[u][b][q].w;
                        }
            }
        } else {
#pragma unroll
            for (int u = 0; u < CU; ++u) {
                const int c = c0 + u * blockDim.x * 4;
                s[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (c >= H) continue;
                for (int b = 0; b < p.nt; ++b)
                    for (int q = 0; q < ksplit; ++q) {
                        const float4 w = *(const float4*)(o + (q * m.R_tgt + p.tgt[b]) * H + c);
                        s[u].x += w.x; s[u].y += w.y; s[u].z += w.z; s[u].w += w.w;
                    }
            }
        }
#pragma unroll
        for (int u = 0; u < CU; ++u) {
            const int c = c0 + u * blockDim.x * 4;
            if (c >= H) continue;
            float4 r = s[u];
            float4* dst = (float4*)(y + t * H + c);
            if (accumulate) {
                const float4 old = *dst;
                r.x = old.x + r.x; r.y = old.y + r.y; r.z = old.z + r.z; r.w = old.w + r.w;
            }
            *dst = r;
        }
    }
}

// h = round(h + y) elementwise (h bf16, round to nearest even, or f32)
__global__ __launch_bounds__(256) void residual_kernel(void* __restrict__ h,
                                                       const float* __restrict__ y, int64_t N,
                                                       int bf16) {
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (i >= N) return;
    const float4 v = *(const float4*)(y + i);
    if (bf16) {
        uint16_t* hb = (uint16_t*)h + i;
        const uint2 q = *(const uint2*)hb;
        const float a0 = bf16_bits_to_f32(q.x & 0xFFFFu), a1 = bf16_bits_to_f32(q.x >> 16);
        const float a2 = bf16_bits_to_f32(q.y & 0xFFFFu), a3 = bf16_bits_to_f32(q.y >> 16);
        uint2 r;
        r.x = (uint32_t)f32_to_bf16_rne(a0 + v.x) | ((uint32_t)f32_to_bf16_rne(a1 + v.y) << 16);
        r.y = (uint32_t)f32_to_bf16_rne(a2 + v.z) | ((uint32_t)f32_to_bf16_rne(a3 + v.w) << 16);
        *(uint2*)hb = r;
    } else {
        float4* hf = (float4*)((float*)h + i);
        const float4 a = *hf;
        *hf = make_float4(a.x + v.x, a.y + v.y, a.z + v.z, a.w + v.w);
    }
}

}  // namespace

hipError_t launch_residual(void* h, const float* y, int64_t N, bool bf16, hipStream_t s) {
    if (N == 0) return hipSuccess;
    residual_kernel<<<(unsigned)ceil_div(N / 4, 256), 256, 0, s>>>(h, y, N, bf16 ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_mix(const float* u, void* z, float* zscale, const MixMap& m, int64_t T, int F,
                      hipStream_t s) {
    if (T == 0) return hipSuccess;
    const int threads = F / 8 >= 256 ? 256 : ((F / 8 + 63) / 64) * 64;
    const int kslots = m.bits ? m.K : 1;
    if (zscale) {
        // single pass when a thread's share of every target row fits in 64 registers
        const int kk = kslots <= 1 ? 1 : (kslots <= 2 ? 2 : (kslots <= 4 ? 4 : 8));
        const int cpt = (kk == 8 && F / 4 <= 1024) ? 4 : 8;   // columns per thread
        const int chunks = F / cpt;
        const int threads_r = chunks >= 1024 ? 1024 : ((chunks + 63) / 64) * 64;
        const int iter = (chunks + threads_r - 1) / threads_r;
        const int it = iter <= 1 ? 1 : (iter <= 2 ? 2 : (iter <= 4 ? 4 : (iter <= 8 ? 8 : 16)));  // 16: two-pass
        const unsigned blocks = (unsigned)T;
        if (kk * it <= 8) {
            auto go = [&](auto fn) {
                fn(blocks, threads_r, u, z, zscale, m, F, s);
                return hipGetLastError();
            };
            switch (kk * 100 + it) {
                case 101: return go(launch_mix_regs<1, 1, 8>);
                case 102: return go(launch_mix_regs<1, 2, 8>);
                case 104: return go(launch_mix_regs<1, 4, 8>);
                case 108: return go(launch_mix_regs<1, 8, 8>);
                case 201: return go(launch_mix_regs<2, 1, 8>);
                case 202: return go(launch_mix_regs<2, 2, 8>);
                case 204: return go(launch_mix_regs<2, 4, 8>);
                case 401: return go(launch_mix_regs<4, 1, 8>);
                case 402: return go(launch_mix_regs<4, 2, 8>);
                case 801: return cpt == 4 ? go(launch_mix_regs<8, 1, 4>) : go(launch_mix_regs<8, 1, 8>);
                default: break;
            }
        }
        mix_kernel<true><<<(unsigned)T, threads, 0, s>>>(u, z, zscale, m, F);
    } else
        mix_kernel<false><<<(unsigned)T, threads, 0, s>>>(u, z, zscale, m, F);
    return hipGetLastError();
}

hipError_t launch_combine(const float* o, int ksplit, const MixMap& m, int64_t T, int H, float* y,
                          int accumulate, hipStream_t s) {
    if (T == 0) return hipSuccess;
    const int threads = H / 4 >= 256 ? 256 : ((H / 4 + 63) / 64) * 64;
    const int K = m.bits ? m.K : 1;
    const int kmax = K <= 1 ? 1 : (K <= 2 ? 2 : (K <= 4 ? 4 : 8));
    const int ks = ksplit == 1 || ksplit == 2 ? ksplit : 0;
    // a few tokens (decode): the columns of a token are split over several workgroups, so that
    // the chip is not left to a handful of long-running ones
    const int col_blocks = (H + threads * 8 - 1) / (threads * 8);
    const int split = T >= 1024 ? 1 : col_blocks;
    auto go = [&](auto kern) {
        kern<<<dim3((unsigned)T, (unsigned)split), threads, 0, s>>>(o, ksplit, m, H, y, accumulate);
        return hipGetLastError();
    };
    switch (kmax * 10 + ks) {
        case 11: return go(combine_kernel<1, 1>);
        case 12: return go(combine_kernel<1, 2>);
        case 21: return go(combine_kernel<2, 1>);
        case 22: return go(combine_kernel<2, 2>);
        case 41: return go(combine_kernel<4, 1>);
        case 42: return go(combine_kernel<4, 2>);
        case 81: return go(combine_kernel<8, 1>);
        case 82: return go(combine_kernel<8, 2>);
        default: return go(combine_kernel<8, 0>);
    }
}

}  // namespace pcm
