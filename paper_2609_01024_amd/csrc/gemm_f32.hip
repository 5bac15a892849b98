// Grouped float32 GEMMs for float32 layers (same operations as the bf16 kernels:
// expansion with fused SwiGLU, down projection store or accumulate). Vector FMA with
// LDS tiles of 64 rows x 64 weight rows x 16 K; each thread owns a 4 x 4 block. Small
// float32 layers are bound by launch latency, not arithmetic.
#include "internal.h"

namespace pcm {
namespace {

constexpr int FBM = 64, FBN = 64, FBK = 16;

__device__ bool find_tile_f32(const int32_t* __restrict__ offsets, int n, int64_t a_rows, int64_t mt,
                              int* s_tile) {
    if (offsets == nullptr) {
        if (mt * FBM >= a_rows) return false;
        s_tile[0] = 0;
        s_tile[1] = (int)(mt * FBM);
        s_tile[2] = (int)min<int64_t>(a_rows, (mt + 1) * FBM);
        return true;
    }
    if (threadIdx.x == 0) {
        s_tile[0] = -1;
        int64_t start = 0;
        for (int x = 0; x < n; ++x) {
            const int b = offsets[x], c = (int)ceil_div(offsets[x + 1] - b, FBM);
            if (mt >= start && mt < start + c) {
                const int r0 = b + (int)(mt - start) * FBM;
                s_tile[0] = x;
                s_tile[1] = r0;
                s_tile[2] = min(offsets[x + 1], r0 + FBM);
                break;
            }
            start += c;
        }
    }
    __syncthreads();
    return s_tile[0] >= 0;
}

template <int MODE>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs g, int64_t mt_upper) {
    __shared__ float As[FBK][FBM + 4];
    __shared__ float Bs[FBK][FBN + 4];
    __shared__ int s_tile[3];
    const int64_t mt = blockIdx.x % mt_upper;
    const int ntile = (int)(blockIdx.x / mt_upper);
    if (!find_tile_f32(g.offsets, g.n, g.a_rows, mt, s_tile)) return;
    const int e = s_tile[0], row0 = s_tile[1], row1 = s_tile[2];
    const int tid = threadIdx.x, tm = tid / 16, tn = tid % 16;
    const int K = g.K, N = g.N;
    constexpr int kOutCols = (MODE == kExpand) ? FBN / 2 : FBN;

    // staged element: row = tid / 4, k quad = tid % 4
    const int lrow = tid / 4, kq = tid % 4;
    const float* aptr = nullptr;
    {
        const int r = row0 + lrow;
        if (r < row1) {
            int64_t src = r;
            if (g.gather) {
                src = g.gather[r];
                src = src < 0 ? 0 : (src >= g.a_rows ? g.a_rows - 1 : src);
            }
            aptr = (const float*)g.a + src * K + kq * 4;
        }
    }
    const float* bptr = nullptr;
    if (MODE == kExpand) {
        const int half = lrow / (FBN / 2), f = ntile * kOutCols + lrow % (FBN / 2);
        if (f < N) bptr = (const float*)(half ? g.b1 : g.b0) + ((int64_t)e * N + f) * K + kq * 4;
    } else {
        const int h = ntile * kOutCols + lrow;
        if (h < N) bptr = (const float*)g.b0 + ((int64_t)e * N + h) * K + kq * 4;
    }
    int bcol[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
        bcol[j] = (MODE == kExpand) ? (j < 2 ? tn * 2 + j : FBN / 2 + tn * 2 + j - 2) : tn * 4 + j;

    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += FBK) {
        const float4 av = aptr ? *(const float4*)(aptr + k0) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 bv = bptr ? *(const float4*)(bptr + k0) : make_float4(0.f, 0.f, 0.f, 0.f);
        As[kq * 4 + 0][lrow] = av.x; As[kq * 4 + 1][lrow] = av.y;
        As[kq * 4 + 2][lrow] = av.z; As[kq * 4 + 3][lrow] = av.w;
        Bs[kq * 4 + 0][lrow] = bv.x; Bs[kq * 4 + 1][lrow] = bv.y;
        Bs[kq * 4 + 2][lrow] = bv.z; Bs[kq * 4 + 3][lrow] = bv.w;
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < FBK; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][tm * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Bs[kk][bcol[j]];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = row0 + tm * 4 + i;
        if (r >= row1) continue;
        float* out = (float*)g.out + (int64_t)r * N;
        if (MODE == kExpand) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int f = ntile * kOutCols + tn * 2 + j;
                if (f < N) {
                    const float gt = acc[i][j], up = acc[i][j + 2];
                    out[f] = gt / (1.0f + expf(-gt)) * up;
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int h = ntile * kOutCols + tn * 4 + j;
                if (h < N) out[h] = (MODE == kDownAccum && g.accumulate) ? out[h] + acc[i][j] : acc[i][j];
            }
        }
    }
}

}  // namespace

hipError_t launch_gemm_f32(GemmMode mode, const GemmArgs& g, int64_t R, hipStream_t s) {
    const int64_t mt_upper = g.offsets ? ceil_div(R, FBM) + g.n : ceil_div(R, FBM);
    const int out_cols = mode == kExpand ? FBN / 2 : FBN;
    const int64_t grid = mt_upper * ceil_div(g.N, out_cols);
    if (grid <= 0) return hipSuccess;
    switch (mode) {
        case kExpand: gemm_f32_kernel<kExpand><<<(unsigned)grid, 256, 0, s>>>(g, mt_upper); break;
        case kDownStore: gemm_f32_kernel<kDownStore><<<(unsigned)grid, 256, 0, s>>>(g, mt_upper); break;
        default: gemm_f32_kernel<kDownAccum><<<(unsigned)grid, 256, 0, s>>>(g, mt_upper); break;
    }
    return hipGetLastError();
}

}  // namespace pcm
