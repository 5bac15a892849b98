// Per-path execution of the layer (the baselines of the paper's execution-engine ablation):
//   reuse = 1: U_i once per (token, source) (Section 4.3's source-grouped reuse), then one
//              projection per path, o_(t,a,b) = W_down[e_b] u_(t,a) (Eq. of Section 4.1 /
//              Section 4.3 evaluated path by path, without mixing paths that share a target);
//   reuse = 0: additionally one expansion per path (no reuse at all).
//   y_t = [y_t] + sum_{(a,b) in Pi, a-major} beta_ab o_(t,a,b).
//
// Path rows come from the top-k dispatch: every row (t, s) of expert e (s the key slot: the
// target b, or the source a) stands for the paths of token t whose key slot is s, so the
// path rows of expert e are contiguous when each row is expanded in place. An exclusive
// scan of the per-row path counts gives every path its row; within a row the paths follow
// the other slot in ascending order.
#include "internal.h"

namespace pcm {
namespace {

// c[r] = number of paths of the token of row r whose key slot is the row's slot.
__global__ __launch_bounds__(256) void path_count_kernel(const uint64_t* __restrict__ bits,
                                                         const int32_t* __restrict__ row_token,
                                                         const int32_t* __restrict__ row_slot,
                                                         int64_t R, int k, int key_is_target,
                                                         int32_t* __restrict__ c) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= R) return;
    const uint64_t b = bits[row_token[r]];
    const int s = row_slot[r];
    int cnt = 0;
    for (int o = 0; o < k; ++o) {
        const int bit = key_is_target ? (o * k + s) : (s * k + o);
        cnt += (int)((b >> bit) & 1);
    }
    c[r] = cnt;
}

// Exclusive scan of c[0..R) into start[0..R) by one 1024-thread workgroup (each thread a
// contiguous segment); path_offsets[e] = start[expert_offsets[e]], path_offsets[n] = total.
__global__ __launch_bounds__(1024) void path_scan_kernel(const int32_t* __restrict__ c, int64_t R,
                                                         const int32_t* __restrict__ expert_offsets,
                                                         int n, int32_t* __restrict__ start,
                                                         int32_t* __restrict__ path_offsets) {
    __shared__ int32_t sums[1024];
    __shared__ int32_t total_s;
    const int tid = threadIdx.x;
    const int64_t seg = (R + 1023) / 1024;
    const int64_t lo = tid * seg, hi = lo + seg < R ? lo + seg : R;
    int32_t s = 0;
    for (int64_t r = lo; r < hi; ++r) s += c[r];
    sums[tid] = s;
    __syncthreads();
    for (int d = 1; d < 1024; d <<= 1) {
        const int32_t v = tid >= d ? sums[tid - d] : 0;
        __syncthreads();
        sums[tid] += v;
        __syncthreads();
    }
    int32_t run = sums[tid] - s;  // exclusive prefix of this segment
    if (tid == 1023) total_s = sums[1023];
    for (int64_t r = lo; r < hi; ++r) {
        start[r] = run;
        run += c[r];
    }
    __syncthreads();
    for (int e = tid; e <= n; e += 1024) {
        const int64_t row = expert_offsets[e];
        path_offsets[e] = e == n ? total_s : (row < R ? start[row] : total_s);
    }
}

// Fill the path rows of row r: path_token[p] = t, path_row_of[t, a*k + b] = p and, when
// gather_src is given, path_gather[p] = gather_src[t, a*k + b] (reuse = 0: the path's own
// expansion row) or row_of[t*k + a] (reuse = 1: the source's expansion row).
__global__ __launch_bounds__(256) void path_fill_kernel(
    const uint64_t* __restrict__ bits, const int32_t* __restrict__ row_token,
    const int32_t* __restrict__ row_slot, const int32_t* __restrict__ row_of,
    const int32_t* __restrict__ start, int64_t R, int k, int key_is_target,
    const int32_t* __restrict__ gather_src, int32_t* __restrict__ path_token,
    int32_t* __restrict__ path_row_of, int32_t* __restrict__ path_gather) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= R) return;
    const int64_t t = row_token[r];
    const uint64_t b = bits[t];
    const int s = row_slot[r];
    int64_t p = start[r];
    for (int o = 0; o < k; ++o) {
        const int a = key_is_target ? o : s, tg = key_is_target ? s : o;
        if (!((b >> (a * k + tg)) & 1)) continue;
        path_token[p] = (int32_t)t;
        path_row_of[t * k * k + a * k + tg] = (int32_t)p;
        if (path_gather)
            path_gather[p] = gather_src ? gather_src[t * k * k + a * k + tg] : row_of[t * k + a];
        ++p;
    }
}

// y_t = [y_t] + sum over the token's paths (a-major) of beta_ab o[path_row_of[t, a, b]].
__global__ __launch_bounds__(256) void combine_paths_kernel(
    const float* __restrict__ o, const uint64_t* __restrict__ bits, const float* __restrict__ beta,
    const int32_t* __restrict__ path_row_of, int k, int H, int64_t P, float* __restrict__ y,
    int accumulate) {
    const int64_t t = blockIdx.x;
    const uint64_t b = bits[t];
    for (int c = threadIdx.x * 4; c < H; c += blockDim.x * 4) {
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int q = 0; q < k * k; ++q) {
            if (!((b >> q) & 1)) continue;
            int64_t p = path_row_of[t * k * k + q];
            p = p < 0 ? 0 : (p >= P ? P - 1 : p);
            const float w = beta[t * k * k + q];
            const float4 v = *(const float4*)(o + p * H + c);
            s.x = fmaf(w, v.x, s.x); s.y = fmaf(w, v.y, s.y);
            s.z = fmaf(w, v.z, s.z); s.w = fmaf(w, v.w, s.w);
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

hipError_t launch_path_rows(const uint64_t* bits, const int32_t* expert_offsets,
                            const int32_t* row_token, const int32_t* row_slot,
                            const int32_t* row_of, int64_t R, int n, int k, int key_is_target,
                            const int32_t* gather_src, int32_t* c, int32_t* start,
                            int32_t* path_offsets, int32_t* path_token, int32_t* path_row_of,
                            int32_t* path_gather, hipStream_t s) {
    if (R == 0) return hipSuccess;
    const unsigned blocks = (unsigned)ceil_div(R, 256);
    path_count_kernel<<<blocks, 256, 0, s>>>(bits, row_token, row_slot, R, k, key_is_target, c);
    path_scan_kernel<<<1, 1024, 0, s>>>(c, R, expert_offsets, n, start, path_offsets);
    path_fill_kernel<<<blocks, 256, 0, s>>>(bits, row_token, row_slot, row_of, start, R, k,
                                            key_is_target, gather_src, path_token, path_row_of,
                                            path_gather);
    return hipGetLastError();
}

hipError_t launch_combine_paths(const float* o, const uint64_t* bits, const float* beta,
                                const int32_t* path_row_of, int64_t T, int k, int H, int64_t P,
                                float* y, int accumulate, hipStream_t s) {
    if (T == 0) return hipSuccess;
    const int threads = H / 4 >= 256 ? 256 : ((H / 4 + 63) / 64) * 64;
    combine_paths_kernel<<<(unsigned)T, threads, 0, s>>>(o, bits, beta, path_row_of, k, H, P, y,
                                                         accumulate);
    return hipGetLastError();
}

}  // namespace pcm
