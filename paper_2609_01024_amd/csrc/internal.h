// Internal declarations shared by the HIP sources of libpcomoe (not part of the ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pcm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kMaxK = 8;
constexpr int kMaxN = 256;
constexpr int kPathBlock = 1024;  // tokens per block of the path/index build

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// float32 -> bfloat16 bits, round to nearest even (inputs are finite).
__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ inline float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Launchers (each returns hipGetLastError() of its launches).
hipError_t launch_route(const float* logits, int64_t T, int n, int k, int32_t* ids, float* w,
                        hipStream_t s);
hipError_t launch_build_paths(const int32_t* ids, const float* w, const uint8_t* mask, int64_t T,
                              int n, int k, int beta_mode, uint64_t* bits, float* beta,
                              int32_t* offsets, int32_t* row_token, int32_t* row_slot,
                              int32_t* row_of, int32_t* block_counts, hipStream_t s);
size_t build_paths_ws_bytes(int64_t T, int n);

enum GemmMode { kExpand = 0, kDownStore = 1, kDownAccum = 2 };

// Layout of a bf16 layer's projection input z (and of a dense FFN's SwiGLU output): a
// float32 value v is carried as the bfloat16 pair hi = rn(v), lo = rn(v - hi), which
// represents v to about 2^-17 relative. Row r holds F/32 blocks of [32 hi | 32 lo], so one
// 32-wide K step of the down GEMM reads 128 contiguous bytes of a row.
// The down GEMM multiplies both halves by the same weight tile, so the projection sees
// the float32 value instead of a single bfloat16 rounding of it.
constexpr int kSplitBlock = 32;

struct GemmArgs {
    const void* a;              // expand: x [T,H] (rows gathered); down: z (split bf16 or f32)
    const void* b0;             // expand: w_gate [n,F,H]; down: w_down [n,H,F]
    const void* b1;             // expand: w_up [n,F,H]; down: unused
    void* out;                  // expand: u [R,F] f32 (or split bf16, see split_out);
                                // down-store: o [R,H] f32; down-accum: y [R,H] f32
    const int32_t* offsets;     // [n+1] rows of each group (NULL: one group of a_rows rows)
    const int32_t* gather;      // expand: row_token [R] (NULL: identity); down: unused
    int64_t a_rows;             // rows of `a` (gathered indices are clamped to it)
    int n;                      // groups
    int K;                      // contraction length (H for expand, F for down)
    int N;                      // output columns (F for expand, H for down)
    int accumulate;             // down-accum: add into out
    int split_out;              // expand (bf16): write u as split hi/lo pairs instead of f32
};

hipError_t launch_gemm_bf16(GemmMode mode, const GemmArgs& g, int64_t R, hipStream_t s);
hipError_t launch_gemm_f32(GemmMode mode, const GemmArgs& g, int64_t R, hipStream_t s);

// z_(t,b) = sum_a beta_ab u_(t,a); u is f32 [R,F]; z is split bf16 (split) or f32 [R,F].
hipError_t launch_mix(bool split, const float* u, void* z, const uint64_t* bits, const float* beta,
                      const int32_t* row_of, int64_t T, int k, int F, hipStream_t s);
hipError_t launch_combine(const float* o, const int32_t* row_of, int64_t T, int k, int H,
                          float* y, int accumulate, hipStream_t s);

}  // namespace pcm
