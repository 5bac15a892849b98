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
constexpr int kPathBlock = 256;   // tokens per block of the path/index build

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// float32 -> bfloat16 bits, round to nearest even (inputs are finite).
__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ inline float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Largest 32-bit value across the wavefront, the same on every lane (all 64 lanes active):
// DPP moves that pair lane i with i^1, i^2, its mirror in 8 and its mirror in 16 leave each
// row of 16 lanes with its maximum (each move folds into the max instruction); two row
// broadcasts then fold row 0 into row 1 and row 2 into row 3 (lane 15 of a row to the next
// row), and rows 0-1 into rows 2-3 (lane 31 to both), so lane 63 holds the wave's maximum,
// which one read into a scalar register hands to every lane.
template <int CTRL>
__device__ inline uint32_t dpp_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}
__device__ inline uint32_t wave_max_u32(uint32_t v) {
    v = max(v, dpp_u32<0xB1>(v));   // quad_perm [1,0,3,2]: lane ^ 1
    v = max(v, dpp_u32<0x4E>(v));   // quad_perm [2,3,0,1]: lane ^ 2
    v = max(v, dpp_u32<0x141>(v));  // row_half_mirror: the other quad of 8
    v = max(v, dpp_u32<0x140>(v));  // row_mirror: the other half of 16
    // The row broadcasts write only the rows their row mask names, the other rows keep v, which
    // the compiler's DPP intrinsics would express as a copy, a move and a max; as one
    // instruction each (the two wait states a DPP read of a VALU result needs come first).
    asm volatile(
        "s_nop 1\n\t"
        "v_max_u32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_max_u32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
        "s_nop 1"
        : "+v"(v));
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}
// Inclusive prefix sum across the wavefront (all 64 lanes active): lane l gets v[0] + ... +
// v[l]. Within each row of 16 lanes, adds of the value shifted by 1, 2 and 3 lanes (lanes
// shifted in from outside the row read 0) leave sums of up to 4 lanes; adds of the running sum
// shifted by 4 into the upper three banks of 4 lanes and by 8 into the upper two complete each
// row; the row broadcasts used by wave_max_u32 then carry rows 0 and 2 into rows 1 and 3, and
// rows 0-1 into rows 2-3.
__device__ inline int wave_incl_scan_i32(int v) {
    int s = v + __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true);  // row_shr:1
    s += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true);          // row_shr:2
    s += __builtin_amdgcn_update_dpp(0, v, 0x113, 0xF, 0xF, true);          // row_shr:3
    asm volatile(
        "s_nop 1\n\t"
        "v_add_u32_dpp %0, %0, %0 row_shr:4 bank_mask:0xe\n\t"
        "s_nop 1\n\t"
        "v_add_u32_dpp %0, %0, %0 row_shr:8 bank_mask:0xc\n\t"
        "s_nop 1\n\t"
        "v_add_u32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa\n\t"
        "s_nop 1\n\t"
        "v_add_u32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc\n\t"
        "s_nop 1"
        : "+v"(s));
    return s;
}
// Largest 64-bit value across the wavefront: the largest high word, then, when more than
// one lane holds it, the largest low word among those lanes.
__device__ inline uint64_t wave_max_u64(uint64_t v) {
    const uint32_t hv = (uint32_t)(v >> 32), lv = (uint32_t)v;
    const uint32_t hi = wave_max_u32(hv);
    const uint64_t holders = __ballot(hv == hi);
    uint32_t lo;
    if (__popcll(holders) == 1)
        lo = (uint32_t)__builtin_amdgcn_readlane((int)lv, __ffsll((unsigned long long)holders) - 1);
    else
        lo = wave_max_u32(hv == hi ? lv : 0u);
    return ((uint64_t)hi << 32) | lo;
}

// Launchers (each returns hipGetLastError() of its launches).
hipError_t launch_route(const float* logits, int64_t T, int n, int k, int32_t* ids, float* w,
                        hipStream_t s);
// logits = x W_r^T (float32 accumulate; written when logits != NULL) fused with the top-k;
// bf16 uses `part` (router_ws_bytes) for the K-split partial sums.
hipError_t launch_router(bool bf16, const void* x, const void* wr, int64_t T, int H, int n, int k,
                         float* logits, int32_t* ids, float* w, float* part, hipStream_t s);
size_t router_ws_bytes(int64_t T, int H, int n);
hipError_t launch_build_paths(const int32_t* ids, const float* w, const uint8_t* mask, int64_t T,
                              int n, int k, int beta_mode, uint64_t* bits, float* beta,
                              int32_t* offsets, int32_t* row_token, int32_t* row_slot,
                              int32_t* row_of, int32_t* block_counts, hipStream_t s);
size_t build_paths_ws_bytes(int64_t T, int n);
// The fused indexing operation (route, path table, dispatch layout) over a packed mask
// [n][ceil(n/64)] u64, and the packing of a u8 mask.
hipError_t launch_mask_pack(const uint8_t* mask, int n, uint64_t* packed, hipStream_t s);
hipError_t launch_route_paths(const float* logits, const uint64_t* packed, int64_t T, int n, int k,
                              int beta_mode, int32_t* ids, float* w, uint64_t* bits, float* beta,
                              int32_t* offsets, int32_t* row_token, int32_t* row_slot,
                              int32_t* row_of, void* ws, hipStream_t s);
size_t route_paths_ws_bytes(int64_t T, int n);

enum GemmMode { kExpand = 0, kDownStore = 1, kDownAccum = 2 };
// Flag on a projection mode inside the bf16 GEMM kernels: the projection weights are already
// float16 (GemmArgs::b_f16), so the kernels use them as read instead of widening each bf16
// fragment. The flag only ever sits on kDownStore or kDownAccum.
constexpr int kHalfW = 4;
constexpr int base_mode(int mode) { return mode & 3; }
constexpr bool half_weights(int mode) { return (mode & kHalfW) != 0; }

// Projection input of a bf16 layer. z (float32 in the mix) is stored as float16 after
// multiplying row r by a power of two chosen from the row's largest |z| (so the largest
// element sits just below 2^14); row_scale[r] holds the inverse, applied exactly in the
// down GEMM's epilogue. float16 keeps 11 significant bits, eight times the precision of
// a single bfloat16 rounding, and runs at the bfloat16 MFMA rate; the row scaling keeps
// any activation magnitude inside float16's range.
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));
constexpr int kZScaleExp = 14;

struct GemmArgs {
    const void* a;              // expand: x [T,H] (rows gathered); down: z [R,F] (f16 or f32)
    const void* b0;             // expand: w_gate [n,F,H]; down: w_down [n,H,F]
    const void* b1;             // expand: w_up [n,F,H]; down: unused
    void* out;                  // expand: u [R,F] f32; down-store: o [R,H] f32;
                                // down-accum: y [R,H] f32
    const float* row_scale;     // down (bf16 layers): inverse scale of each z row
    const int32_t* offsets;     // [n+1] rows of each group (NULL: one group of a_rows rows)
    const int32_t* gather;      // row of `a` behind each output row (NULL: identity); the
                                // down modes' row_scale follows the gathered row
    int64_t a_rows;             // rows of `a` (gathered indices are clamped to it)
    int n;                      // groups
    int K;                      // contraction length (H for expand, F for down)
    int N;                      // output columns (F for expand, H for down)
    int accumulate;             // down-accum: add into out
    int ksplit;                 // down-store: K split into ksplit slices, slice s writes
                                // out + s * rows_total * N (the combine adds the slices)
    int64_t rows_total;         // rows of `out` per slice (down-store with ksplit > 1)
    int b_f16;                  // down (bf16 layers): b0 holds float16 weights (widened once,
                                // as pcm_widen_f16 does) instead of bf16 ones
};

// Kernel choices of a bf16 GEMM launch that a caller may force (tests and measurement, through
// the *_tuned entry points). The defaults choose by shape; every choice gives the same bits.
struct GemmTune {
    char tile = 0;          // 0: by mean rows per group; 'S' streaming, 'M' medium, 'L' large tiles
    int order = -1;         // large tiles: -1 by shape; 0 grouped, 1 longest first, 2 expert-major
    int window = 0;         // expert-major window (0: 8)
    int group_n = 0;        // N tiles per group of the grouped order (0: 4)
    int stream_depth = -1;  // streaming kernel: -1 by mode; 0 register ring; 2, 3, 4, 6 LDS slots
};

// Number of K slices the projection of R rows uses (1 or 2): split when the output tiles
// alone would leave the chip's 256 compute units idle for much of the last round. `tile` is
// a forced tile kernel (GemmTune::tile) or 0.
int down_ksplit(int64_t R, int n, int H, int F, char tile);

hipError_t launch_gemm_bf16(GemmMode mode, const GemmArgs& g, int64_t R, hipStream_t s,
                            const GemmTune& tune);
hipError_t launch_gemm_f32(GemmMode mode, const GemmArgs& g, int64_t R, hipStream_t s);

// Per-token path structure read by the mix and the combine. Token t has n_src[t] source
// slots a (U rows src_row[t*K + a]) and n_tgt[t] target slots b (z and o rows
// tgt_row[t*K + b]); bit a*K + b of bits[t] marks the path a -> b, weighted by
// beta[t, a, b]. bits == NULL: identity (one slot, z_t = u_t, weight 1).
struct MixMap {
    const uint64_t* bits;
    const float* beta;
    const int32_t* src_row;
    const int32_t* tgt_row;
    const int32_t* n_src;   // NULL: K
    const int32_t* n_tgt;   // NULL: K
    int K;
    int64_t R_src, R_tgt;   // row counts of U and of z / o (indices are clamped to them)
    const int32_t* live;    // identity only: rows from *live on are skipped (NULL: none)
};

// z_(t,b) = sum_a beta_ab u_(t,a); u is f32; z is f16 (scaled rows, inverse scales in
// zscale) when zscale != NULL, else f32.
hipError_t launch_mix(const float* u, void* z, float* zscale, const MixMap& m, int64_t T, int F,
                      hipStream_t s);
// y_t = [y_t] + sum_b o_(t,b), o holding ksplit slices of R_tgt rows.
hipError_t launch_combine(const float* o, int ksplit, const MixMap& m, int64_t T, int H, float* y,
                          int accumulate, hipStream_t s);

// h = round(h + y) over N elements (N a multiple of 4; h bf16 or f32).
hipError_t launch_residual(void* h, const float* y, int64_t N, bool bf16, hipStream_t s);
// bf16 -> float16 (round to nearest even; the conversion the projection applies to each bf16
// weight fragment), count values.
hipError_t launch_widen_f16(const uint16_t* src, int64_t count, uint16_t* dst, hipStream_t s);

// Grouped dispatch of counts[t] <= K distinct experts per token (ids [T,K]).
hipError_t launch_dispatch(const int32_t* ids, const int32_t* counts, int64_t T, int n, int K,
                           int32_t* offsets, int32_t* row_token, int32_t* row_slot,
                           int32_t* row_of, int32_t* block_counts, hipStream_t s);

// Per-path execution (baselines): path rows keyed by the target (key_is_target = 1) or the
// source slot of each path, expanded in place from the top-k dispatch rows.
hipError_t launch_path_rows(const uint64_t* bits, const int32_t* expert_offsets,
                            const int32_t* row_token, const int32_t* row_slot,
                            const int32_t* row_of, int64_t R, int n, int k, int key_is_target,
                            const int32_t* gather_src, int32_t* c, int32_t* start,
                            int32_t* path_offsets, int32_t* path_token, int32_t* path_row_of,
                            int32_t* path_gather, hipStream_t s);
hipError_t launch_combine_paths(const float* o, const uint64_t* bits, const float* beta,
                                const int32_t* path_row_of, int64_t T, int k, int H, int64_t P,
                                float* y, int accumulate, hipStream_t s);

// Scored compositional routing.
hipError_t launch_path_layout(const uint8_t* mask, const float* bias, int n, int32_t* count,
                              uint32_t* pair, float* pair_bias, hipStream_t s);
hipError_t launch_route_scored(const float* g_base, const float* g_tgt, float lambda,
                               const int32_t* count, const uint32_t* pair, const float* pair_bias,
                               int64_t T, int n, int K, int32_t* sel_pair, float* sel_score,
                               int32_t* n_src, int32_t* src_expert, int32_t* n_tgt,
                               int32_t* tgt_expert, uint64_t* bits, float* beta, hipStream_t s);

}  // namespace pcm
