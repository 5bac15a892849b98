/*
 * pcomoe.h -- C ABI of the path-compositional MoE layer (PCoMoE, arXiv 2609.01024)
 * on AMD Instinct MI355X (gfx950).
 *
 * One layer, per token h with router logits l (Section 2, vanilla MoE; Section 4):
 *   1. route          top-k experts e_0..e_{k-1} of l (logit descending, ties to the lower
 *                     id) and weights p_a = softmax over the k selected logits.
 *   2. build paths    Pi(h) = {(a, b) : m[e_a][e_b] = 1 or a == b} over the token's slots,
 *                     with the diagonal of the compatibility mask forced to 1 (Section 4.2,
 *                     m_ii = 1; Section 4.3, fallback to vanilla); path weights beta_ab;
 *                     the grouped dispatch layout (rows sorted by expert, then token).
 *   3. expand         U_(t,a) = SiLU(W_gate[e_a] x_t) * (W_up[e_a] x_t), once per
 *                     (token, source) pair (Section 4.1 U_e; Section 4.3 source-grouped reuse).
 *   4. project and    y_t = sum_{(a,b) in Pi} beta_ab W_down[e_b] U_(t,a)  (Section 4.1 path
 *      combine        aggregation, Section 4.3 source-grouped form), computed as
 *                     y_t = sum_b W_down[e_b] z_(t,b) with z_(t,b) = sum_a beta_ab U_(t,a),
 *                     which is the same sum because W_down is linear (Section 4.1 D_e).
 *
 * Conventions for every call:
 *   - Pointers named as device pointers must be device memory of the current HIP device,
 *     16-byte aligned; arrays are dense and row-major. The caller owns every buffer; the
 *     library never allocates or frees memory and holds no mutable global state (except
 *     pcm_project_combine_noalloc's per-GPU scratch array and its looked-up addresses).
 *   - `stream` is a hipStream_t (NULL = the default stream). Work is enqueued and the call
 *     returns without synchronising. Device-side faults surface at the caller's next sync.
 *   - Arguments are validated on the host before anything is enqueued. On error nothing
 *     is enqueued and outputs are untouched. T = 0 is a successful no-op.
 *   - Limits: 1 <= k <= min(n, 8); n <= 256; H and F multiples of 64; T*k < 2^31.
 *   - Logits must be finite. Index arrays passed back in (topk_ids, the pcm_paths layout)
 *     must be what the library produced; other values give undefined results, but every
 *     gathered index is clamped, so memory outside the buffers is never touched.
 */
#ifndef PCOMOE_H
#define PCOMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum pcm_status {
    PCM_OK = 0,
    PCM_ERR_ARG = 1,          /* null pointer, misaligned pointer, negative size, k > n ... */
    PCM_ERR_UNSUPPORTED = 2,  /* outside the limits above */
    PCM_ERR_WORKSPACE = 3,    /* ws_bytes smaller than pcm_workspace_bytes(...) */
    PCM_ERR_HIP = 4           /* a launch failed (hipGetLastError) */
} pcm_status;

typedef enum pcm_dtype {
    PCM_F32 = 0,   /* x and weights float32; FMA on the vector ALUs */
    PCM_BF16 = 1,  /* x and weights bfloat16; float32 accumulate throughout. The expansion
                      runs on bf16 MFMA and keeps u in float32; the projection input z is
                      carried as row-scaled float16 (11 significant bits) and the bf16
                      projection weights are widened to float16 in registers, so the
                      projection runs on f16 MFMA. Precondition on the projection weights
                      (w_down, and the shared expert's): |w| <= 65504, float16's largest value
                      (larger values become inf). Values with |w| >= 2^-17 widen exactly (a
                      bfloat16 there has at most 8 significant bits, all of which float16's
                      normal and upper subnormal range keep); smaller values round to the nearest
                      multiple of 2^-24 (float16's subnormal spacing; absolute error <= 2^-25),
                      so that magnitudes of 2^-25 or less become 0 */
    PCM_BF16_F16DOWN = 2  /* a PCM_BF16 layer whose projection weights (w_down, and the shared
                      expert's w_down) are passed as float16, widened once from the bf16
                      weights by pcm_widen_f16: the projection then uses them as read instead
                      of widening every fragment it loads, with bit-identical results. Every
                      other operand is as for PCM_BF16; calls that take no projection weights
                      treat this value as PCM_BF16. */
} pcm_dtype;

/* Path weights beta_ab for (a, b) in Pi (p = the renormalised router weights).
 * The paper names beta without a formula; the default is the reading under which a
 * diagonal-only mask reproduces the vanilla layer exactly (beta_aa = p_a, as Section 4.1
 * requires) and an all-pairs mask gives the product p_a p_b:
 *   SRC_COND: beta_ab = p_a p_b / sum_{b' : (a,b') in Pi} p_b'   (sum over Pi is 1)
 *   PRODUCT:  beta_ab = p_a p_b
 *   GLOBAL:   beta_ab = p_a p_b / sum_{(a',b') in Pi} p_a' p_b'                       */
typedef enum pcm_beta_mode {
    PCM_BETA_SRC_COND = 0,
    PCM_BETA_PRODUCT = 1,
    PCM_BETA_GLOBAL = 2
} pcm_beta_mode;

typedef enum pcm_op {
    PCM_OP_BUILD_PATHS = 0,
    PCM_OP_EXPAND = 1,
    PCM_OP_PROJECT_COMBINE = 2,
    PCM_OP_DENSE_SWIGLU = 3,
    PCM_OP_ROUTE_SCORED = 4,
    PCM_OP_LAYER_PER_PATH = 5,
    PCM_OP_ROUTE_LOGITS = 6,
    PCM_OP_ROUTE_PATHS = 7
} pcm_op;

/* Path table and grouped dispatch layout of T tokens (caller-owned device buffers).
 * A "row" is one (token, slot) pair; rows are ordered by (expert ascending, token
 * ascending), so the rows of expert e are [expert_offsets[e], expert_offsets[e+1]). */
typedef struct pcm_paths {
    uint64_t* path_bits;       /* [T]      bit a*k+b set iff (a, b) in Pi(token)            */
    float* beta;               /* [T,k,k]  beta[t][a][b]; exactly 0 where the bit is clear   */
    int32_t* expert_offsets;   /* [n+1]    first row of each expert; [n] = T*k              */
    int32_t* row_token;        /* [T*k]    token of each row                                 */
    int32_t* row_slot;         /* [T*k]    slot a of each row                                */
    int32_t* row_of;           /* [T*k]    row of pair (t, a) at index t*k + a               */
} pcm_paths;

/* Route (Section 2's top-k selection; Section 4.3's fused indexing starts here).
 * logits [T,n] f32 (device). Outputs (device): topk_ids [T,k] i32, experts of slots
 * 0..k-1 by logit descending with ties to the lower id (signed zeros are equal);
 * topk_w [T,k] f32, softmax over the k selected logits. */
pcm_status pcm_route(const float* logits, int64_t T, int n, int k, int32_t* topk_ids,
                     float* topk_w, void* stream);

/* The router's own GEMM fused with the routing above: logits[t, e] = x_t . W_r[e]
 * (the scores the router computes from the hidden state, Section 2), float32 accumulation
 * (bf16: products on the matrix cores), then pcm_route's top-k and softmax on those float32
 * values. x [T,H] and w_router [n,H] of `dtype` (device); logits [T,n] f32 is written when
 * not NULL; topk_ids / topk_w as pcm_route. H must be a multiple of 64. The bf16 path splits
 * K into slices whose partial sums are added in a fixed order (deterministic).
 * ws: pcm_workspace_bytes(PCM_OP_ROUTE_LOGITS, T, H, 0, n, k, dtype) bytes. */
pcm_status pcm_route_logits(pcm_dtype dtype, const void* x, const void* w_router, int64_t T,
                            int H, int n, int k, float* logits, int32_t* topk_ids, float* topk_w,
                            void* ws, size_t ws_bytes, void* stream);

/* Build the path table and dispatch layout (Section 4.2's mask with m_ii = 1, applied
 * before any weighting; Section 4.3's source-grouped dispatch metadata).
 * topk_ids/topk_w [T,k] from pcm_route; mask [n,n] u8 (device), row = expansion source
 * expert i, column = projection target expert j, nonzero = allowed; its diagonal is
 * ignored (treated as 1). Fills every array of *out (the struct itself is host memory).
 * Deterministic: integer outputs are bit-identical from run to run.
 * ws: device workspace of pcm_workspace_bytes(PCM_OP_BUILD_PATHS, T, 0, 0, n, k, 0). */
pcm_status pcm_build_paths(const int32_t* topk_ids, const float* topk_w, const uint8_t* mask,
                           int64_t T, int n, int k, pcm_beta_mode beta_mode,
                           const pcm_paths* out, void* ws, size_t ws_bytes, void* stream);

/* Offline per-layer layout of the compatibility mask for pcm_route_paths (Section 4.3's
 * indexing reads a mask fixed per layer, Section 4.2 with m_ii = 1). mask [n,n] u8 (device),
 * as pcm_build_paths; packed [n, ceil(n/64)] u64 (device, caller-owned): bit j % 64 of word
 * [i][j / 64] is set iff mask[i][j] != 0 or i == j; bits at j >= n are 0. One launch. */
pcm_status pcm_mask_pack(const uint8_t* mask, int n, uint64_t* packed, void* stream);

/* Section 4.3's fused indexing operation: pcm_route's top-k and softmax, pcm_build_paths's
 * path bits and beta, and the grouped dispatch layout, from the logits and a packed mask.
 * One launch when T <= 64 (one token per wavefront; the last workgroup to finish builds the
 * dispatch layout); otherwise a launch that routes, forms the path table and counts rows
 * per (32-token block, expert), then one that places the rows. Outputs are
 * bit-identical to pcm_route followed by pcm_build_paths with the mask that packed_mask
 * was packed from, and deterministic. logits [T,n] f32 (device); packed_mask from
 * pcm_mask_pack; topk_ids [T,k] i32 and topk_w [T,k] f32 (device) as pcm_route; *out as
 * pcm_build_paths (all of its arrays written). Limits and errors as pcm_build_paths.
 * ws: pcm_workspace_bytes(PCM_OP_ROUTE_PATHS, T, 0, 0, n, k, 0) bytes (device, 16-byte
 * aligned; 256 when T <= 64). Its first 256 bytes hold a completion counter of the
 * single-launch case: they must be zero before the first call that uses this workspace,
 * and every call leaves them zero (the rest needs no initialisation). Calls that overlap
 * in time must not share a workspace. */
pcm_status pcm_route_paths(const float* logits, const uint64_t* packed_mask, int64_t T, int n,
                           int k, pcm_beta_mode beta_mode, int32_t* topk_ids, float* topk_w,
                           const pcm_paths* out, void* ws, size_t ws_bytes, void* stream);

/* Expansion side, once per (token, source) row (Section 4.1 U_e; Section 4.3 reuse):
 * u[r,:] = SiLU(x[row_token[r]] W_gate[e]^T) * (x[row_token[r]] W_up[e]^T) for the rows r
 * of expert e. x [T,H] and w_gate/w_up [n,F,H] of `dtype`; u [T*k,F] float32 (device).
 * bf16: MFMA products accumulate in float32; SiLU and the product are float32 and u is
 * stored unrounded. ws: pcm_workspace_bytes(PCM_OP_EXPAND, ...) bytes (0; may be NULL). */
pcm_status pcm_expand(pcm_dtype dtype, const void* x, const void* w_gate, const void* w_up,
                      const pcm_paths* paths, int64_t T, int H, int F, int n, int k, void* u,
                      void* ws, size_t ws_bytes, void* stream);

/* Projection side and combine (Section 4.1 D_e and path aggregation; Section 4.3):
 * z_(t,b) = sum_{a : (a,b) in Pi} beta_ab u_(t,a)   (float32),
 * o_(t,b) = W_down[e_b] z_(t,b)                     (float32 accumulate),
 * y_t = [y_t if accumulate] + sum_{b ascending} o_(t,b).
 * For bf16 layers each z row is multiplied by a power of two that puts its largest
 * element just below 2^14 and stored as float16; the down GEMM multiplies its output row
 * by the inverse (exact), so any activation magnitude stays inside float16's range.
 * u [T*k,F] f32 from pcm_expand, w_down [n,H,F] of `dtype`, y [T,H] f32 (device).
 * ws: pcm_workspace_bytes(PCM_OP_PROJECT_COMBINE, ...) bytes (holds z and o). */
pcm_status pcm_project_combine(pcm_dtype dtype, const void* u, const void* w_down,
                               const pcm_paths* paths, int64_t T, int H, int F, int n, int k,
                               float* y, int accumulate, void* ws, size_t ws_bytes,
                               void* stream);

/* pcm_project_combine for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops such as a decode step, harnesses that forbid allocation): the
 * same computation, kernels and result, with z, its scales and o kept in a scratch array
 * inside the library instead of a caller workspace. It allocates nothing. The array holds
 * PCM_NOALLOC_SCRATCH_BYTES (16 MiB) per GPU, is reserved on every GPU the library runs on
 * until the process ends, and its address on a device is looked up on the first call made
 * with that device current. Sizes whose workspace
 * (pcm_workspace_bytes(PCM_OP_PROJECT_COMBINE, T, H, F, n, k, dtype)) exceeds the array give
 * PCM_ERR_UNSUPPORTED (a decode-shaped layer, T = 32, H = 7168, F = 2048, k = 8, needs
 * 8.0 MiB). All calls on one GPU share its array and each leaves its intermediates there:
 * calls that overlap on one GPU (other streams, other host threads) race and must be
 * serialised by the caller. Arguments as pcm_project_combine. */
#define PCM_NOALLOC_SCRATCH_BYTES (16u << 20)
pcm_status pcm_project_combine_noalloc(pcm_dtype dtype, const void* u, const void* w_down,
                                      const pcm_paths* paths, int64_t T, int H, int F, int n,
                                      int k, float* y, int accumulate, void* stream);

/* A dense SwiGLU FFN applied to every token with weight 1 (Section 2's expert F_e), for an
 * always-on shared expert that sits beside the routed experts and outside the path
 * space: y_t = [y_t if accumulate] + W_down (SiLU(W_gate x_t) * (W_up x_t)).
 * The SwiGLU output is kept in float32 and, for bf16 layers, enters the down projection
 * as row-scaled float16 like pcm_project_combine's z.
 * x [T,H], w_gate/w_up [Fs,H], w_down [H,Fs] of `dtype`; y [T,H] f32 (device).
 * ws: pcm_workspace_bytes(PCM_OP_DENSE_SWIGLU, T, H, Fs, 1, 1, dtype) bytes. */
pcm_status pcm_dense_swiglu(pcm_dtype dtype, const void* x, const void* w_gate,
                            const void* w_up, const void* w_down, int64_t T, int H, int Fs,
                            float* y, int accumulate, void* ws, size_t ws_bytes, void* stream);

/* Residual connection around the layer in a stack of layers (each MoE layer's output is
 * added to the hidden state it read): h = h + y elementwise, rounded to h's dtype (bf16:
 * round to nearest even). h [T,H] of `dtype`, y [T,H] f32 (device); H a multiple of 64. */
pcm_status pcm_residual_add(pcm_dtype dtype, void* h, const float* y, int64_t T, int H,
                            void* stream);

/* Offline weight layout for PCM_BF16_F16DOWN (projection weights are fixed per layer, like the
 * packed mask of pcm_mask_pack): w_f16[i] = w_bf16[i] rounded to float16, to nearest even,
 * exactly as the projection kernels widen each bf16 weight fragment for PCM_BF16 (so the
 * PCM_BF16 precondition on w_down applies). w_bf16 and w_f16 are device arrays of `count`
 * 16-bit values (count >= 0; 16-byte aligned; they must not overlap). One launch. */
pcm_status pcm_widen_f16(const void* w_bf16, int64_t count, void* w_f16, void* stream);

/* Per-path execution of the layer, a baseline for the target-mixed projection above: the
 * path-level aggregation of Section 4.1 evaluated one projection per path, as in Section
 * 4.3's source-grouped form, with no mixing of paths that share a target:
 *   reuse = 1: U_(t,a) once per (token, source) (Section 4.3's reuse);
 *   reuse = 0: U recomputed for every path (no reuse at all);
 *   o_(t,a,b) = W_down[e_b] U_(t,a) for every (a, b) in Pi,
 *   y_t = [y_t if accumulate] + sum_{(a,b) in Pi, a-major} beta_ab o_(t,a,b).
 * Same inputs, path table and result (to rounding) as pcm_expand + pcm_project_combine; bf16
 * layers project row-scaled float16 U rows. Sized for at most T*k*k paths.
 * ws: pcm_workspace_bytes(PCM_OP_LAYER_PER_PATH, T, H, F, n, k, dtype) bytes. */
pcm_status pcm_layer_per_path(pcm_dtype dtype, const void* x, const void* w_gate,
                              const void* w_up, const void* w_down, const pcm_paths* paths,
                              int64_t T, int H, int F, int n, int k, int reuse, float* y,
                              int accumulate, void* ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------- scored routing
 * The router the paper runs at inference (Section 4.2's compatibility-aware path score
 * and Section 4.3's TopK over the active path set):
 *   s_ij = g_base_i + b_ij + lambda g_tgt_j over A = {(i, j) : m_ij = 1}, m_ii = 1;
 *   Pi = the K best paths (ties to the lower i*n + j), beta = softmax of their scores;
 *   S = the distinct sources, each expanded once; T_i = the targets of source i;
 *   y = sum_{i in S} sum_{j in T_i} beta_ij D_j(U_i(h)).
 * The score is formed in float32 as fmaf(lambda, g_tgt_j, g_base_i + b_ij). K <= min(n, 8). */

/* Active pairs of one layer, materialised once (Section 4.3's offline path layout).
 * Caller-owned device buffers: count [1] i32; pair [n*n] u32 ((i << 16) | j of each active
 * pair in ascending i*n + j); bias [n*n] f32 (b_ij of each active pair). */
typedef struct pcm_path_layout {
    int32_t* count;
    uint32_t* pair;
    float* bias;
} pcm_path_layout;

/* Selected paths, groups and the two dispatch layouts of T tokens (caller-owned device
 * buffers). Source slots a < n_src[t] index the token's distinct sources and target slots
 * b < n_tgt[t] its distinct targets, both in ascending expert order. Expansion rows
 * (one per (token, source)) and projection rows (one per (token, target)) are each
 * ordered by (expert ascending, token ascending); at most T*K of each are used. */
typedef struct pcm_scored_paths {
    int32_t* sel_pair;         /* [T,K]    i*n + j of each selected path, selection order     */
    float* sel_score;          /* [T,K]    its score                                           */
    int32_t* n_src;            /* [T]      distinct sources                                    */
    int32_t* src_expert;       /* [T,K]    ascending; -1 from n_src on                         */
    int32_t* n_tgt;            /* [T]      distinct targets                                    */
    int32_t* tgt_expert;       /* [T,K]    ascending; -1 from n_tgt on                         */
    uint64_t* path_bits;       /* [T]      bit a*K+b: path src_expert[a] -> tgt_expert[b]      */
    float* beta;               /* [T,K,K]  weight of path (a, b); 0 where the bit is clear     */
    int32_t* src_offsets;      /* [n+1]    expansion rows of each expert                       */
    int32_t* src_row_token;    /* [T*K]    token of each expansion row                         */
    int32_t* src_row_slot;     /* [T*K]    source slot of each expansion row                   */
    int32_t* src_row_of;       /* [T*K]    expansion row of (t, a); -1 from n_src on           */
    int32_t* tgt_offsets;      /* [n+1]    projection rows of each expert                      */
    int32_t* tgt_row_token;    /* [T*K]                                                         */
    int32_t* tgt_row_slot;     /* [T*K]                                                         */
    int32_t* tgt_row_of;       /* [T*K]    projection row of (t, b); -1 from n_tgt on          */
} pcm_scored_paths;

/* Build the active-pair layout of a layer from mask [n,n] u8 (row = source i, column =
 * target j; the diagonal is treated as 1) and the compatibility bias [n,n] f32 (device). */
pcm_status pcm_path_layout_build(const uint8_t* mask, const float* bias, int n,
                                 const pcm_path_layout* out, void* stream);

/* Route T tokens over the layer's active pairs: selection, source / target groups,
 * weights and both dispatch layouts in one call (Section 4.3's fused indexing).
 * g_base, g_tgt [T,n] f32 (device); lambda finite. Deterministic.
 * ws: pcm_workspace_bytes(PCM_OP_ROUTE_SCORED, T, 0, 0, n, K, 0) bytes. */
pcm_status pcm_route_scored(const float* g_base, const float* g_tgt, float lambda,
                            const pcm_path_layout* layout, int64_t T, int n, int K,
                            const pcm_scored_paths* out, void* ws, size_t ws_bytes, void* stream);

/* pcm_expand over the expansion rows of scored routing: one row per (token, distinct
 * source). u [T*K,F] f32; rows from src_offsets[n] on are not written. */
pcm_status pcm_expand_scored(pcm_dtype dtype, const void* x, const void* w_gate,
                             const void* w_up, const pcm_scored_paths* paths, int64_t T, int H,
                             int F, int n, int K, void* u, void* ws, size_t ws_bytes,
                             void* stream);

/* pcm_project_combine for scored routing: z_(t,b) = sum_{a : (a,b) in Pi} beta_ab u_(t,a)
 * over the token's source and target slots, o_(t,b) = W_down[tgt_expert[b]] z_(t,b),
 * y_t = [y_t] + sum_{b ascending} o_(t,b); the same float16 projection input as
 * pcm_project_combine. ws: pcm_workspace_bytes(PCM_OP_PROJECT_COMBINE, T, H, F, n, K,
 * dtype) bytes. */
pcm_status pcm_project_combine_scored(pcm_dtype dtype, const void* u, const void* w_down,
                                      const pcm_scored_paths* paths, int64_t T, int H, int F,
                                      int n, int K, float* y, int accumulate, void* ws,
                                      size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------- tests and measurement
 * A layer never needs these. The *_tuned calls are the calls above with a pcm_tuning that
 * forces kernel choices the library otherwise makes by shape (every choice computes the same
 * bits) and that records HIP events between the internal stages of a call; tuning = NULL is
 * the plain call. They let tests check each kernel on the same inputs and let benchmarks time
 * each stage on the stream it runs on. Values outside the documented sets give PCM_ERR_ARG. */
typedef struct pcm_tuning {
    int tile;              /* 0: chosen by the mean rows per expert; 'S' the few-row streaming
                              kernel, 'M' the medium tiles, 'L' the large tiles on four waves,
                              'W' the large tiles on eight waves (two per SIMD; the default
                              for an expansion that takes the large tiles); for 'L' and 'W'
                              the medium tiles run instead where 32-bit buffer offsets would
                              not reach */
    int order_expand;      /* work order of the large tiles in expansion GEMMs: -1 by shape,
                              0 grouped, 1 longest first, 2 expert-major */
    int order_down;        /* the same for projection GEMMs */
    int em_window;         /* workgroups per expert-major window (0: 8) */
    int group_n;           /* N tiles per group of the grouped order (0: 4) */
    int stream_depth;      /* streaming kernel: -1 by GEMM side; 0 the register-ring kernel;
                              2, 3, 4 or 6 LDS ring slots */
    void* stage_events[4]; /* hipEvent_t each, or NULL: the project-and-combine calls record
                              them on `stream` before the mix, before the projection GEMM,
                              before the combine and after it (the caller creates them) */
} pcm_tuning;

pcm_status pcm_expand_tuned(pcm_dtype dtype, const void* x, const void* w_gate, const void* w_up,
                            const pcm_paths* paths, int64_t T, int H, int F, int n, int k, void* u,
                            void* ws, size_t ws_bytes, void* stream, const pcm_tuning* tuning);
pcm_status pcm_project_combine_tuned(pcm_dtype dtype, const void* u, const void* w_down,
                                     const pcm_paths* paths, int64_t T, int H, int F, int n, int k,
                                     float* y, int accumulate, void* ws, size_t ws_bytes,
                                     void* stream, const pcm_tuning* tuning);
pcm_status pcm_dense_swiglu_tuned(pcm_dtype dtype, const void* x, const void* w_gate,
                                  const void* w_up, const void* w_down, int64_t T, int H, int Fs,
                                  float* y, int accumulate, void* ws, size_t ws_bytes, void* stream,
                                  const pcm_tuning* tuning);
pcm_status pcm_expand_scored_tuned(pcm_dtype dtype, const void* x, const void* w_gate,
                                   const void* w_up, const pcm_scored_paths* paths, int64_t T,
                                   int H, int F, int n, int K, void* u, void* ws, size_t ws_bytes,
                                   void* stream, const pcm_tuning* tuning);
pcm_status pcm_project_combine_scored_tuned(pcm_dtype dtype, const void* u, const void* w_down,
                                            const pcm_scored_paths* paths, int64_t T, int H, int F,
                                            int n, int K, float* y, int accumulate, void* ws,
                                            size_t ws_bytes, void* stream,
                                            const pcm_tuning* tuning);

/* Where pcm_project_combine(_tuned) keeps its intermediates inside its workspace, so that a
 * test can read them back after the call: the projection input z [T*k, F] (bf16 layers:
 * float16 rows, each multiplied by a power of two; f32 layers: float32) at byte *z_off; the
 * inverse of each z row's power of two [T*k] f32 at *zscale_off (bf16 layers; 0 otherwise);
 * the projected rows o [ksplit, T*k, H] f32 at *o_off, K slice s of row r at (s*T*k + r)*H
 * (the combine adds the slices in order). All outputs are host pointers. */
pcm_status pcm_project_workspace_layout(pcm_dtype dtype, int64_t T, int H, int F, int n, int k,
                                        const pcm_tuning* tuning, size_t* z_off,
                                        size_t* zscale_off, size_t* o_off, int* ksplit);

/* Device workspace bytes an operation needs (0 if none). Returns 0 for invalid sizes. */
size_t pcm_workspace_bytes(pcm_op op, int64_t T, int H, int F, int n, int k, pcm_dtype dtype);

/* Static description of a status code (never NULL). */
const char* pcm_status_string(pcm_status status);

/* ABI version of this header (major * 100 + minor). */
int pcm_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* PCOMOE_H */
