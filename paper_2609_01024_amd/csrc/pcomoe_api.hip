// C ABI of libpcomoe: host-side validation, workspace layout and launch sequencing.
// Every check runs before anything is enqueued; the library never allocates, frees or
// synchronises.
#include "pcomoe.h"

#include <mutex>

#include "internal.h"

using namespace pcm;

// Scratch of pcm_project_combine_noalloc: z, its row scales and o live here instead of in a
// caller workspace. Each GPU the library runs on holds its own copy until the process ends.
// Host code never uses the array's name as an address: the device address of this GPU's copy
// comes from hipGetSymbolAddress (scratch_on_current_device).
static __device__ __align__(256) unsigned char scratch[PCM_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch` per device (set once)

// The address of the current device's scratch array, looked up on the first call made with
// that device current.
pcm_status scratch_on_current_device(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return PCM_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return PCM_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return PCM_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return PCM_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

pcm_status check_shape(int64_t T, int n, int k) {
    if (T < 0 || n < 1 || k < 1 || k > n) return PCM_ERR_ARG;
    if (k > kMaxK || n > kMaxN) return PCM_ERR_UNSUPPORTED;
    if (T * (int64_t)k >= ((int64_t)1 << 31)) return PCM_ERR_UNSUPPORTED;
    return PCM_OK;
}

pcm_status check_dims(int H, int F) {
    if (H < 1 || F < 1) return PCM_ERR_ARG;
    if (H % 64 || F % 64) return PCM_ERR_UNSUPPORTED;
    return PCM_OK;
}

pcm_status check_paths(const pcm_paths* p) {
    if (!p || !p->path_bits || !p->beta || !p->expert_offsets || !p->row_token || !p->row_slot ||
        !p->row_of)
        return PCM_ERR_ARG;
    return PCM_OK;
}

pcm_status from_hip(hipError_t e) { return e == hipSuccess ? PCM_OK : PCM_ERR_HIP; }

pcm_status check_scored(const pcm_scored_paths* p) {
    if (!p || !p->sel_pair || !p->sel_score || !p->n_src || !p->src_expert || !p->n_tgt ||
        !p->tgt_expert || !p->path_bits || !p->beta || !p->src_offsets || !p->src_row_token ||
        !p->src_row_slot || !p->src_row_of || !p->tgt_offsets || !p->tgt_row_token ||
        !p->tgt_row_slot || !p->tgt_row_of)
        return PCM_ERR_ARG;
    return PCM_OK;
}

pcm_status check_layout(const pcm_path_layout* l) {
    if (!l || !l->count || !l->pair || !l->bias) return PCM_ERR_ARG;
    return PCM_OK;
}

// The kernel choices of a pcm_tuning (NULL: every default) for the expansion or the
// projection side; PCM_ERR_ARG for a value outside the documented set.
pcm_status to_tune(const pcm_tuning* t, bool expansion, GemmTune* out) {
    *out = GemmTune();
    if (!t) return PCM_OK;
    if (t->tile != 0 && t->tile != 'S' && t->tile != 'M' && t->tile != 'L' && t->tile != 'W')
        return PCM_ERR_ARG;
    if (t->order_expand < -1 || t->order_expand > 2 || t->order_down < -1 || t->order_down > 2)
        return PCM_ERR_ARG;
    if (t->em_window < 0 || t->group_n < 0) return PCM_ERR_ARG;
    const int d = t->stream_depth;
    if (d != -1 && d != 0 && d != 2 && d != 3 && d != 4 && d != 6) return PCM_ERR_ARG;
    out->tile = (char)t->tile;
    out->order = expansion ? t->order_expand : t->order_down;
    out->window = t->em_window;
    out->group_n = t->group_n;
    out->stream_depth = d;
    return PCM_OK;
}

// Records stage event i of a tuning (if any) on the stream.
hipError_t stage_event(const pcm_tuning* t, int i, hipStream_t s) {
    if (!t || !t->stage_events[i]) return hipSuccess;
    return hipEventRecord((hipEvent_t)t->stage_events[i], s);
}

// Layer dtypes: PCM_BF16_F16DOWN is a bf16 layer whose projection weights are float16.
bool dtype_ok(pcm_dtype d) { return d == PCM_F32 || d == PCM_BF16 || d == PCM_BF16_F16DOWN; }
bool is_bf16(pcm_dtype d) { return d == PCM_BF16 || d == PCM_BF16_F16DOWN; }

// Workspace of the projection of R rows of n groups: z [R,F] (f16 for bf16 layers, f32
// otherwise), the per-row inverse scales [R] f32 (bf16 layers), then, when `with_o`, the
// projected rows o [ksplit, R, H] f32 (K slices of the projection); parts 256-byte aligned.
struct ProjWs {
    size_t zscale_off, o_off, total;
    int ksplit;
};
ProjWs proj_ws(size_t R, int n, int H, int F, pcm_dtype dt, bool with_o, char tile = 0) {
    ProjWs w;
    w.ksplit = (with_o && is_bf16(dt)) ? down_ksplit((int64_t)R, n, H, F, tile) : 1;
    const size_t z = align_up(R * F * (is_bf16(dt) ? 2 : 4), 256);
    w.zscale_off = z;
    w.o_off = z + (is_bf16(dt) ? align_up(R * sizeof(float), 256) : 0);
    w.total = w.o_off + (with_o ? align_up((size_t)w.ksplit * R * H * sizeof(float), 256) : 0);
    return w;
}

// Workspace of the per-path execution (baseline), P = T*k*k rows at most:
//   c, start [R] i32; path offsets [n+1] x2; path_token [P] x2; path_row_of [T*k*k] x2;
//   path_gather [P]; U [P or R, F] f32; z [P or R, F] (f16 + scales [P] for bf16); o [P, H] f32.
struct PathWs {
    size_t c, start, off_t, off_s, tok_t, tok_s, rof_t, rof_s, gather, u, z, zscale, o, total;
};
PathWs path_ws(int64_t T, int H, int F, int n, int k, pcm_dtype dt) {
    PathWs w{};
    const size_t R = (size_t)T * k, P = (size_t)T * k * k;
    size_t at = 0;
    auto take = [&](size_t bytes) { const size_t o = at; at += align_up(bytes, 256); return o; };
    w.c = take(R * 4);
    w.start = take(R * 4);
    w.off_t = take((size_t)(n + 1) * 4);
    w.off_s = take((size_t)(n + 1) * 4);
    w.tok_t = take(P * 4);
    w.tok_s = take(P * 4);
    w.rof_t = take(P * 4);
    w.rof_s = take(P * 4);
    w.gather = take(P * 4);
    w.u = take(P * F * 4);
    w.z = take(P * F * (is_bf16(dt) ? 2 : 4));
    w.zscale = take(is_bf16(dt) ? P * 4 : 0);
    w.o = take(P * H * 4);
    w.total = at;
    return w;
}

}  // namespace

extern "C" {

int pcm_abi_version(void) { return 123; }

const char* pcm_status_string(pcm_status s) {
    switch (s) {
        case PCM_OK: return "PCM_OK: success";
        case PCM_ERR_ARG: return "PCM_ERR_ARG: invalid argument (null or misaligned pointer, bad size, k > n)";
        case PCM_ERR_UNSUPPORTED: return "PCM_ERR_UNSUPPORTED: outside the supported limits (k <= 8, n <= 256, H and F multiples of 64, T*k < 2^31)";
        case PCM_ERR_WORKSPACE: return "PCM_ERR_WORKSPACE: workspace smaller than pcm_workspace_bytes()";
        case PCM_ERR_HIP: return "PCM_ERR_HIP: a HIP launch failed";
    }
    return "unknown pcm_status";
}

size_t pcm_workspace_bytes(pcm_op op, int64_t T, int H, int F, int n, int k, pcm_dtype dtype) {
    if (T < 0 || n < 1 || k < 1) return 0;
    switch (op) {
        case PCM_OP_BUILD_PATHS: return build_paths_ws_bytes(T, n);
        case PCM_OP_ROUTE_PATHS: return route_paths_ws_bytes(T, n);
        case PCM_OP_EXPAND: return 0;
        case PCM_OP_PROJECT_COMBINE:
            if (H < 1 || F < 1) return 0;
            return proj_ws((size_t)T * k, n, H, F, dtype, true).total;
        case PCM_OP_ROUTE_LOGITS:
            if (H < 1 || H % 64) return 0;
            return is_bf16(dtype) ? router_ws_bytes(T, H, n) : 0;
        case PCM_OP_LAYER_PER_PATH:
            if (H < 1 || F < 1) return 0;
            return path_ws(T, H, F, n, k, dtype).total;
        case PCM_OP_ROUTE_SCORED:  // block counts of the source and the target dispatch
            return 2 * build_paths_ws_bytes(T, n);
        case PCM_OP_DENSE_SWIGLU:  // the SwiGLU output u [T,F] f32, then a projection input
            if (H < 1 || F < 1) return 0;
            return align_up((size_t)T * F * sizeof(float), 256) +
                   (is_bf16(dtype) ? proj_ws((size_t)T, 1, H, F, dtype, false).total : 0);
    }
    return 0;
}

pcm_status pcm_route(const float* logits, int64_t T, int n, int k, int32_t* topk_ids,
                     float* topk_w, void* stream) {
    pcm_status st = check_shape(T, n, k);
    if (st != PCM_OK) return st;
    if (T == 0) return PCM_OK;
    if (!logits || !topk_ids || !topk_w) return PCM_ERR_ARG;
    if (!aligned16(logits) || !aligned16(topk_ids) || !aligned16(topk_w)) return PCM_ERR_ARG;
    return from_hip(launch_route(logits, T, n, k, topk_ids, topk_w, (hipStream_t)stream));
}

pcm_status pcm_route_logits(pcm_dtype dtype, const void* x, const void* w_router, int64_t T,
                            int H, int n, int k, float* logits, int32_t* topk_ids, float* topk_w,
                            void* ws, size_t ws_bytes, void* stream) {
    pcm_status st = check_shape(T, n, k);
    if (st != PCM_OK) return st;
    if (H < 1) return PCM_ERR_ARG;
    if (H % 64) return PCM_ERR_UNSUPPORTED;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    if (T == 0) return PCM_OK;
    if (!x || !w_router || !topk_ids || !topk_w) return PCM_ERR_ARG;
    if (!aligned16(x) || !aligned16(w_router) || !aligned16(topk_ids) || !aligned16(topk_w) ||
        (logits && !aligned16(logits)))
        return PCM_ERR_ARG;
    const size_t need = is_bf16(dtype) ? router_ws_bytes(T, H, n) : 0;
    if (ws_bytes < need || (need && !ws)) return PCM_ERR_WORKSPACE;
    if (need && !aligned16(ws)) return PCM_ERR_ARG;
    return from_hip(launch_router(is_bf16(dtype), x, w_router, T, H, n, k, logits, topk_ids,
                                  topk_w, (float*)ws, (hipStream_t)stream));
}

pcm_status pcm_residual_add(pcm_dtype dtype, void* h, const float* y, int64_t T, int H,
                            void* stream) {
    if (T < 0 || H < 1) return PCM_ERR_ARG;
    if (H % 64) return PCM_ERR_UNSUPPORTED;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    if (T == 0) return PCM_OK;
    if (!h || !y || !aligned16(h) || !aligned16(y)) return PCM_ERR_ARG;
    return from_hip(launch_residual(h, y, T * (int64_t)H, is_bf16(dtype), (hipStream_t)stream));
}

pcm_status pcm_widen_f16(const void* w_bf16, int64_t count, void* w_f16, void* stream) {
    if (count < 0) return PCM_ERR_ARG;
    if (count == 0) return PCM_OK;
    if (!w_bf16 || !w_f16 || !aligned16(w_bf16) || !aligned16(w_f16)) return PCM_ERR_ARG;
    return from_hip(launch_widen_f16((const uint16_t*)w_bf16, count, (uint16_t*)w_f16,
                                     (hipStream_t)stream));
}

pcm_status pcm_build_paths(const int32_t* topk_ids, const float* topk_w, const uint8_t* mask,
                           int64_t T, int n, int k, pcm_beta_mode beta_mode, const pcm_paths* out,
                           void* ws, size_t ws_bytes, void* stream) {
    pcm_status st = check_shape(T, n, k);
    if (st != PCM_OK) return st;
    if (beta_mode < PCM_BETA_SRC_COND || beta_mode > PCM_BETA_GLOBAL) return PCM_ERR_ARG;
    if (T == 0) return PCM_OK;
    if (!topk_ids || !topk_w || !mask || check_paths(out) != PCM_OK) return PCM_ERR_ARG;
    if (!aligned16(topk_ids) || !aligned16(topk_w) || !aligned16(mask) ||
        !aligned16(out->path_bits) || !aligned16(out->beta) || !aligned16(out->expert_offsets) ||
        !aligned16(out->row_token) || !aligned16(out->row_slot) || !aligned16(out->row_of))
        return PCM_ERR_ARG;
    const size_t need = build_paths_ws_bytes(T, n);
    if (ws_bytes < need || (need && !ws)) return PCM_ERR_WORKSPACE;
    if (need && !aligned16(ws)) return PCM_ERR_ARG;
    return from_hip(launch_build_paths(topk_ids, topk_w, mask, T, n, k, (int)beta_mode,
                                       out->path_bits, out->beta, out->expert_offsets,
                                       out->row_token, out->row_slot, out->row_of, (int32_t*)ws,
                                       (hipStream_t)stream));
}

pcm_status pcm_mask_pack(const uint8_t* mask, int n, uint64_t* packed, void* stream) {
    if (n < 1) return PCM_ERR_ARG;
    if (n > kMaxN) return PCM_ERR_UNSUPPORTED;
    if (!mask || !packed || !aligned16(mask) || !aligned16(packed)) return PCM_ERR_ARG;
    return from_hip(launch_mask_pack(mask, n, packed, (hipStream_t)stream));
}

pcm_status pcm_route_paths(const float* logits, const uint64_t* packed_mask, int64_t T, int n,
                           int k, pcm_beta_mode beta_mode, int32_t* topk_ids, float* topk_w,
                           const pcm_paths* out, void* ws, size_t ws_bytes, void* stream) {
    pcm_status st = check_shape(T, n, k);
    if (st != PCM_OK) return st;
    if (beta_mode < PCM_BETA_SRC_COND || beta_mode > PCM_BETA_GLOBAL) return PCM_ERR_ARG;
    if (T == 0) return PCM_OK;
    if (!logits || !packed_mask || !topk_ids || !topk_w || check_paths(out) != PCM_OK)
        return PCM_ERR_ARG;
    if (!aligned16(logits) || !aligned16(packed_mask) || !aligned16(topk_ids) ||
        !aligned16(topk_w) || !aligned16(out->path_bits) || !aligned16(out->beta) ||
        !aligned16(out->expert_offsets) || !aligned16(out->row_token) ||
        !aligned16(out->row_slot) || !aligned16(out->row_of))
        return PCM_ERR_ARG;
    const size_t need = route_paths_ws_bytes(T, n);
    if (ws_bytes < need || !ws) return PCM_ERR_WORKSPACE;
    if (!aligned16(ws)) return PCM_ERR_ARG;
    return from_hip(launch_route_paths(logits, packed_mask, T, n, k, (int)beta_mode, topk_ids,
                                       topk_w, out->path_bits, out->beta, out->expert_offsets,
                                       out->row_token, out->row_slot, out->row_of, ws,
                                       (hipStream_t)stream));
}

pcm_status pcm_expand_tuned(pcm_dtype dtype, const void* x, const void* w_gate, const void* w_up,
                            const pcm_paths* paths, int64_t T, int H, int F, int n, int k, void* u,
                            void* ws, size_t ws_bytes, void* stream, const pcm_tuning* tuning) {
    (void)ws;
    (void)ws_bytes;
    pcm_status st = check_shape(T, n, k);
    if (st != PCM_OK) return st;
    if ((st = check_dims(H, F)) != PCM_OK) return st;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    GemmTune tune;
    if ((st = to_tune(tuning, true, &tune)) != PCM_OK) return st;
    if (T == 0) return PCM_OK;
    if (!x || !w_gate || !w_up || !u || check_paths(paths) != PCM_OK) return PCM_ERR_ARG;
    if (!aligned16(x) || !aligned16(w_gate) || !aligned16(w_up) || !aligned16(u)) return PCM_ERR_ARG;
    GemmArgs g{};
    g.a = x;
    g.b0 = w_gate;
    g.b1 = w_up;
    g.out = u;
    g.offsets = paths->expert_offsets;
    g.gather = paths->row_token;
    g.a_rows = T;
    g.n = n;
    g.K = H;
    g.N = F;
    const int64_t R = T * k;
    hipStream_t s = (hipStream_t)stream;
    return from_hip(is_bf16(dtype) ? launch_gemm_bf16(kExpand, g, R, s, tune)
                                      : launch_gemm_f32(kExpand, g, R, s));
}

pcm_status pcm_expand(pcm_dtype dtype, const void* x, const void* w_gate, const void* w_up,
                      const pcm_paths* paths, int64_t T, int H, int F, int n, int k, void* u,
                      void* ws, size_t ws_bytes, void* stream) {
    return pcm_expand_tuned(dtype, x, w_gate, w_up, paths, T, H, F, n, k, u, ws, ws_bytes, stream,
                            nullptr);
}

pcm_status pcm_project_combine_tuned(pcm_dtype dtype, const void* u, const void* w_down,
                                     const pcm_paths* paths, int64_t T, int H, int F, int n, int k,
                                     float* y, int accumulate, void* ws, size_t ws_bytes,
                                     void* stream, const pcm_tuning* tuning) {
    pcm_status st = check_shape(T, n, k);
    if (st != PCM_OK) return st;
    if ((st = check_dims(H, F)) != PCM_OK) return st;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    GemmTune tune;
    if ((st = to_tune(tuning, false, &tune)) != PCM_OK) return st;
    if (T == 0) return PCM_OK;
    if (!u || !w_down || !y || check_paths(paths) != PCM_OK) return PCM_ERR_ARG;
    if (!aligned16(u) || !aligned16(w_down) || !aligned16(y)) return PCM_ERR_ARG;
    const int64_t R = T * k;
    const ProjWs w = proj_ws((size_t)R, n, H, F, dtype, true, tune.tile);
    if (!ws || ws_bytes < w.total) return PCM_ERR_WORKSPACE;
    if (!aligned16(ws)) return PCM_ERR_ARG;
    void* z = ws;
    const bool bf16 = is_bf16(dtype);
    float* zscale = bf16 ? (float*)((char*)ws + w.zscale_off) : nullptr;
    float* o = (float*)((char*)ws + w.o_off);
    hipStream_t s = (hipStream_t)stream;
    MixMap m{};
    m.bits = paths->path_bits;
    m.beta = paths->beta;
    m.src_row = m.tgt_row = paths->row_of;
    m.K = k;
    m.R_src = m.R_tgt = R;
    hipError_t e = stage_event(tuning, 0, s);
    if (e == hipSuccess) e = launch_mix((const float*)u, z, zscale, m, T, F, s);
    if (e == hipSuccess) e = stage_event(tuning, 1, s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    GemmArgs g{};
    g.a = z;
    g.b0 = w_down;
    g.b_f16 = dtype == PCM_BF16_F16DOWN;
    g.out = o;
    g.row_scale = zscale;
    g.offsets = paths->expert_offsets;
    g.a_rows = R;
    g.n = n;
    g.K = F;
    g.N = H;
    g.ksplit = w.ksplit;
    g.rows_total = R;
    e = bf16 ? launch_gemm_bf16(kDownStore, g, R, s, tune) : launch_gemm_f32(kDownStore, g, R, s);
    if (e == hipSuccess) e = stage_event(tuning, 2, s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    e = launch_combine(o, w.ksplit, m, T, H, y, accumulate, s);
    if (e == hipSuccess) e = stage_event(tuning, 3, s);
    return from_hip(e);
}

pcm_status pcm_project_combine(pcm_dtype dtype, const void* u, const void* w_down,
                               const pcm_paths* paths, int64_t T, int H, int F, int n, int k,
                               float* y, int accumulate, void* ws, size_t ws_bytes, void* stream) {
    return pcm_project_combine_tuned(dtype, u, w_down, paths, T, H, F, n, k, y, accumulate, ws,
                                     ws_bytes, stream, nullptr);
}

pcm_status pcm_project_combine_noalloc(pcm_dtype dtype, const void* u, const void* w_down,
                                      const pcm_paths* paths, int64_t T, int H, int F, int n,
                                      int k, float* y, int accumulate, void* stream) {
    // the same checks, in the same order, as pcm_project_combine_tuned, before the scratch
    // size (so that bad arguments report PCM_ERR_ARG / UNSUPPORTED as there)
    pcm_status st = check_shape(T, n, k);
    if (st != PCM_OK) return st;
    if ((st = check_dims(H, F)) != PCM_OK) return st;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    if (T == 0) return PCM_OK;
    if (!u || !w_down || !y || check_paths(paths) != PCM_OK) return PCM_ERR_ARG;
    if (!aligned16(u) || !aligned16(w_down) || !aligned16(y)) return PCM_ERR_ARG;
    const size_t need = proj_ws((size_t)(T * k), n, H, F, dtype, true).total;
    if (need > (size_t)PCM_NOALLOC_SCRATCH_BYTES) return PCM_ERR_UNSUPPORTED;
    void* ws = nullptr;
    if ((st = scratch_on_current_device(&ws)) != PCM_OK) return st;
    // every byte of z, the scales and o that the combine reads is written earlier in the same
    // call (one z row per (token, target) by the mix, every o element by the projection), so
    // nothing is cleared
    return pcm_project_combine_tuned(dtype, u, w_down, paths, T, H, F, n, k, y, accumulate, ws,
                                     need, stream, nullptr);
}

pcm_status pcm_project_workspace_layout(pcm_dtype dtype, int64_t T, int H, int F, int n, int k,
                                        const pcm_tuning* tuning, size_t* z_off,
                                        size_t* zscale_off, size_t* o_off, int* ksplit) {
    pcm_status st = check_shape(T, n, k);
    if (st != PCM_OK) return st;
    if ((st = check_dims(H, F)) != PCM_OK) return st;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    GemmTune tune;
    if ((st = to_tune(tuning, false, &tune)) != PCM_OK) return st;
    if (!z_off || !zscale_off || !o_off || !ksplit) return PCM_ERR_ARG;
    const ProjWs w = proj_ws((size_t)(T * k), n, H, F, dtype, true, tune.tile);
    *z_off = 0;
    *zscale_off = is_bf16(dtype) ? w.zscale_off : 0;
    *o_off = w.o_off;
    *ksplit = w.ksplit;
    return PCM_OK;
}

pcm_status pcm_dense_swiglu_tuned(pcm_dtype dtype, const void* x, const void* w_gate,
                                  const void* w_up, const void* w_down, int64_t T, int H, int Fs,
                                  float* y, int accumulate, void* ws, size_t ws_bytes, void* stream,
                                  const pcm_tuning* tuning) {
    if (T < 0) return PCM_ERR_ARG;
    pcm_status st = check_dims(H, Fs);
    if (st != PCM_OK) return st;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    GemmTune tune_up, tune_down;
    if ((st = to_tune(tuning, true, &tune_up)) != PCM_OK) return st;
    if ((st = to_tune(tuning, false, &tune_down)) != PCM_OK) return st;
    if (T >= ((int64_t)1 << 31)) return PCM_ERR_UNSUPPORTED;
    if (T == 0) return PCM_OK;
    if (!x || !w_gate || !w_up || !w_down || !y) return PCM_ERR_ARG;
    if (!aligned16(x) || !aligned16(w_gate) || !aligned16(w_up) || !aligned16(w_down) || !aligned16(y))
        return PCM_ERR_ARG;
    const bool bf16 = is_bf16(dtype);
    const size_t u_bytes = align_up((size_t)T * Fs * sizeof(float), 256);
    const ProjWs w = proj_ws((size_t)T, 1, H, Fs, dtype, false);
    const size_t need = u_bytes + (bf16 ? w.total : 0);
    if (!ws || ws_bytes < need) return PCM_ERR_WORKSPACE;
    if (!aligned16(ws)) return PCM_ERR_ARG;
    hipStream_t s = (hipStream_t)stream;
    float* u = (float*)ws;
    GemmArgs g{};
    g.a = x;
    g.b0 = w_gate;
    g.b1 = w_up;
    g.out = u;
    g.offsets = nullptr;
    g.gather = nullptr;
    g.a_rows = T;
    g.n = 1;
    g.K = H;
    g.N = Fs;
    hipError_t e = bf16 ? launch_gemm_bf16(kExpand, g, T, s, tune_up) : launch_gemm_f32(kExpand, g, T, s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    void* z = u;
    float* zscale = nullptr;
    if (bf16) {  // row-scaled float16 projection input
        z = (char*)ws + u_bytes;
        zscale = (float*)((char*)z + w.zscale_off);
        MixMap id{};  // identity: z_t = u_t
        id.K = 1;
        id.R_src = id.R_tgt = T;
        e = launch_mix(u, z, zscale, id, T, Fs, s);
        if (e != hipSuccess) return PCM_ERR_HIP;
    }
    GemmArgs d{};
    d.a = z;
    d.row_scale = zscale;
    d.b0 = w_down;
    d.b_f16 = dtype == PCM_BF16_F16DOWN;
    d.out = y;
    d.offsets = nullptr;
    d.a_rows = T;
    d.n = 1;
    d.K = Fs;
    d.N = H;
    d.accumulate = accumulate;
    e = bf16 ? launch_gemm_bf16(kDownAccum, d, T, s, tune_down) : launch_gemm_f32(kDownAccum, d, T, s);
    return from_hip(e);
}

pcm_status pcm_dense_swiglu(pcm_dtype dtype, const void* x, const void* w_gate, const void* w_up,
                            const void* w_down, int64_t T, int H, int Fs, float* y, int accumulate,
                            void* ws, size_t ws_bytes, void* stream) {
    return pcm_dense_swiglu_tuned(dtype, x, w_gate, w_up, w_down, T, H, Fs, y, accumulate, ws,
                                  ws_bytes, stream, nullptr);
}

pcm_status pcm_layer_per_path(pcm_dtype dtype, const void* x, const void* w_gate,
                              const void* w_up, const void* w_down, const pcm_paths* paths,
                              int64_t T, int H, int F, int n, int k, int reuse, float* y,
                              int accumulate, void* ws, size_t ws_bytes, void* stream) {
    pcm_status st = check_shape(T, n, k);
    if (st != PCM_OK) return st;
    if ((st = check_dims(H, F)) != PCM_OK) return st;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    if (T * (int64_t)k * k >= ((int64_t)1 << 31)) return PCM_ERR_UNSUPPORTED;
    if (T == 0) return PCM_OK;
    if (!x || !w_gate || !w_up || !w_down || !y || check_paths(paths) != PCM_OK) return PCM_ERR_ARG;
    if (!aligned16(x) || !aligned16(w_gate) || !aligned16(w_up) || !aligned16(w_down) || !aligned16(y))
        return PCM_ERR_ARG;
    const PathWs w = path_ws(T, H, F, n, k, dtype);
    if (!ws || ws_bytes < w.total) return PCM_ERR_WORKSPACE;
    if (!aligned16(ws)) return PCM_ERR_ARG;
    char* b = (char*)ws;
    auto i32 = [&](size_t off) { return (int32_t*)(b + off); };
    const int64_t R = T * k, P = T * (int64_t)k * k;
    const bool bf16 = is_bf16(dtype);
    hipStream_t s = (hipStream_t)stream;
    float* u = (float*)(b + w.u);
    void* z = b + w.z;
    float* zscale = bf16 ? (float*)(b + w.zscale) : nullptr;
    float* o = (float*)(b + w.o);
    hipError_t e;
    GemmArgs g{};
    g.a = x;
    g.b0 = w_gate;
    g.b1 = w_up;
    g.out = u;
    g.a_rows = T;
    g.n = n;
    g.K = H;
    g.N = F;
    int64_t u_rows;
    const int32_t* gather_src = nullptr;
    if (reuse) {  // one expansion row per (token, source): the top-k dispatch itself
        g.offsets = paths->expert_offsets;
        g.gather = paths->row_token;
        u_rows = R;
    } else {      // one expansion row per path, keyed by its source
        e = launch_path_rows(paths->path_bits, paths->expert_offsets, paths->row_token,
                             paths->row_slot, paths->row_of, R, n, k, 0, nullptr, i32(w.c),
                             i32(w.start), i32(w.off_s), i32(w.tok_s), i32(w.rof_s), nullptr, s);
        if (e != hipSuccess) return PCM_ERR_HIP;
        g.offsets = i32(w.off_s);
        g.gather = i32(w.tok_s);
        u_rows = P;
        gather_src = i32(w.rof_s);
    }
    e = bf16 ? launch_gemm_bf16(kExpand, g, u_rows, s, GemmTune()) : launch_gemm_f32(kExpand, g, u_rows, s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    if (bf16) {  // U rows as row-scaled float16, no mixing
        MixMap id{};
        id.K = 1;
        id.R_src = id.R_tgt = u_rows;
        id.live = reuse ? nullptr : i32(w.off_s) + n;
        e = launch_mix(u, z, zscale, id, u_rows, F, s);
        if (e != hipSuccess) return PCM_ERR_HIP;
    } else {
        z = u;
    }
    // one projection row per path, keyed by its target, gathering its source's z row
    e = launch_path_rows(paths->path_bits, paths->expert_offsets, paths->row_token,
                         paths->row_slot, paths->row_of, R, n, k, 1, gather_src, i32(w.c),
                         i32(w.start), i32(w.off_t), i32(w.tok_t), i32(w.rof_t), i32(w.gather), s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    GemmArgs d{};
    d.a = z;
    d.b0 = w_down;
    d.b_f16 = dtype == PCM_BF16_F16DOWN;
    d.out = o;
    d.row_scale = zscale;
    d.offsets = i32(w.off_t);
    d.gather = i32(w.gather);
    d.a_rows = u_rows;
    d.n = n;
    d.K = F;
    d.N = H;
    d.ksplit = 1;
    d.rows_total = P;
    e = bf16 ? launch_gemm_bf16(kDownStore, d, P, s, GemmTune()) : launch_gemm_f32(kDownStore, d, P, s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    return from_hip(launch_combine_paths(o, paths->path_bits, paths->beta, i32(w.rof_t), T, k, H, P,
                                         y, accumulate, s));
}

pcm_status pcm_path_layout_build(const uint8_t* mask, const float* bias, int n,
                                 const pcm_path_layout* out, void* stream) {
    if (n < 1) return PCM_ERR_ARG;
    if (n > kMaxN) return PCM_ERR_UNSUPPORTED;
    if (!mask || !bias || check_layout(out) != PCM_OK) return PCM_ERR_ARG;
    return from_hip(launch_path_layout(mask, bias, n, out->count, out->pair, out->bias,
                                       (hipStream_t)stream));
}

pcm_status pcm_route_scored(const float* g_base, const float* g_tgt, float lambda,
                            const pcm_path_layout* layout, int64_t T, int n, int K,
                            const pcm_scored_paths* out, void* ws, size_t ws_bytes, void* stream) {
    pcm_status st = check_shape(T, n, K);
    if (st != PCM_OK) return st;
    if (!(lambda == lambda) || lambda - lambda != 0.0f) return PCM_ERR_ARG;  // NaN or inf
    if (T == 0) return PCM_OK;
    if (!g_base || !g_tgt || check_layout(layout) != PCM_OK || check_scored(out) != PCM_OK)
        return PCM_ERR_ARG;
    const size_t one = build_paths_ws_bytes(T, n);
    if (ws_bytes < 2 * one || (one && !ws)) return PCM_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e = launch_route_scored(g_base, g_tgt, lambda, layout->count, layout->pair,
                                       layout->bias, T, n, K, out->sel_pair, out->sel_score,
                                       out->n_src, out->src_expert, out->n_tgt, out->tgt_expert,
                                       out->path_bits, out->beta, s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    int32_t* bc = (int32_t*)ws;
    e = launch_dispatch(out->src_expert, out->n_src, T, n, K, out->src_offsets, out->src_row_token,
                        out->src_row_slot, out->src_row_of, bc, s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    return from_hip(launch_dispatch(out->tgt_expert, out->n_tgt, T, n, K, out->tgt_offsets,
                                    out->tgt_row_token, out->tgt_row_slot, out->tgt_row_of,
                                    one ? (int32_t*)((char*)ws + one) : nullptr, s));
}

pcm_status pcm_expand_scored_tuned(pcm_dtype dtype, const void* x, const void* w_gate,
                                   const void* w_up, const pcm_scored_paths* paths, int64_t T,
                                   int H, int F, int n, int K, void* u, void* ws, size_t ws_bytes,
                                   void* stream, const pcm_tuning* tuning) {
    (void)ws;
    (void)ws_bytes;
    pcm_status st = check_shape(T, n, K);
    if (st != PCM_OK) return st;
    if ((st = check_dims(H, F)) != PCM_OK) return st;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    GemmTune tune;
    if ((st = to_tune(tuning, true, &tune)) != PCM_OK) return st;
    if (T == 0) return PCM_OK;
    if (!x || !w_gate || !w_up || !u || check_scored(paths) != PCM_OK) return PCM_ERR_ARG;
    if (!aligned16(x) || !aligned16(w_gate) || !aligned16(w_up) || !aligned16(u)) return PCM_ERR_ARG;
    GemmArgs g{};
    g.a = x;
    g.b0 = w_gate;
    g.b1 = w_up;
    g.out = u;
    g.offsets = paths->src_offsets;
    g.gather = paths->src_row_token;
    g.a_rows = T;
    g.n = n;
    g.K = H;
    g.N = F;
    const int64_t R = T * K;  // upper bound: the rows in use are src_offsets[n]
    hipStream_t s = (hipStream_t)stream;
    return from_hip(is_bf16(dtype) ? launch_gemm_bf16(kExpand, g, R, s, tune)
                                      : launch_gemm_f32(kExpand, g, R, s));
}

pcm_status pcm_expand_scored(pcm_dtype dtype, const void* x, const void* w_gate, const void* w_up,
                             const pcm_scored_paths* paths, int64_t T, int H, int F, int n, int K,
                             void* u, void* ws, size_t ws_bytes, void* stream) {
    return pcm_expand_scored_tuned(dtype, x, w_gate, w_up, paths, T, H, F, n, K, u, ws, ws_bytes,
                                   stream, nullptr);
}

pcm_status pcm_project_combine_scored_tuned(pcm_dtype dtype, const void* u, const void* w_down,
                                            const pcm_scored_paths* paths, int64_t T, int H, int F,
                                            int n, int K, float* y, int accumulate, void* ws,
                                            size_t ws_bytes, void* stream,
                                            const pcm_tuning* tuning) {
    pcm_status st = check_shape(T, n, K);
    if (st != PCM_OK) return st;
    if ((st = check_dims(H, F)) != PCM_OK) return st;
    if (!dtype_ok(dtype)) return PCM_ERR_ARG;
    GemmTune tune;
    if ((st = to_tune(tuning, false, &tune)) != PCM_OK) return st;
    if (T == 0) return PCM_OK;
    if (!u || !w_down || !y || check_scored(paths) != PCM_OK) return PCM_ERR_ARG;
    if (!aligned16(u) || !aligned16(w_down) || !aligned16(y)) return PCM_ERR_ARG;
    const int64_t R = T * K;  // row bound of U, z and o
    const ProjWs w = proj_ws((size_t)R, n, H, F, dtype, true, tune.tile);
    if (!ws || ws_bytes < w.total) return PCM_ERR_WORKSPACE;
    if (!aligned16(ws)) return PCM_ERR_ARG;
    void* z = ws;
    const bool bf16 = is_bf16(dtype);
    float* zscale = bf16 ? (float*)((char*)ws + w.zscale_off) : nullptr;
    float* o = (float*)((char*)ws + w.o_off);
    hipStream_t s = (hipStream_t)stream;
    MixMap m{};
    m.bits = paths->path_bits;
    m.beta = paths->beta;
    m.src_row = paths->src_row_of;
    m.tgt_row = paths->tgt_row_of;
    m.n_src = paths->n_src;
    m.n_tgt = paths->n_tgt;
    m.K = K;
    m.R_src = m.R_tgt = R;
    hipError_t e = stage_event(tuning, 0, s);
    if (e == hipSuccess) e = launch_mix((const float*)u, z, zscale, m, T, F, s);
    if (e == hipSuccess) e = stage_event(tuning, 1, s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    GemmArgs g{};
    g.a = z;
    g.b0 = w_down;
    g.b_f16 = dtype == PCM_BF16_F16DOWN;
    g.out = o;
    g.row_scale = zscale;
    g.offsets = paths->tgt_offsets;
    g.a_rows = R;
    g.n = n;
    g.K = F;
    g.N = H;
    g.ksplit = w.ksplit;
    g.rows_total = R;
    e = bf16 ? launch_gemm_bf16(kDownStore, g, R, s, tune) : launch_gemm_f32(kDownStore, g, R, s);
    if (e == hipSuccess) e = stage_event(tuning, 2, s);
    if (e != hipSuccess) return PCM_ERR_HIP;
    e = launch_combine(o, w.ksplit, m, T, H, y, accumulate, s);
    if (e == hipSuccess) e = stage_event(tuning, 3, s);
    return from_hip(e);
}

pcm_status pcm_project_combine_scored(pcm_dtype dtype, const void* u, const void* w_down,
                                      const pcm_scored_paths* paths, int64_t T, int H, int F, int n,
                                      int K, float* y, int accumulate, void* ws, size_t ws_bytes,
                                      void* stream) {
    return pcm_project_combine_scored_tuned(dtype, u, w_down, paths, T, H, F, n, K, y, accumulate,
                                            ws, ws_bytes, stream, nullptr);
}

}  // extern "C"
