// Grouped bf16 GEMMs on the gfx950 matrix cores (v_mfma_f32_16x16x32_bf16, float32
// accumulate) for the two sides of a SwiGLU expert (Section 4.1):
//   expand:  U[r, f] = SiLU(x[tok(r)] . W_gate[e][f]) * (x[tok(r)] . W_up[e][f])
//            one row per (token, source) pair, rows of expert e contiguous (Section 4.3),
//            x rows gathered through row_token; SwiGLU fused into the epilogue; U kept in
//            float32. bf16 x bf16 MFMA (v_mfma_f32_16x16x32_bf16).
//   down:    O[r, h] = row_scale[r'] * (Z[r'] . W_down[e][h]), r' = gather[r] or r
//                                                  (store, or accumulate into y
//                                                  for a dense FFN whose rows are tokens)
//            Z arrives as row-scaled float16; each bf16 W_down fragment is widened to
//            float16 in registers after its LDS read (exact in float16's normal range), and
//            the product runs on v_mfma_f32_16x16x32_f16 at the same rate.
// Both operands are K-contiguous (x rows and W rows run along H; Z rows and W_down rows
// along F), so a lane's 8 consecutive K values of a row are one 16-byte load.
//
// Three kernel shapes share the epilogue and the work decomposition:
//  * "interleaved" (large tiles, 256 x 256): four waves, one per SIMD, each owning a 128 x 128
//    block of C in 256 accumulation registers, or eight waves, two per SIMD, each owning a
//    128 x 64 block in 128 (the expansion's default: while one wave of a SIMD waits, the other
//    can issue MFMAs; same loads, same bits). Global -> LDS direct buffer loads
//    (buffer_load_dwordx4 ... lds, no register staging: one 32-bit offset per lane for the
//    whole tile, the stage's K offset in a scalar register) of 64-wide K stages, two stages
//    of A and three of B (the weights, mostly fetched from HBM, get two stages of latency
//    budget, the activations one), each load covering 8 whole 128-byte rows; one workgroup
//    barrier per 32-wide substep,
//    within which each wave issues its 64 MFMAs interleaved with the fragment reads of the
//    next substep (and, once per stage, the loads of A two stages and of B three stages
//    ahead). LDS rows are
//    128 bytes; the 16-byte chunk c of row r sits at position c ^ ((r >> 1) & 7), which
//    keeps the fragment reads (16 rows x 4 chunks per instruction) free of bank conflicts.
//    A group's last tile with at most 128 rows runs as a 128 x 256 tile (64 x 128 per wave)
//    in the same launch.
//  * "staged" (medium tiles): loads through registers into two LDS stages of 64-wide K
//    steps; rows of 128 bytes with chunk c of row r at position c ^ ((r >> 1) & 7). Runs
//    only where the large tiles' 32-bit buffer offsets would not reach.
//  * "stream" (fewer than 16 rows per group, decode): each wave streams its 32 weight rows
//    and its activation block through a ring of its own in LDS (no barrier), every direct
//    load covering whole 128-byte lines; the weights are the traffic. A register-ring
//    variant (fragments loaded straight into registers several k-steps ahead) runs where
//    the ring's 32-bit offsets would not reach.
// The MFMA takes the weight fragment as its first operand, so each lane's four
// accumulators are four consecutive output columns of one row (16-byte stores). For the
// expansion, a wave's weight rows are half gate and half up for the same columns, so the
// gate and up values of an output element sit in the same lane and register slot.
//
// Work decomposition: the grid is (upper bound of M tiles) x (N tiles) (x K slices). Each
// workgroup finds its group (expert) and row range from the group offsets with one wave-wide
// scan of per-group tile counts; workgroups past the last tile exit. Every order is
// XCD-aware (workgroup ids are dispatched round-robin over the 8 XCDs). Grouped rows of the
// large tiles walk an expert-major order (em_item: all row blocks of one expert for a few
// N tiles at a time, so a weight tile is fetched while every row block that needs it runs);
// a K-split projection lists each XCD's full-height tiles before its 128-row tail tiles
// (il_item); one group of rows (the dense shared expert) and the medium tiles use the
// grouped order of tile_of.
#include <type_traits>

#include "internal.h"

#define PCM_LDS __attribute__((address_space(3)))

namespace pcm {
namespace {

// s_waitcnt immediates (gfx9 encoding: vmcnt[3:0]+[15:14], expcnt[6:4], lgkmcnt[11:8])
constexpr int waitcnt_imm(int vm, int lgkm) {
    return (vm & 0xF) | (7 << 4) | ((lgkm & 0xF) << 8) | (((vm >> 4) & 3) << 14);
}
constexpr int kNoVm = 63, kNoLgkm = 15;

// Find this workgroup's group and row range. Returns false past the last tile.
template <int BM>
__device__ bool find_tile(const int32_t* __restrict__ offsets, int n, int64_t a_rows, int64_t mt,
                          int* s_tile) {
    if (offsets == nullptr) {  // one group: rows [0, a_rows)
        if (mt * BM >= a_rows) return false;
        s_tile[0] = 0;
        s_tile[1] = (int)(mt * BM);
        s_tile[2] = (int)min<int64_t>(a_rows, (mt + 1) * BM);
        return true;
    }
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        if (lane == 0) s_tile[0] = -1;
        int cnt[4], local = 0, lo[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int x = lane * 4 + j;
            int c = 0, b = 0;
            if (x < n) {
                b = offsets[x];
                c = (int)ceil_div(offsets[x + 1] - b, BM);
            }
            cnt[j] = c;
            lo[j] = b;
            local += c;
        }
        const int incl = wave_incl_scan_i32(local);
        int start = incl - local;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (mt >= start && mt < start + cnt[j]) {
                const int x = lane * 4 + j;
                const int r0 = lo[j] + (int)(mt - start) * BM;
                s_tile[0] = x;
                s_tile[1] = r0;
                s_tile[2] = min(offsets[x + 1], r0 + BM);
            }
            start += cnt[j];
        }
    }
    __syncthreads();
    return s_tile[0] >= 0;
}

// Tile of workgroup `bid` in a grid of `grid` (a multiple of 8) workgroups.
// Workgroups are dispatched round-robin over the 8 XCDs (bid % 8), so ids are first
// remapped to make each XCD's share a contiguous run. That run is walked in groups of GN
// N-tiles: inside a group the M-tile varies slowest, so the workgroups resident on one XCD
// at a time share a few weight tiles (same expert, neighbouring M-tiles) and a few
// activation tiles (same M-tile, neighbouring N-tiles) through that XCD's L2.
__device__ inline void tile_from_id(int64_t id, int64_t mt_count, int nt, int GN, int64_t* mt,
                                    int* ntile) {
    const int64_t gsize = (int64_t)GN * mt_count;
    const int64_t grp = id / gsize, in = id % gsize;
    const int64_t gn = min<int64_t>(GN, nt - grp * GN);
    *mt = in / gn;
    *ntile = (int)(grp * GN + in % gn);
}
__device__ inline bool tile_of(int64_t bid, int64_t grid, int64_t mt_upper, int nt, int GN,
                               int64_t* mt, int* ntile) {
    const int64_t id = (bid % 8) * (grid / 8) + bid / 8;
    if (id >= mt_upper * nt) return false;
    tile_from_id(id, mt_upper, nt, GN, mt, ntile);
    return true;
}

// Source row of A row r of the tile (rows past row1 repeat a valid row; their outputs are
// never stored).
__device__ inline int64_t a_source_row(const GemmArgs& g, int r, int row1) {
    if (r >= row1) r = row1 - 1;
    int64_t src = r;
    if (g.gather) {
        src = g.gather[r];
        src = src < 0 ? 0 : (src >= g.a_rows ? g.a_rows - 1 : src);
    }
    return src;
}

// Weight row (element offset of its K = 0) of B row j of the tile; rows past N repeat row
// N - 1 (their outputs are never stored).
template <int MODE, int WTN, int OUT_COLS>
__device__ inline const uint16_t* b_source_row(const GemmArgs& g, int e, int ntile, int j) {
    if (MODE == kExpand) {
        const int grp = j / WTN, jj = j % WTN, half = jj / (WTN / 2);
        int f = ntile * OUT_COLS + grp * (WTN / 2) + jj % (WTN / 2);
        f = f < g.N ? f : g.N - 1;
        return (const uint16_t*)(half ? g.b1 : g.b0) + ((int64_t)e * g.N + f) * g.K;
    }
    int h = ntile * OUT_COLS + j;
    h = h < g.N ? h : g.N - 1;
    return (const uint16_t*)g.b0 + ((int64_t)e * g.N + h) * g.K;
}

// Weight row (within its expert) of B row j of the tile, and whether it is an up row (the
// expansion's second half); rows past N repeat row N - 1 (their outputs are never stored).
// `up` is uniform over a load of 8 rows.
template <int MODE, int WTN, int OUT_COLS>
__device__ inline int b_source_col(const GemmArgs& g, int ntile, int j, bool* up) {
    if (MODE == kExpand) {
        const int grp = j / WTN, jj = j % WTN, half = jj / (WTN / 2);
        const int f = ntile * OUT_COLS + grp * (WTN / 2) + jj % (WTN / 2);
        *up = half != 0;
        return f < g.N ? f : g.N - 1;
    }
    const int h = ntile * OUT_COLS + j;
    *up = false;
    return h < g.N ? h : g.N - 1;
}

// Raw buffer resource over `bytes` bytes at `base` (loads past the end read zero).
__device__ inline __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Row of `a` (and of row_scale) behind output row r.
__device__ inline int64_t scale_row(const GemmArgs& g, int r) {
    if (!g.gather) return r;
    const int64_t s = g.gather[r];
    return s < 0 ? 0 : (s >= g.a_rows ? g.a_rows - 1 : s);
}

// SiLU(g) = g / (1 + e^-g) with the hardware reciprocal (about 1 ulp) instead of an IEEE
// division; for g below about -88, e^-g is +inf and the result is -0.
__device__ inline float silu(float g) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

// Shared epilogue: acc[nb][mb] holds C[row = .. + (lane & 15)][cols c0 .. c0+3].
template <int MODE, int MB, int NBK, int WTM, int WTN, int OUT_COLS>
__device__ inline void epilogue(const GemmArgs& g, const floatx4 (&acc)[NBK][MB], int row0,
                                int row1, int ntile, int wm, int wn, int lane) {
    const int N = g.N;
    // The row scales of all of this lane's rows are loaded first, without branches, and
    // waited for once, in code that every store follows. A scale load that is still in
    // flight where the stores' branches (row and column bounds) merge makes the compiler
    // wait for all outstanding memory operations before each store, the earlier stores
    // included: the 64 stores of a wave then ran one after another (13 us of a 256 x 256
    // projection tile).
    float scs[MB];
    if constexpr (MODE != kExpand) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const int r = min(row0 + wm * WTM + mb * 16 + (lane & 15), row1 - 1);
            scs[mb] = g.row_scale ? g.row_scale[scale_row(g, r)] : 1.0f;
        }
        __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, kNoLgkm));
    }
    if constexpr (MODE == kExpand) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const int r = row0 + wm * WTM + mb * 16 + (lane & 15);
            if (r >= row1) continue;
#pragma unroll
            for (int nb = 0; nb < NBK / 2; ++nb) {
                const int f = ntile * OUT_COLS + wn * (WTN / 2) + nb * 16 + (lane >> 4) * 4;
                if (f >= N) continue;
                const floatx4 gt = acc[nb][mb], up = acc[nb + NBK / 2][mb];
                float v[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = silu(gt[i]) * up[i];
                *(float4*)((float*)g.out + (int64_t)r * N + f) = make_float4(v[0], v[1], v[2], v[3]);
            }
        }
    } else if (base_mode(MODE) == kDownAccum && g.accumulate) {
        // read-modify-write: each row block's values are loaded before its stores
        float* O = (float*)g.out;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const int r = row0 + wm * WTM + mb * 16 + (lane & 15);
            if (r >= row1) continue;
            float4 prev[NBK];
#pragma unroll
            for (int nb = 0; nb < NBK; ++nb) {
                const int h = min(ntile * OUT_COLS + wn * WTN + nb * 16 + (lane >> 4) * 4, N - 4);
                prev[nb] = *(const float4*)(O + (int64_t)r * N + h);
            }
            const float sc = scs[mb];
#pragma unroll
            for (int nb = 0; nb < NBK; ++nb) {
                const int h = ntile * OUT_COLS + wn * WTN + nb * 16 + (lane >> 4) * 4;
                if (h >= N) continue;
                // the stored value plus the scaled product, each rounded (no fused multiply-add),
                // so that accumulating adds exactly what the store path writes
                *(float4*)(O + (int64_t)r * N + h) = make_float4(
                    __fadd_rn(prev[nb].x, __fmul_rn(acc[nb][mb][0], sc)), __fadd_rn(prev[nb].y, __fmul_rn(acc[nb][mb][1], sc)),
                    __fadd_rn(prev[nb].z, __fmul_rn(acc[nb][mb][2], sc)), __fadd_rn(prev[nb].w, __fmul_rn(acc[nb][mb][3], sc)));
            }
        }
    } else {
        float* O = (float*)g.out;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const int r = row0 + wm * WTM + mb * 16 + (lane & 15);
            if (r >= row1) continue;
            const float sc = scs[mb];
#pragma unroll
            for (int nb = 0; nb < NBK; ++nb) {
                const int h = ntile * OUT_COLS + wn * WTN + nb * 16 + (lane >> 4) * 4;
                if (h >= N) continue;
                *(float4*)(O + (int64_t)r * N + h) = make_float4(acc[nb][mb][0] * sc, acc[nb][mb][1] * sc,
                                                                 acc[nb][mb][2] * sc, acc[nb][mb][3] * sc);
            }
        }
    }
}

// bfloat16 -> float16, 8 lanes of a fragment (exact for |w| in float16's normal range)
__device__ inline halfx8 widen_to_f16(const bf16x8& v) {
    const uint4 q = __builtin_bit_cast(uint4, v);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
    halfx8 h;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        h[2 * i] = (_Float16)__uint_as_float(w[i] << 16);
        h[2 * i + 1] = (_Float16)__uint_as_float(w[i] & 0xFFFF0000u);
    }
    return h;
}

// Fragment types and loads of a mode: bf16 x bf16 for the expansion; for the projection
// the weight fragment is widened to float16 as it is read (outside the MFMA stream).
template <int MODE>
struct Frag {
    using T = typename std::conditional<MODE == kExpand, bf16x8, halfx8>::type;
    // a weight fragment as loaded (8 bf16 values, or 8 float16 values for half_weights)
    __device__ static T wide(const bf16x8& v) {
        if constexpr (MODE == kExpand) return v;
        else if constexpr (half_weights(MODE)) return __builtin_bit_cast(halfx8, v);
        else return widen_to_f16(v);
    }
    __device__ static T weights(const char* p) { return wide(*(const bf16x8*)p); }
    __device__ static T acts(const char* p) { return *(const T*)p; }
};
__device__ inline floatx4 mfma_step(const bf16x8& w, const bf16x8& a, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(w, a, c, 0, 0, 0);
}
__device__ inline floatx4 mfma_step(const halfx8& w, const halfx8& a, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(w, a, c, 0, 0, 0);
}

// ---------------------------------------------------------- interleaved kernel
// One wave per SIMD, each owning a 128 x 128 block of C (256 accumulator registers). K runs
// in 64-wide stages; LDS holds two stages of A and three of B (160 KB for 256 x 256 tiles,
// the whole of it: the kernel has no static LDS, and the work item is broadcast through the
// first bytes of the first A stage before its loads are issued). A stage is two 32-wide
// MFMA substeps, and every substep starts at a workgroup barrier. Between two barriers a
// wave issues the 64 MFMAs of one substep from registers, interleaved with the LDS fragment
// reads of the next substep (into the other register set); the first substep of stage kt
// also issues the global->LDS loads of A for stage kt + 2 and of B for stage kt + 3 (into
// the stage slots just freed). A third B stage (weights, mostly fetched from HBM) took the
// Mixtral-shaped expansion from 1583 to 1527 us and its projection from 1162 to 1089 us.
// A load covers 8 whole 128-byte rows, so each fetched cache line is used in full.
template <int BM_, int BNB_, int WM_, int WN_>
struct ICfg {
    static constexpr int BM = BM_, BNB = BNB_, WM = WM_, WN = WN_;
    static constexpr int NW = WM * WN, NT = NW * 64;
    static constexpr int WTM = BM / WM, WTN = BNB / WN, MB = WTM / 16, NBK = WTN / 16;
    static constexpr int A_ROWS = BM;
    static constexpr int A_INSTR = A_ROWS / 8, B_INSTR = BNB / 8;
    static constexpr int QA = A_INSTR / NW, QB = B_INSTR / NW, LPW = QA + QB;
    static constexpr int SA = A_ROWS * 128, SB = BNB * 128;   // one stage of A, of B
    static constexpr int LDS_BYTES = 2 * SA + 3 * SB;          // A: 2 stages, B: 3 stages
    // schedule of a substep: MFMA i is followed by fragment read i / R_EVERY (weights
    // first), load i / L_EVERY and, from slot W_FROM on, WPS dwords of weight widening
    static constexpr int NM = NBK * MB, NR = NBK + MB;
    static constexpr int R_EVERY = 3 * (NR - 1) < NM ? 3 : (2 * (NR - 1) < NM ? 2 : 1);
    static constexpr int L_EVERY = NM / LPW;
    static constexpr int W_FROM = R_EVERY * NBK + 2;
    static constexpr int WPS = (4 * NBK + (NM - W_FROM) - 1) / (NM - W_FROM);
    static_assert(A_INSTR % NW == 0 && B_INSTR % NW == 0, "every wave issues the same loads");
    static_assert(WTM % 16 == 0 && WTN % 32 == 0, "whole MFMA blocks, gate/up halves");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS budget (the kernel has no static LDS)");
    static_assert(LPW <= 63, "vmcnt range");
    static_assert(R_EVERY * (NR - 1) < NM && L_EVERY >= 1 && L_EVERY * (LPW - 1) + 1 < NM, "slots");
    static_assert(W_FROM < NM && (NM - W_FROM) * WPS >= 4 * NBK, "widen slots");
};

// 256 x 256 tiles; an expert's last tile with at most 128 rows runs as a 128 x 256 tile
// (each wave 64 x 128), which halves the MFMA work spent on padding rows.
using LargeIl = ICfg<256, 256, 2, 2>;
using LargeIlTail = ICfg<128, 256, 2, 2>;
// The same tiles on eight waves, two per SIMD (each 128 x 64, 128 accumulators): while one
// wave of a SIMD waits at a barrier or for its fragment reads, the other can issue MFMAs.
using WideIl = ICfg<256, 256, 2, 4>;
using WideIlTail = ICfg<128, 256, 2, 4>;

// MFMA through inline assembly with the accumulator pinned to AGPRs ("a" constraint):
// 256 accumulators per lane exceed what the compiler keeps in AGPRs across a loop without
// copies. FIRST starts from a zero accumulator (srcC = 0).
template <bool FIRST>
__device__ inline void mfma_agpr(floatx4& c, const bf16x8& w, const bf16x8& a) {
    if constexpr (FIRST)
        asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0" : "=a"(c) : "v"(w), "v"(a));
    else
        asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(w), "v"(a));
}
template <bool FIRST>
__device__ inline void mfma_agpr(floatx4& c, const halfx8& w, const halfx8& a) {
    if constexpr (FIRST)
        asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, 0" : "=a"(c) : "v"(w), "v"(a));
    else
        asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+a"(c) : "v"(w), "v"(a));
}

// One dword of a bf16 weight fragment (two values) widened to two float16 values, in
// inline assembly so that it keeps its place in the interleaved instruction stream.
__device__ inline uint32_t widen_pair_asm(uint32_t w) {
    uint32_t out, lo, hi;
    asm volatile(
        "v_lshlrev_b32 %1, 16, %3\n\t"
        "v_and_b32 %2, 0xffff0000, %3\n\t"
        "v_cvt_pk_f16_f32 %0, %1, %2"
        : "=v"(out), "=&v"(lo), "=&v"(hi)
        : "v"(w));
    return out;
}

// bf16 -> float16 of a weight array (count values) by the same instructions as the widening
// of each fragment in the projection kernels, so that projecting with the widened copy gives
// the bits the bf16 weights give: 8 values per thread and step, then the count % 8 last ones.
__global__ __launch_bounds__(256) void widen_kernel(const uint16_t* __restrict__ src, int64_t count,
                                                    uint16_t* __restrict__ dst) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t n8 = count / 8, first = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int64_t i = first; i < n8; i += stride) {
        const uint4 v = ((const uint4*)src)[i];
        uint4 o;
        o.x = widen_pair_asm(v.x);
        o.y = widen_pair_asm(v.y);
        o.z = widen_pair_asm(v.z);
        o.w = widen_pair_asm(v.w);
        ((uint4*)dst)[i] = o;
    }
    const int64_t i = n8 * 8 + first;
    if (i < count) dst[i] = (uint16_t)widen_pair_asm((uint32_t)src[i]);
}

// One tile of configuration C: rows [row0, row1) of group e, N tile ntile, K slice kslice.
template <class C, int MODE>
__device__ __forceinline__ void il_tile(const GemmArgs& g, char* lds, int e, int row0, int row1,
                                        int ntile, int kslice) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / C::WN, wn = wave % C::WN;
    const int K = g.K / g.ksplit;
    const int64_t k_byte0 = (int64_t)kslice * K * 2;
    constexpr int kOutCols = (MODE == kExpand) ? C::BNB / 2 : C::BNB;

    // load q of a lane: LDS row blk * 8 + lane / 8 of the A or B region, 16-byte position
    // lane % 8, holding chunk (lane % 8) ^ ((row >> 1) & 7) of that row. Loads are buffer
    // loads: a 32-bit byte offset per lane (fixed for the tile) and the stage's K offset as
    // the uniform scalar offset, against resources for `a` and for expert e's weights.
    uint32_t voff[C::LPW];
    int dst[C::LPW];
    const int lrow = lane >> 3;
    const int64_t wbytes = (int64_t)g.N * g.K * 2;   // one expert's weights
    const __amdgpu_buffer_rsrc_t ra = buffer_rsrc(g.a, (uint32_t)((int64_t)g.a_rows * g.K * 2));
    const __amdgpu_buffer_rsrc_t rb0 = buffer_rsrc((const char*)g.b0 + e * wbytes, (uint32_t)wbytes);
    const __amdgpu_buffer_rsrc_t rb1 =
        MODE == kExpand ? buffer_rsrc((const char*)g.b1 + e * wbytes, (uint32_t)wbytes) : rb0;
    bool up[C::LPW];
    // source rows of this lane's A loads: with a gather, every index is loaded before any is
    // used (one wait instead of one per load)
    int srows[C::QA];
#pragma unroll
    for (int q = 0; q < C::QA; ++q) srows[q] = min(row0 + (q * C::NW + wave) * 8 + lrow, row1 - 1);
    if (g.gather) {
#pragma unroll
        for (int q = 0; q < C::QA; ++q) srows[q] = g.gather[srows[q]];
#pragma unroll
        for (int q = 0; q < C::QA; ++q)
            srows[q] = srows[q] < 0 ? 0 : (srows[q] >= g.a_rows ? (int)(g.a_rows - 1) : srows[q]);
    }
#pragma unroll
    for (int q = 0; q < C::LPW; ++q) {
        up[q] = false;
        if (q < C::QA) {
            const int blk = q * C::NW + wave, lr = blk * 8 + lrow;
            const int chunk = (lane & 7) ^ ((lr >> 1) & 7);
            const int64_t srow = srows[q];
            voff[q] = (uint32_t)(srow * (int64_t)g.K * 2 + k_byte0 + chunk * 16);
            dst[q] = blk * 1024;
        } else {
            const int blk = (q - C::QA) * C::NW + wave, lb = blk * 8 + lrow;
            const int chunk = (lane & 7) ^ ((lb >> 1) & 7);
            const int f = b_source_col<MODE, C::WTN, kOutCols>(g, ntile, lb, &up[q]);
            voff[q] = (uint32_t)((int64_t)f * g.K * 2 + k_byte0 + chunk * 16);
            dst[q] = blk * 1024;
        }
    }
    // A stage i at lds + i * SA (i < 2), B stage i at lds + 2 * SA + i * SB (i < 3)
    auto load = [&](int q, int ksa, int ksb, char* abase, char* bbase) {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(q < C::QA ? ra : (up[q] ? rb1 : rb0),
                                                 (PCM_LDS void*)((q < C::QA ? abase : bbase) + dst[q]), 16, voff[q],
                                                 (q < C::QA ? ksa : ksb) * 128, 0, 0);
    };
    char* const A0 = lds;
    char* const B0 = lds + 2 * C::SA;

    floatx4 acc[C::NBK][C::MB];
    const int KT2 = K / 64;
    // fragment of row (lane & 15), chunk 4 * sub + (lane >> 4) of a 16-row block
    const int fr = lane & 15;
    const int foff0 = fr * 128 + (((lane >> 4) ^ (fr >> 1)) * 16);
    const int foff1 = fr * 128 + (((4 + (lane >> 4)) ^ (fr >> 1)) * 16);
    using FT = typename Frag<MODE>::T;
    FT af[2][C::MB], bf[2][C::NBK];
    bf16x8 braw[C::NBK];
    uint32_t bw[C::NBK][4];
    auto b_at = [&](const char* S, int nb, int fo) { return S + (wn * C::WTN + nb * 16) * 128 + fo; };
    auto a_at = [&](const char* S, int mb, int fo) { return S + (wm * C::WTM + mb * 16) * 128 + fo; };
    auto barrier = [&]() {
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
    };
    constexpr int NM = C::NM, NR = C::NR, R_EVERY = C::R_EVERY, L_EVERY = C::L_EVERY;
    constexpr int W_FROM = C::W_FROM, WPS = C::WPS;
    // One 32-wide substep: the MFMAs of (ca, cb), the fragment reads of the next substep
    // from the A and B stages SAr, SBr at chunk offset fo, and (LOADS, the first substep of a
    // stage) every load of A stage ksa into slot la and of B stage ksb into slot lb. It
    // starts with this wave's fragment reads complete and a barrier; a LOADS substep first
    // waits until only the newest B loads (the next B stage, issued after the A loads of the
    // stage its reads need) may be in flight, so that stage has landed, and the barrier
    // makes the slots it loads free (read by every wave).
    // The barrier also keeps VALU writes of fragment registers (the prologue's widening)
    // at least two wait states ahead of the MFMAs that read them: the MFMAs are inline
    // assembly, which the compiler's hazard checks do not see.
    auto sub = [&](auto first, auto loads, FT (&ca)[C::MB], FT (&cb)[C::NBK],
                   FT (&na)[C::MB], FT (&nb_)[C::NBK], const char* SAr, const char* SBr, int fo, int ksa, int ksb,
                   char* la, char* lb) {
        // a LOADS substep waits for the stage its reads need; only the B loads issued after
        // that stage's A loads (the next B stage) may stay in flight
        __builtin_amdgcn_s_waitcnt(waitcnt_imm(decltype(loads)::value ? C::QB : kNoVm, 0));
        barrier();
#pragma unroll
        for (int i = 0; i < NM; ++i) {
            mfma_agpr<decltype(first)::value>(acc[i / C::MB][i % C::MB], cb[i / C::MB], ca[i % C::MB]);
            if (i % R_EVERY == 0 && i / R_EVERY < NR) {
                const int j = i / R_EVERY;
                if (j < C::NBK) {
                    if constexpr (MODE == kExpand || half_weights(MODE)) nb_[j] = *(const FT*)b_at(SBr, j, fo);
                    else braw[j] = *(const bf16x8*)b_at(SBr, j, fo);
                } else {
                    na[j - C::NBK] = Frag<MODE>::acts(a_at(SAr, j - C::NBK, fo));
                }
            }
            if constexpr (decltype(loads)::value)
                if (i % L_EVERY == 1 && i / L_EVERY < C::LPW) load(i / L_EVERY, ksa, ksb, la, lb);
            if constexpr (MODE != kExpand && !half_weights(MODE)) {
#pragma unroll
                for (int w = 0; w < WPS; ++w) {
                    const int d = (i - W_FROM) * WPS + w;
                    if (i >= W_FROM && d < 4 * C::NBK) {
                        const uint4 q4 = __builtin_bit_cast(uint4, braw[d / 4]);
                        const uint32_t wv = (d % 4 == 0) ? q4.x : (d % 4 == 1) ? q4.y : (d % 4 == 2) ? q4.z : q4.w;
                        bw[d / 4][d % 4] = widen_pair_asm(wv);
                        if (d % 4 == 3)
                            nb_[d / 4] = __builtin_bit_cast(FT, uint4{bw[d / 4][0], bw[d / 4][1], bw[d / 4][2], bw[d / 4][3]});
                    }
                }
            }
        }
    };
    using T_ = std::true_type;
    using F_ = std::false_type;

    // prologue: stages 0 and 1 in flight, stage 0 landed, the fragments of substep 0 read
    // stages 0 and 1 of A and stages 0-2 of B in flight (in that order: A0 B0 A1 B1 B2),
    // stage 0 landed, the fragments of substep 0 read
    const int s1 = KT2 > 1 ? 1 : 0, s2 = KT2 > 2 ? 2 : KT2 - 1;
#pragma unroll
    for (int q = 0; q < C::LPW; ++q) load(q, 0, 0, A0, B0);
#pragma unroll
    for (int q = 0; q < C::LPW; ++q) load(q, s1, s1, A0 + C::SA, B0 + C::SB);
#pragma unroll
    for (int q = C::QA; q < C::LPW; ++q) load(q, s2, s2, A0, B0 + 2 * C::SB);
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(C::QA + 2 * C::QB, kNoLgkm));
    barrier();
#pragma unroll
    for (int nb = 0; nb < C::NBK; ++nb) bf[0][nb] = Frag<MODE>::weights(b_at(B0, nb, foff0));
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) af[0][mb] = Frag<MODE>::acts(a_at(A0, mb, foff0));
    // substep 0: stage 0, first half; reads its second half
    sub(T_{}, F_{}, af[0], bf[0], af[1], bf[1], A0, B0, foff1, 0, 0, A0, B0);
    int bi = 0;                                          // kt % 3
    for (int kt = 0; kt + 1 < KT2; ++kt) {
        const int bn = bi == 2 ? 0 : bi + 1;
        char* ca = A0 + (kt & 1) * C::SA;               // stage kt: free after the barrier
        char* cb = B0 + bi * C::SB;
        const char* na = A0 + ((kt + 1) & 1) * C::SA;
        const char* nbp = B0 + bn * C::SB;
        // past the end: re-read, never used
        const int ksa = kt + 2 < KT2 ? kt + 2 : KT2 - 1, ksb = kt + 3 < KT2 ? kt + 3 : KT2 - 1;
        // second half of stage kt; reads the first half of stage kt+1; loads A kt+2, B kt+3
        sub(F_{}, T_{}, af[1], bf[1], af[0], bf[0], na, nbp, foff0, ksa, ksb, ca, cb);
        // first half of stage kt+1; reads its second half
        sub(F_{}, F_{}, af[0], bf[0], af[1], bf[1], na, nbp, foff1, ksa, ksb, ca, cb);
        bi = bn;
    }
    // second half of the last stage: MFMAs only (after the two wait states its fragments'
    // last VALU writes need)
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 1" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < NM; ++i) mfma_agpr<false>(acc[i / C::MB][i % C::MB], bf[1][i / C::MB], af[1][i % C::MB]);
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 0));
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    GemmArgs gs = g;
    if (kslice) gs.out = (float*)g.out + (int64_t)kslice * g.rows_total * g.N;
    // the expansion, and a projection that adds into its output: the shared epilogue
    if (MODE == kExpand || (base_mode(MODE) == kDownAccum && g.accumulate)) {
        epilogue<MODE, C::MB, C::NBK, C::WTM, C::WTN, kOutCols>(gs, acc, row0, row1, ntile, wm, wn, lane);
        return;
    }
    // The projection's epilogue through LDS: each wave writes its outputs (the row scale
    // applied) in the MFMA layout (16 rows x 16 columns per block) into a private LDS area,
    // 64 rows at a time, and reads them back in row order, so that each store covers whole
    // rows with lanes in address order (2 rows of the wave's 128 columns) instead of half
    // lines of 16 rows: OLMoE-shaped projection-and-combine -4.3%, fine-grained -2.5%, the
    // 256 KB of float32 per tile being a quarter of the tile's time there (the expansion,
    // with half the output bytes per tile, was not faster this way). LDS row ro holds
    // 16-byte chunk c at position c ^ (ro & FM) (conflict-free writes of 16 rows x 1 chunk
    // and reads of 1 row x 16 chunks).
    constexpr int OUTW = C::WTN;                                     // output columns per wave
    constexpr int LPR = OUTW / 4;                                    // 16-byte chunks per row
    constexpr int RPI = 64 / LPR;                                     // rows per store
    constexpr int PM = C::MB < 4 ? C::MB : 4;                        // 16-row blocks per pass
    constexpr int RS = OUTW * 4;                                      // LDS row stride, bytes
    constexpr int FM = (LPR - 1) < 15 ? (LPR - 1) : 15;
    static_assert(C::MB % PM == 0 && 64 % LPR == 0 && C::NW * PM * 16 * RS <= C::LDS_BYTES, "LDS epilogue");
    float scs[C::MB];   // row scales, loaded first and waited for once
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) {
        const int r = min(row0 + wm * C::WTM + mb * 16 + (lane & 15), row1 - 1);
        scs[mb] = g.row_scale ? g.row_scale[scale_row(g, r)] : 1.0f;
    }
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, kNoLgkm));
    barrier();   // every wave's fragment reads of the last stage are done
    char* wl = lds + wave * (PM * 16 * RS);
    const int c0 = ntile * kOutCols + wn * OUTW;
    float* O = (float*)gs.out;
    const int N = g.N;
#pragma unroll
    for (int ps = 0; ps < C::MB / PM; ++ps) {
#pragma unroll
        for (int ml = 0; ml < PM; ++ml) {
            const int mb = ps * PM + ml, ro = ml * 16 + (lane & 15);
            const float sc = scs[mb];
#pragma unroll
            for (int nb = 0; nb < C::NBK; ++nb) {
                const float4 v = make_float4(acc[nb][mb][0] * sc, acc[nb][mb][1] * sc,
                                             acc[nb][mb][2] * sc, acc[nb][mb][3] * sc);
                const int c = nb * 4 + (lane >> 4);
                *(float4*)(wl + ro * RS + 16 * (c ^ (ro & FM))) = v;
            }
        }
#pragma unroll
        for (int i = 0; i < PM * 16 / RPI; ++i) {
            const int ro = i * RPI + lane / LPR, c = lane % LPR;
            const float4 v = *(const float4*)(wl + ro * RS + 16 * (c ^ (ro & FM)));
            const int r = row0 + wm * C::WTM + ps * PM * 16 + ro, col = c0 + c * 4;
            if (r < row1 && col < N) *(float4*)(O + (int64_t)r * N + col) = v;
        }
    }
}

// Work item of workgroup bid for the large-tile kernel, longest first. A group of c rows has
// c / BM full tiles and, if rows remain, one remainder tile: a long item when more than TBM
// rows remain, a short (tail-shape) item otherwise. Workgroups are dispatched round-robin over
// the 8 XCDs (bid % 8) and in bid order within each; each XCD's run of ids holds its eighth of
// the long items (every K slice) and then its eighth of the short items, so the short tiles
// fill the last round instead of lengthening it. Within each list the order is the grouped
// one of tile_from_id. Wave 0 counts and searches; the result is broadcast through LDS
// (s_item: group, row0, row1, ntile, kslice, valid). Returns false past the last item.
template <int BM, int TBM>
__device__ bool il_item(const GemmArgs& g, int nt, int GN, int* s_item) {
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        int lo[4], hi[4], full[4], nl[4], ns[4], suml = 0, sums = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int x = lane * 4 + j;
            int c = 0, b = 0;
            if (g.offsets == nullptr) {
                if (x == 0) c = (int)g.a_rows;
            } else if (x < g.n) {
                b = g.offsets[x];
                c = g.offsets[x + 1] - b;
            }
            const int rem = c % BM;
            lo[j] = b;
            hi[j] = b + c;
            full[j] = c / BM;
            nl[j] = full[j] + (rem > TBM ? 1 : 0);
            ns[j] = (rem > 0 && rem <= TBM) ? 1 : 0;
            suml += nl[j];
            sums += ns[j];
        }
        const int incl = wave_incl_scan_i32(suml), incs = wave_incl_scan_i32(sums);
        // 32-bit arithmetic throughout: the host keeps item counts (times 8) within range
        // the short list in halves: 2 * nt N-tiles of half width
        const int Lt = __builtin_amdgcn_readlane(incl, 63), St = __builtin_amdgcn_readlane(incs, 63);
        const int LT = Lt * nt * g.ksplit, ST = St * 2 * nt * g.ksplit;
        const int x8 = (int)(blockIdx.x % 8), j8 = (int)(blockIdx.x / 8);
        const int l0 = x8 * LT / 8, l1 = (x8 + 1) * LT / 8;
        const int s0 = x8 * ST / 8, s1 = (x8 + 1) * ST / 8;
        bool valid = true, is_long = true;
        int item = 0, count = Lt;
        if (j8 < l1 - l0) {
            item = l0 + j8;
        } else if (j8 - (l1 - l0) < s1 - s0) {
            item = s0 + j8 - (l1 - l0);
            is_long = false;
            count = St;
        } else {
            valid = false;
        }
        if (lane == 0) {
            s_item[5] = valid ? 1 : 0;
            s_item[6] = is_long ? 0 : 1;
        }
        if (valid) {
            const int ntl = is_long ? nt : 2 * nt, gnl = is_long ? GN : 2 * GN;
            const int per_slice = count * ntl;
            const int kslice = item / per_slice;
            // grouped order within the list (as tile_from_id)
            const int id = item - kslice * per_slice;
            const int gsize = gnl * count;
            const int grp = id / gsize, in = id - grp * gsize;
            const int gn = min(gnl, ntl - grp * gnl);
            const int m = in / gn;
            const int ntile = grp * gnl + (in - m * gn);
            // group holding list entry m: this lane's groups start at the exclusive prefix
            int start = is_long ? incl - suml : incs - sums;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int cnt = is_long ? nl[j] : ns[j];
                if (m >= start && m < start + cnt) {
                    const int r0 = lo[j] + (is_long ? (m - start) * BM : full[j] * BM);
                    s_item[0] = lane * 4 + j;
                    s_item[1] = r0;
                    s_item[2] = min(hi[j], r0 + BM);
                    s_item[3] = ntile;
                    s_item[4] = kslice;
                }
                start += cnt;
            }
        }
    }
    __syncthreads();
    return s_item[5] != 0;
}

// Work item of workgroup bid in the expert-major order. Group x has m_x = ceil(rows / BM)
// M-tiles; its m_x * nt items are walked in blocks of gn_x N-tiles (gn_x = window / m_x,
// at least 1), the M-tile varying slowest within a block, so that the `window` workgroups
// an XCD runs at once cover all of a group's rows for a few N-tiles: each weight tile is
// fetched while every row block that needs it runs, each activation tile once per block.
// Each XCD (bid % 8) takes a contiguous eighth of the list (every K slice, slice-major), or,
// for groups of at least 16 N tiles in multiples of 8, every eighth window (below). A last
// row block of at most TBM rows runs as the shorter tail tile.
// Wave 0 counts and searches; the result is broadcast through LDS as for il_item.
template <int BM, int TBM>
__device__ bool em_item(const GemmArgs& g, int nt, int window, int* s_item) {
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        int lo[4], cnt[4], m[4], local = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int x = lane * 4 + j;
            int c = 0, b = 0;
            if (g.offsets == nullptr) {
                if (x == 0) c = (int)g.a_rows;
            } else if (x < g.n) {
                b = g.offsets[x];
                c = g.offsets[x + 1] - b;
            }
            lo[j] = b;
            cnt[j] = c;
            m[j] = (c + BM - 1) / BM;
            local += m[j] * nt;
        }
        const int x8 = (int)(blockIdx.x % 8), j8 = (int)(blockIdx.x / 8);
        if (g.ksplit == 1 && nt % 8 == 0 && nt >= 16) {
            // Window-interleaved assignment: a group's N tiles are cut into windows of gw tiles,
            // gw the largest divisor of nt / 8 not above window / m (so that every window has
            // the same width and their number is a multiple of 8), and window i runs on XCD
            // i % 8. Every XCD then holds exactly an eighth of every group's items and works
            // through the groups in step with the others (the same mix of tile shapes at the
            // same time), instead of the XCDs holding different groups whose tiles take
            // different times (Mixtral-shaped expansion -1.9%); within a window the M-tile
            // varies slowest. With fewer than 16 N tiles a group's activation rows would be
            // fetched by every XCD for one N tile each (OLMoE-shaped projection +5%), so the
            // contiguous eighths below stay.
            // A group whose last row block takes the tail tile walks its windows over the full
            // row blocks first and then that row block over the same N tiles. Within an XCD the
            // hardware deals workgroups to its four shader arrays in strict rotation, one
            // array's turn waiting for a free compute unit there; with the tail row inside every
            // window the tail tiles repeat with the window's period and, where that period is
            // even, fall on the same one or two arrays, whose turns then come round faster than
            // the others' (Mixtral-shaped expansion: per-workgroup timelines, all 70 tail tiles
            // of an XCD on two of its arrays, 13% more work on the other two). A run of one
            // group's tail tiles gives every array the same mix: the mean gap between two tiles
            // on a compute unit fell from 4.8 to 1.1 us, the expansion 0.7% faster (its tiles
            // run slower with the compute units fuller, the clock falling under the load).
            const int n8 = nt / 8;
            int gw[4], mf[4], xl = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int last = cnt[j] - (m[j] - 1) * BM;   // rows of the last row block
                mf[j] = (m[j] > 0 && last <= TBM) ? m[j] - 1 : m[j];
                const int lim = window / (mf[j] > 0 ? mf[j] : 1);
                int d = lim < 1 ? 1 : (lim > n8 ? n8 : lim);
                while (n8 % d != 0) --d;
                gw[j] = d;
                xl += m[j] * n8;
            }
            const int xincl = wave_incl_scan_i32(xl);
            const bool valid = j8 < __builtin_amdgcn_readlane(xincl, 63);
            if (lane == 0) s_item[5] = valid ? 1 : 0;
            if (valid) {
                int start = xincl - xl;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int items = m[j] * n8;
                    if (j8 >= start && j8 < start + items) {
                        const int q = j8 - start;
                        int mm, col;
                        if (q < mf[j] * n8) {              // the full row blocks, window by window
                            const int gsize = gw[j] * mf[j];
                            const int kw = q / gsize, in = q - kw * gsize;
                            mm = in / gw[j];
                            col = (kw * 8 + x8) * gw[j] + (in - mm * gw[j]);   // window kw * 8 + x8
                        } else {                           // the tail row block, same N tiles
                            const int t = q - mf[j] * n8;
                            mm = m[j] - 1;
                            col = ((t / gw[j]) * 8 + x8) * gw[j] + t % gw[j];
                        }
                        const int r0 = lo[j] + mm * BM;
                        s_item[0] = lane * 4 + j;
                        s_item[1] = r0;
                        s_item[2] = min(lo[j] + cnt[j], r0 + BM);
                        s_item[3] = col;
                        s_item[4] = 0;
                    }
                    start += items;
                }
            }
        } else {
            const int incl = wave_incl_scan_i32(local);
            // 32-bit arithmetic throughout: the host keeps item counts (times 8) within range
            const int Tt = __builtin_amdgcn_readlane(incl, 63), TT = Tt * g.ksplit;
            const int l0 = x8 * TT / 8, l1 = (x8 + 1) * TT / 8;
            const bool valid = j8 < l1 - l0;
            if (lane == 0) s_item[5] = valid ? 1 : 0;
            if (valid) {
                const int item = l0 + j8;
                const int kslice = item / Tt;
                const int id = item - kslice * Tt;
                int start = incl - local;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int items = m[j] * nt;
                    if (id >= start && id < start + items) {
                        const int l = id - start;
                        int gn = window / m[j];
                        gn = gn < 1 ? 1 : (gn > nt ? nt : gn);
                        const int gsize = gn * m[j];
                        const int grp = l / gsize, in = l - grp * gsize;
                        const int gcols = min(gn, nt - grp * gn);
                        const int mm = in / gcols;
                        const int r0 = lo[j] + mm * BM;
                        s_item[0] = lane * 4 + j;
                        s_item[1] = r0;
                        s_item[2] = min(lo[j] + cnt[j], r0 + BM);
                        s_item[3] = grp * gn + (in - mm * gcols);
                        s_item[4] = kslice;
                    }
                    start += items;
                }
            }
        }
    }
    __syncthreads();
    return s_item[5] != 0;
}

// Work orders of the large-tile kernel.
enum IlOrder { kGrouped = 0, kLongestFirst = 1, kExpertMajor = 2 };

// order (an IlOrder): kLongestFirst is the order of il_item, kGrouped the grouped order of
// tile_of, kExpertMajor the order of em_item (group_n is then the window).
template <class C, class CT, int MODE>
__global__ __launch_bounds__(C::NT) void gemm_il_kernel(GemmArgs g, int64_t mt_upper, int nt,
                                                         int group_n, int order) {
    // half of a tail tile (128 x 128 for the large tiles, each wave 64 x 64): the longest-first
    // order runs each tail item as two of these, so that shorter items fill the last round
    using CH = ICfg<CT::BM, C::BNB / 2, CT::WM, CT::WN>;
    static_assert(CT::NT == C::NT && CT::BNB == C::BNB && CT::BM <= C::BM && CT::WTN == C::WTN,
                  "the tail tile runs on the same workgroup and N tiling");
    static_assert(CH::NT == C::NT && CH::LDS_BYTES <= C::LDS_BYTES, "the half tail tile fits");
    extern __shared__ __attribute__((aligned(1024))) char lds[];
    int* const s_item = (int*)lds;   // read into registers before the stage loads overwrite it
    int e, row0, row1, ntile, kslice;
    if (order == kLongestFirst) {          // workgroup-uniform branches and returns
        if (!il_item<C::BM, CT::BM>(g, nt, group_n, s_item)) return;
        e = s_item[0], row0 = s_item[1], row1 = s_item[2], ntile = s_item[3], kslice = s_item[4];
        const int half = s_item[6];
        __syncthreads();
        if (half) {                        // half of a tail item: N-tile of half width
            il_tile<CH, MODE>(g, lds, e, row0, row1, ntile, kslice);
            return;
        }
    } else if (order == kExpertMajor) {
        if (!em_item<C::BM, CT::BM>(g, nt, group_n, s_item)) return;
        e = s_item[0], row0 = s_item[1], row1 = s_item[2], ntile = s_item[3], kslice = s_item[4];
        __syncthreads();
    } else {
        int64_t mt;
        const int64_t per_slice = gridDim.x / g.ksplit;
        kslice = (int)(blockIdx.x / per_slice);
        if (!tile_of(blockIdx.x % per_slice, per_slice, mt_upper, nt, group_n, &mt, &ntile)) return;
        if (!find_tile<C::BM>(g.offsets, g.n, g.a_rows, mt, s_item)) return;
        e = s_item[0], row0 = s_item[1], row1 = s_item[2];
        __syncthreads();
    }
    if (row1 - row0 <= CT::BM)
        il_tile<CT, MODE>(g, lds, e, row0, row1, ntile, kslice);
    else
        il_tile<C, MODE>(g, lds, e, row0, row1, ntile, kslice);
}

// --------------------------------------------------------------- staged kernel
template <int BM_, int BNB_, int WM_, int WN_>
struct SCfg {
    static constexpr int BM = BM_, BNB = BNB_, WM = WM_, WN = WN_;
    static constexpr int NT = WM * WN * 64;
    static constexpr int WTM = BM / WM, WTN = BNB / WN, MB = WTM / 16, NBK = WTN / 16;
    static constexpr int A_ROWS = BM;                      // 128-byte LDS rows: 64 K values
    static constexpr int A_CHUNKS = A_ROWS * 8, B_CHUNKS = BNB * 8;
    static constexpr int A_PER_T = (A_CHUNKS + NT - 1) / NT, B_PER_T = (B_CHUNKS + NT - 1) / NT;
    static constexpr int STAGE = (A_ROWS + BNB) * 128;
    static constexpr int LDS_BYTES = 2 * STAGE;
    static_assert(WTM % 16 == 0 && WTN % 32 == 0, "whole MFMA blocks, gate/up halves");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
    static_assert(A_CHUNKS % NT == 0 && B_CHUNKS % NT == 0, "every thread owns whole chunks");
};

using MediumStaged = SCfg<128, 128, 2, 2>;

template <class C, int MODE>
__global__ __launch_bounds__(C::NT) void gemm_staged_kernel(GemmArgs g, int64_t mt_upper, int nt,
                                                            int group_n) {
    extern __shared__ __attribute__((aligned(1024))) char lds[];
    __shared__ int s_tile[3];
    int64_t mt;
    int ntile;
    if (!tile_of(blockIdx.x, gridDim.x, mt_upper, nt, group_n, &mt, &ntile)) return;
    if (!find_tile<C::BM>(g.offsets, g.n, g.a_rows, mt, s_tile)) return;
    const int e = s_tile[0], row0 = s_tile[1], row1 = s_tile[2];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / C::WN, wn = wave % C::WN;
    const int K = g.K;
    constexpr int kOutCols = (MODE == kExpand) ? C::BNB / 2 : C::BNB;

    // chunk i of a stage: LDS row i / 8, logical chunk i % 8 (16 bytes), stored at position
    // (i % 8) ^ ((row >> 1) & 7); every thread owns A_PER_T + B_PER_T chunks
    const char* aptr[C::A_PER_T];
    const char* bptr[C::B_PER_T];
    int aoff[C::A_PER_T], boff[C::B_PER_T];
#pragma unroll
    for (int i = 0; i < C::A_PER_T; ++i) {
        const int c = tid + i * C::NT, lr = c / 8, kc = c % 8;
        const int64_t srow = a_source_row(g, row0 + lr, row1);
        aptr[i] = (const char*)g.a + srow * (int64_t)K * 2 + kc * 16;
        aoff[i] = lr * 128 + ((kc ^ ((lr >> 1) & 7)) * 16);
    }
#pragma unroll
    for (int i = 0; i < C::B_PER_T; ++i) {
        const int c = tid + i * C::NT, j = c / 8, kc = c % 8;
        bptr[i] = (const char*)b_source_row<MODE, C::WTN, kOutCols>(g, e, ntile, j) + kc * 16;
        boff[i] = (C::A_ROWS + j) * 128 + ((kc ^ ((j >> 1) & 7)) * 16);
    }

    uint4 ra[C::A_PER_T], rb[C::B_PER_T];
#define PCM_STAGED_GLOAD(kt)                                                              \
    do {                                                                                  \
        _Pragma("unroll") for (int i = 0; i < C::A_PER_T; ++i)                            \
            ra[i] = *(const uint4*)(aptr[i] + (int64_t)(kt) * 128);                       \
        _Pragma("unroll") for (int i = 0; i < C::B_PER_T; ++i)                            \
            rb[i] = *(const uint4*)(bptr[i] + (int64_t)(kt) * 128);                       \
    } while (0)
#define PCM_STAGED_LSTORE(buf)                                                            \
    do {                                                                                  \
        char* S_ = lds + (buf) * C::STAGE;                                                \
        _Pragma("unroll") for (int i = 0; i < C::A_PER_T; ++i) *(uint4*)(S_ + aoff[i]) = ra[i]; \
        _Pragma("unroll") for (int i = 0; i < C::B_PER_T; ++i) *(uint4*)(S_ + boff[i]) = rb[i]; \
    } while (0)

    floatx4 acc[C::NBK][C::MB];
#pragma unroll
    for (int nb = 0; nb < C::NBK; ++nb)
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb) acc[nb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int KT = K / 64;
    PCM_STAGED_GLOAD(0);
    PCM_STAGED_LSTORE(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        // unconditional (the last step re-reads itself into the idle stage): a conditional
        // load keeps the staging registers out of SROA and in scratch memory
        PCM_STAGED_GLOAD(kt + 1 < KT ? kt + 1 : kt);
        const char* S = lds + cur * C::STAGE;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int ck = ks * 4 + (lane >> 4);
            const int off = (lane & 15) * 128 + ((ck ^ (((lane & 15) >> 1) & 7)) * 16);
            typename Frag<MODE>::T bfr[C::NBK], afr[C::MB];
#pragma unroll
            for (int nb = 0; nb < C::NBK; ++nb)
                bfr[nb] = Frag<MODE>::weights(S + (C::A_ROWS + wn * C::WTN + nb * 16) * 128 + off);
#pragma unroll
            for (int mb = 0; mb < C::MB; ++mb)
                afr[mb] = Frag<MODE>::acts(S + (wm * C::WTM + mb * 16) * 128 + off);
#pragma unroll
            for (int nb = 0; nb < C::NBK; ++nb)
#pragma unroll
                for (int mb = 0; mb < C::MB; ++mb) acc[nb][mb] = mfma_step(bfr[nb], afr[mb], acc[nb][mb]);
        }
        PCM_STAGED_LSTORE(cur ^ 1);
        __syncthreads();
    }
#undef PCM_STAGED_GLOAD
#undef PCM_STAGED_LSTORE
    epilogue<MODE, C::MB, C::NBK, C::WTM, C::WTN, kOutCols>(g, acc, row0, row1, ntile, wm, wn, lane);
}


// --------------------------------------------------------------- stream kernel
// Few rows per group (decode): the weights are the traffic. Each wave owns NB 16-row weight
// blocks (for the expansion, gate rows of NB / 2 blocks of 16 columns and the up rows of the
// same columns; for the projection, NB * 16 output columns) and one 16-row block of
// activation rows, and loads MFMA fragments straight from global memory into a ring of SDP
// register sets, SDP k-steps ahead of the MFMAs (no LDS). A lane reads 16 bytes of one row
// per k-step (row lane & 15, K offset 8 * (lane >> 4)), the same mapping for weights and
// activations; the activation fragment is shared by the wave's NB weight blocks.
constexpr int SROWS = 16;      // activation rows per tile
constexpr int SWAVES = 4;

template <int MODE, int NB, int SDP>
__global__ __launch_bounds__(SWAVES * 64) void gemm_stream_kernel(GemmArgs g, int64_t mt_upper,
                                                                 int nt, int n_fastest) {
    static_assert(NB % 2 == 0 && (NB + 1) * (SDP - 1) <= 63, "gate/up halves; vmcnt range");
    __shared__ int s_tile[3];
    const int64_t mt = n_fastest ? blockIdx.x / nt : blockIdx.x % mt_upper;
    const int ntile = n_fastest ? (int)(blockIdx.x % nt) : (int)(blockIdx.x / mt_upper);
    if (!find_tile<SROWS>(g.offsets, g.n, g.a_rows, mt, s_tile)) return;
    const int e = s_tile[0], row0 = s_tile[1], row1 = s_tile[2];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int K = g.K, N = g.N;
    // output columns of this wave: expansion NB * 8 (gate + up rows), projection NB * 16
    constexpr int kWaveCols = (MODE == kExpand) ? NB * 8 : NB * 16;
    const int col0 = (ntile * SWAVES + wave) * kWaveCols;
    if (col0 >= N) return;  // wave-uniform; no barrier follows
    const int r16 = lane & 15, kg = lane >> 4;
    // weight row of block b for this lane
    const uint16_t* wp[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        int wr;
        const uint16_t* base;
        if (MODE == kExpand) {
            wr = col0 + (b % (NB / 2)) * 16 + r16;
            base = (const uint16_t*)(b >= NB / 2 ? g.b1 : g.b0);
        } else {
            wr = col0 + b * 16 + r16;
            base = (const uint16_t*)g.b0;
        }
        wr = wr < N ? wr : N - 1;
        wp[b] = base + ((int64_t)e * N + wr) * K + kg * 8;
    }
    const uint16_t* ap = (const uint16_t*)g.a + a_source_row(g, row0 + r16, row1) * (int64_t)K + kg * 8;

    floatx4 acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[b] = floatx4{0.f, 0.f, 0.f, 0.f};
    bf16x8 wbuf[SDP][NB], abuf[SDP];
    const int KT = K / 32;
    auto load = [&](int slot, int kt) {
#pragma unroll
        for (int b = 0; b < NB; ++b) wbuf[slot][b] = *(const bf16x8*)(wp[b] + kt * 32);
        abuf[slot] = *(const bf16x8*)(ap + kt * 32);
    };
#pragma unroll
    for (int j = 0; j < SDP; ++j)
        if (j < KT) load(j, j);
    for (int base = 0; base < KT; base += SDP) {
#pragma unroll
        for (int j = 0; j < SDP; ++j) {
            const int kt = base + j;
            if (kt >= KT) break;
            // this step's NB + 1 loads have landed (the newer steps may still be in flight)
            if (kt + SDP - 1 < KT) __builtin_amdgcn_s_waitcnt(waitcnt_imm((NB + 1) * (SDP - 1), kNoLgkm));
            else __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, kNoLgkm));
            if constexpr (MODE == kExpand) {
#pragma unroll
                for (int b = 0; b < NB; ++b) acc[b] = mfma_step(wbuf[j][b], abuf[j], acc[b]);
            } else {
                const halfx8 a16 = __builtin_bit_cast(halfx8, abuf[j]);
#pragma unroll
                for (int b = 0; b < NB; ++b) acc[b] = mfma_step(Frag<MODE>::wide(wbuf[j][b]), a16, acc[b]);
            }
            if (kt + SDP < KT) load(j, kt + SDP);
        }
    }
    // epilogue: lane holds output columns c..c+3 (c = 4 * (lane >> 4)) of activation row r16
    // in each block
    const int r = row0 + r16;
    if (r >= row1) return;
    if (MODE == kExpand) {
#pragma unroll
        for (int b = 0; b < NB / 2; ++b) {
            const int f = col0 + b * 16 + 4 * kg;
            if (f >= N) continue;
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = silu(acc[b][i]) * acc[b + NB / 2][i];
            *(float4*)((float*)g.out + (int64_t)r * N + f) = make_float4(v[0], v[1], v[2], v[3]);
        }
    } else {
        const float sc = g.row_scale ? g.row_scale[scale_row(g, r)] : 1.0f;
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int h = col0 + b * 16 + 4 * kg;
            if (h >= N) continue;
            float4 v = make_float4(acc[b][0] * sc, acc[b][1] * sc, acc[b][2] * sc, acc[b][3] * sc);
            float4* dst = (float4*)((float*)g.out + (int64_t)r * N + h);
            if (base_mode(MODE) == kDownAccum && g.accumulate) {
                const float4 o = *dst;
                v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
            }
            *dst = v;
        }
    }
}

// LDS-ring streaming kernel: the streaming kernel with its operands staged through a per-wave
// LDS ring. A weight load of the register-ring kernel covers 16 rows x 64 bytes (the MFMA operand
// layout puts four lanes on a row), half a cache line per row, and the weight stream then ran
// at 5.4 TB/s; here each direct buffer -> LDS load covers 8 rows x 128 bytes (the 64 K values
// of two MFMA steps, whole lines) and the MFMA fragments are read back from LDS. Ring slot j of
// a wave holds NB blocks of 16 weight rows and one block of the 16 activation rows, each row
// 128 bytes with chunk c of row r at position c ^ ((r >> 1) & 7) (conflict-free fragment
// reads); D slots, D - 1 pairs in flight. No barrier: each wave owns its ring, and a slot is
// reloaded only after the MFMAs that used its fragments. With the activations in the ring as
// well, the loop holds no load into registers, whose waits the compiler would place itself
// (it drained every load in flight at the loop head). K is a multiple of 64 (as the layer
// entry points require of H and F), and `a` and one group's weights are below 4 GiB (32-bit
// buffer offsets); otherwise the register-ring kernel runs.
// (The body is a device function: the buffer resources and LDS-destination loads it uses have
// no host form, and the host pass does not emit a kernel whose own body uses them.)
template <int MODE, int NB, int D>
__device__ __forceinline__ void lstream_tile(const GemmArgs& g, char* lds, int e, int row0, int row1,
                                             int ntile) {
    static_assert(NB % 2 == 0 && D >= 2 && (D - 1) * (2 * NB + 2) <= 63, "gate/up halves; vmcnt range");
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int K = g.K, N = g.N;
    constexpr int kWaveCols = (MODE == kExpand) ? NB * 8 : NB * 16;
    const int col0 = (ntile * SWAVES + wave) * kWaveCols;
    if (col0 >= N) return;  // wave-uniform; no barrier follows
    constexpr int kSlot = (NB + 1) * 2048;   // NB weight blocks, then the activation block
    char* ring = lds + wave * (D * kSlot);
    // weight row (within expert e) behind row R of block b; rows past N repeat row N - 1
    auto wrow = [&](int b, int R) {
        const int wr = (MODE == kExpand) ? col0 + (b % (NB / 2)) * 16 + R : col0 + b * 16 + R;
        return wr < N ? wr : N - 1;
    };
    const int64_t wbytes = (int64_t)N * K * 2;
    const __amdgpu_buffer_rsrc_t rb0 = buffer_rsrc((const char*)g.b0 + e * wbytes, (uint32_t)wbytes);
    const __amdgpu_buffer_rsrc_t rb1 =
        MODE == kExpand ? buffer_rsrc((const char*)g.b1 + e * wbytes, (uint32_t)wbytes) : rb0;
    // load (b, h) of a pair: rows h * 8 + lane / 8 of block b, position lane % 8
    uint32_t voff[NB][2];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int R = h * 8 + (lane >> 3);
            const int chunk = (lane & 7) ^ ((R >> 1) & 7);
            voff[b][h] = (uint32_t)(wrow(b, R) * (int64_t)K * 2 + chunk * 16);
        }
    // activation loads (h = 0, 1): rows h * 8 + lane / 8, position lane % 8
    const __amdgpu_buffer_rsrc_t ra = buffer_rsrc(g.a, (uint32_t)((int64_t)g.a_rows * K * 2));
    uint32_t aoff[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int R = h * 8 + (lane >> 3);
        const int chunk = (lane & 7) ^ ((R >> 1) & 7);
        aoff[h] = (uint32_t)(a_source_row(g, row0 + R, row1) * (int64_t)K * 2 + chunk * 16);
    }
    const int r16 = lane & 15, kg = lane >> 4;
    // the projection's row scale, loaded and waited for before the loop (a load into a
    // register still in flight across the loop makes the compiler wait for every load in it)
    float sc = 1.0f;
    if constexpr (MODE != kExpand) {
        if (g.row_scale) sc = g.row_scale[scale_row(g, min(row0 + r16, row1 - 1))];
        __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, kNoLgkm));
    }
    // fragment of row r16, chunk 4 * step + kg
    const int fo0 = r16 * 128 + ((kg ^ ((r16 >> 1) & 7)) * 16);
    const int fo1 = r16 * 128 + (((4 + kg) ^ ((r16 >> 1) & 7)) * 16);

    floatx4 acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[b] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int KP = K / 64;
    auto issue = [&](int j, int p) {
        char* slot = ring + j * kSlot;
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int h = 0; h < 2; ++h)
                __builtin_amdgcn_raw_ptr_buffer_load_lds((MODE == kExpand && b >= NB / 2) ? rb1 : rb0,
                                                         (PCM_LDS void*)(slot + b * 2048 + h * 1024), 16,
                                                         voff[b][h], p * 128, 0, 0);
#pragma unroll
        for (int h = 0; h < 2; ++h)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (PCM_LDS void*)(slot + NB * 2048 + h * 1024), 16,
                                                     aoff[h], p * 128, 0, 0);
    };
#pragma unroll
    for (int j = 0; j < D - 1; ++j)
        if (j < KP) issue(j, j);
    for (int base = 0; base < KP; base += D) {
#pragma unroll
        for (int j = 0; j < D; ++j) {
            const int p = base + j;
            if (p >= KP) break;
            // slot (j + D - 1) % D held pair p - 1, whose fragments the previous MFMAs used
            if (p + D - 1 < KP) issue((j + D - 1) % D, p + D - 1);
            // pair p has landed: only the pairs issued after it may still be in flight
            if (p + D - 1 < KP) __builtin_amdgcn_s_waitcnt(waitcnt_imm((D - 1) * (2 * NB + 2), kNoLgkm));
            else __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, kNoLgkm));
            const char* slot = ring + j * kSlot;
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                const int fo = st ? fo1 : fo0;
                const bf16x8 av = *(const bf16x8*)(slot + NB * 2048 + fo);
                if constexpr (MODE == kExpand) {
#pragma unroll
                    for (int b = 0; b < NB; ++b)
                        acc[b] = mfma_step(*(const bf16x8*)(slot + b * 2048 + fo), av, acc[b]);
                } else {
                    const halfx8 a16 = __builtin_bit_cast(halfx8, av);
#pragma unroll
                    for (int b = 0; b < NB; ++b)
                        acc[b] = mfma_step(Frag<MODE>::weights(slot + b * 2048 + fo), a16, acc[b]);
                }
            }
        }
    }
    // epilogue: lane holds output columns c..c+3 (c = 4 * (lane >> 4)) of activation row r16
    // in each block
    const int r = row0 + r16;
    if (r >= row1) return;
    if (MODE == kExpand) {
#pragma unroll
        for (int b = 0; b < NB / 2; ++b) {
            const int f = col0 + b * 16 + 4 * kg;
            if (f >= N) continue;
            float v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = silu(acc[b][i]) * acc[b + NB / 2][i];
            *(float4*)((float*)g.out + (int64_t)r * N + f) = make_float4(v[0], v[1], v[2], v[3]);
        }
    } else {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int h = col0 + b * 16 + 4 * kg;
            if (h >= N) continue;
            float4 v = make_float4(acc[b][0] * sc, acc[b][1] * sc, acc[b][2] * sc, acc[b][3] * sc);
            float4* dst = (float4*)((float*)g.out + (int64_t)r * N + h);
            if (base_mode(MODE) == kDownAccum && g.accumulate) {
                const float4 o = *dst;
                v.x = __fadd_rn(o.x, v.x); v.y = __fadd_rn(o.y, v.y);
                v.z = __fadd_rn(o.z, v.z); v.w = __fadd_rn(o.w, v.w);
            }
            *dst = v;
        }
    }
}

template <int MODE, int NB, int D>
__global__ __launch_bounds__(SWAVES * 64) void gemm_lstream_kernel(GemmArgs g, int64_t mt_upper,
                                                                  int nt, int n_fastest) {
    extern __shared__ __attribute__((aligned(1024))) char lds[];
    __shared__ int s_tile[3];
    const int64_t mt = n_fastest ? blockIdx.x / nt : blockIdx.x % mt_upper;
    const int ntile = n_fastest ? (int)(blockIdx.x % nt) : (int)(blockIdx.x / mt_upper);
    if (!find_tile<SROWS>(g.offsets, g.n, g.a_rows, mt, s_tile)) return;
    lstream_tile<MODE, NB, D>(g, lds, s_tile[0], s_tile[1], s_tile[2], ntile);
}

template <int MODE, int NB, int D>
hipError_t launch_lstream_cfg(const GemmArgs& g, int64_t R, hipStream_t s) {
    const int64_t mt_upper = g.offsets ? ceil_div(R, SROWS) + g.n : ceil_div(R, SROWS);
    constexpr int kWgCols = SWAVES * ((MODE == kExpand) ? NB * 8 : NB * 16);
    constexpr int kLds = SWAVES * D * (NB + 1) * 2048;
    const int nt = (int)ceil_div(g.N, kWgCols);
    const int64_t grid = mt_upper * nt;
    if (grid <= 0) return hipSuccess;
    // set on every launch (idempotent, and the library keeps no state between calls)
    const hipError_t err = hipFuncSetAttribute((const void*)gemm_lstream_kernel<MODE, NB, D>,
                                               hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
    if (err != hipSuccess) return err;
    const int n_fastest = MODE == kExpand ? 1 : 0;
    gemm_lstream_kernel<MODE, NB, D><<<dim3((unsigned)grid), dim3(SWAVES * 64), kLds, s>>>(g, mt_upper, nt, n_fastest);
    return hipGetLastError();
}

template <int MODE, int NB, int SDP>
hipError_t launch_stream_cfg(const GemmArgs& g, int64_t R, hipStream_t s) {
    const int64_t mt_upper = g.offsets ? ceil_div(R, SROWS) + g.n : ceil_div(R, SROWS);
    constexpr int kWgCols = SWAVES * ((MODE == kExpand) ? NB * 8 : NB * 16);
    const int nt = (int)ceil_div(g.N, kWgCols);
    const int64_t grid = mt_upper * nt;
    if (grid <= 0) return hipSuccess;
    // the expansion runs a group's N tiles back to back (its gathered activation rows are then
    // shared through L2: 6% faster on the decode-shaped layer); the projection interleaves
    // the groups (4% faster than N tiles back to back there)
    const int n_fastest = MODE == kExpand ? 1 : 0;
    gemm_stream_kernel<MODE, NB, SDP><<<dim3((unsigned)grid), dim3(SWAVES * 64), 0, s>>>(g, mt_upper, nt, n_fastest);
    return hipGetLastError();
}

// Register-ring kernel: two 16-row blocks per wave, eight k-steps in flight (four or six
// blocks, or six steps, measured 1-3% slower on the decode-shaped layer).
template <int MODE>
hipError_t launch_stream(const GemmArgs& g, int64_t R, hipStream_t s, int depth) {
    // the LDS-ring kernel (whole-line weight loads) where its constraints hold; ring depth 3
    // for the expansion and 2 for the projection (decode-shaped layer: 2-6 within 0.5% for the
    // expansion; the projection 3% slower at 3 and 45% at 4, where the compiler waits for every
    // load in flight before the fragment reads and only one workgroup fits a compute unit);
    // a forced depth of 0 runs the register-ring kernel
    if (g.K % 64 == 0 && g.a_rows * g.K * 2 < (int64_t(1) << 32) && (int64_t)g.N * g.K * 2 < (int64_t(1) << 32)) {
        const int dv = depth >= 0 ? depth : (MODE == kExpand ? 3 : 2);
        if (dv == 2) return launch_lstream_cfg<MODE, 2, 2>(g, R, s);
        if (dv == 4) return launch_lstream_cfg<MODE, 2, 4>(g, R, s);
        if (dv == 6) return launch_lstream_cfg<MODE, 2, 6>(g, R, s);
        if (dv != 0) return launch_lstream_cfg<MODE, 2, 3>(g, R, s);
    }
    return launch_stream_cfg<MODE, 2, 8>(g, R, s);
}

// ---------------------------------------------------------------------- launch
template <class C, int MODE, bool IL, class CT = LargeIlTail>
hipError_t launch_cfg(const GemmArgs& g, int64_t R, hipStream_t s, const GemmTune& t) {
    // set on every launch (idempotent, and the library keeps no state between calls)
    const void* fn;
    if constexpr (IL)
        fn = (const void*)gemm_il_kernel<C, CT, MODE>;
    else
        fn = (const void*)gemm_staged_kernel<C, MODE>;
    const hipError_t err = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
    if (err != hipSuccess) return err;
    const int64_t mt_upper = g.offsets ? ceil_div(R, C::BM) + g.n : ceil_div(R, C::BM);
    constexpr int kOutCols = (MODE == kExpand) ? C::BNB / 2 : C::BNB;
    const int nt = (int)ceil_div(g.N, kOutCols);
    if (mt_upper * nt <= 0) return hipSuccess;
    const int group_n = t.group_n > 0 ? t.group_n : 4;
    if constexpr (IL) {
        // default: expert-major for grouped rows, except for a projection whose tiles fill fewer
        // than 4 rounds of the chip (or that splits K), which takes the longest-first order (its
        // short items fill the last round; the expert-major order was 17% slower on the
        // Mixtral-shaped projection without a K split); one group of rows the orders tuned for it
        int order = t.order;
        if (order < 0 || order > 2) {
            if (g.offsets == nullptr) order = MODE == kExpand ? kGrouped : kLongestFirst;
            else order = (MODE != kExpand && (g.ksplit > 1 || mt_upper * nt < 4 * 256))
                             ? kLongestFirst : kExpertMajor;
        }
        // the searches of il_item and em_item run in 32-bit integers (item counts times 8)
        if ((mt_upper + g.n + 1) * nt * g.ksplit >= (int64_t(1) << 27)) order = kGrouped;
        int64_t grid;
        int gparam = group_n;
        if (order == kLongestFirst) {
            // each XCD's run holds at most ceil(long / 8) + ceil(2 * short / 8) items, where
            // long + short <= mt_upper * nt * ksplit and short <= groups * nt * ksplit
            const int64_t groups = g.offsets ? g.n : 1;
            grid = (ceil_div((mt_upper + groups) * nt * g.ksplit, 8) + 2) * 8;
        } else if (order == kExpertMajor) {
            // each XCD's run holds at most ceil(items / 8) <= ceil(mt_upper * nt * ksplit / 8)
            // window 8: with three weight stages 0.2-1.1% ahead of 12, 16 and 24 on the three
            // grouped workloads (12 was best with two)
            grid = ceil_div(mt_upper * nt * g.ksplit, 8) * 8;
            gparam = t.window > 0 ? t.window : 8;
        } else {
            grid = ceil_div(mt_upper * nt, 8) * 8 * g.ksplit;
        }
        gemm_il_kernel<C, CT, MODE><<<dim3((unsigned)grid), dim3(C::NT), C::LDS_BYTES, s>>>(
            g, mt_upper, nt, gparam, order);
    } else {
        const int64_t grid = ceil_div(mt_upper * nt, 8) * 8 * g.ksplit;
        gemm_staged_kernel<C, MODE><<<dim3((unsigned)grid), dim3(C::NT), C::LDS_BYTES, s>>>(g, mt_upper, nt, group_n);
    }
    return hipGetLastError();
}

// Tile shape: a forced choice (tile = 'S', 'M' or 'L', for tests and tuning), otherwise by the
// mean rows per group (below 16 the streaming kernel, else the large tiles). The large tiles
// address `a` and one group's weights through 32-bit buffer offsets, so both must stay below
// 4 GiB (a_bytes: all rows of `a`; w_bytes: one group's weights).
char pick_tile(int64_t R, int groups, int64_t a_bytes, int64_t w_bytes, char tile) {
    const bool large_ok = a_bytes < (int64_t(1) << 32) && w_bytes < (int64_t(1) << 32);
    if (tile == 'S' || tile == 'M' || tile == 'L' || tile == 'W')
        return (tile == 'L' || tile == 'W') && !large_ok ? 'M' : tile;
    // below 16 rows per group the streaming kernel (weights streamed once, little MFMA work
    // wasted on padding); from 16 on the large tiles, which were faster than the medium ones
    // at every size measured (Mixtral-shaped, 1024 tokens: 2.6 -> 0.87 ms for the two GEMMs
    // and the combine) and than the streaming kernel from 16 rows per group on; the medium
    // tiles only where the large tiles' 32-bit offsets would not reach
    const int64_t mean = R / (groups > 0 ? groups : 1);
    if (mean < 16) return 'S';
    return large_ok ? 'L' : 'M';
}

}  // namespace

int down_ksplit(int64_t R, int n, int H, int F, char tile) {
    // only the large-tile kernel slices K; its grid is (R/256 + n) x (H/256) tiles. Below one
    // round of the chip the K split doubles the workgroups; from one round on the longest-first
    // order (tail items as halves) fills the last round as well without the second o slice
    // (Mixtral-shaped projection and combine 922 -> 902 us, with 268 MB less o traffic)
    const char t = pick_tile(R, n, R * F * 2, (int64_t)H * F * 2, tile);
    if (t != 'L' && t != 'W') return 1;
    const int64_t tiles = (ceil_div(R, 256) + n) * ceil_div(H, 256);
    return (tiles < 256 && (F / 2) % 64 == 0 && F / 32 >= 128) ? 2 : 1;
}

namespace {
template <int MODE>
hipError_t launch_mode(const GemmArgs& g, int64_t R, hipStream_t s, const GemmTune& tune, char t) {
    if (t == 'S') return launch_stream<MODE>(g, R, s, tune.stream_depth);
    if (t == 'M') return launch_cfg<MediumStaged, MODE, false>(g, R, s, tune);
    // the large tiles: eight waves for the expansion, four for the projections (interleaved
    // A/B, bit-identical: expansion -2.7% / -2.4% / -0.3% on the Mixtral-, OLMoE- and
    // fine-grained-shaped layers, projections +1% to +1.7%)
    if (t == 'W' || (t == 'L' && MODE == kExpand && tune.tile != 'L'))
        return launch_cfg<WideIl, MODE, true, WideIlTail>(g, R, s, tune);
    return launch_cfg<LargeIl, MODE, true>(g, R, s, tune);
}
}  // namespace

hipError_t launch_gemm_bf16(GemmMode mode, const GemmArgs& g0, int64_t R, hipStream_t s,
                            const GemmTune& tune) {
    GemmArgs g = g0;
    if (g.ksplit < 1) g.ksplit = 1;
    const char t = pick_tile(R, g.offsets ? g.n : 1, g.a_rows * g.K * 2, (int64_t)g.N * g.K * 2, tune.tile);
    if (g.ksplit > 1 && (mode != kDownStore || (t != 'L' && t != 'W'))) return hipErrorInvalidValue;
    switch (mode) {
        case kExpand: return launch_mode<kExpand>(g, R, s, tune, t);
        case kDownStore:
            return g.b_f16 ? launch_mode<kDownStore | kHalfW>(g, R, s, tune, t)
                           : launch_mode<kDownStore>(g, R, s, tune, t);
        default:
            return g.b_f16 ? launch_mode<kDownAccum | kHalfW>(g, R, s, tune, t)
                           : launch_mode<kDownAccum>(g, R, s, tune, t);
    }
}

hipError_t launch_widen_f16(const uint16_t* src, int64_t count, uint16_t* dst, hipStream_t s) {
    if (count <= 0) return hipSuccess;
    const int64_t n8 = count / 8;
    const int64_t blocks = n8 > 0 ? (ceil_div(n8, 256) < 8192 ? ceil_div(n8, 256) : 8192) : 1;
    widen_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(src, count, dst);
    return hipGetLastError();
}

}  // namespace pcm
