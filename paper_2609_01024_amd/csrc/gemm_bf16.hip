// Grouped bf16 GEMMs on the gfx950 matrix cores (v_mfma_f32_16x16x32_bf16, float32
// accumulate) for the two sides of a SwiGLU expert (Section 4.1):
//   expand:  U[r, f] = SiLU(x[tok(r)] . W_gate[e][f]) * (x[tok(r)] . W_up[e][f])
//            one row per (token, source) pair, rows of expert e contiguous (Section 4.3),
//            x rows gathered through row_token; SwiGLU fused into the epilogue; U kept in
//            float32 (or written as split hi/lo bf16 pairs for a dense FFN).
//   down:    O[r, h] = Z[r] . W_down[e][h]        (store, or accumulate into y for a
//                                                  dense FFN whose rows are tokens)
//            Z arrives as split hi/lo bf16 pairs; each weight fragment is multiplied by
//            both halves, so the product sees Z to ~2^-17 relative.
// Both operands are K-contiguous (x rows and W rows run along H; Z rows and W_down rows
// along F), so a lane's 8 consecutive K values of a row are one 16-byte load.
//
// Tile: BM rows x BNB weight rows x 64 K per stage, two LDS stages (global loads of
// stage k+1 overlap the MFMAs of stage k). LDS rows are padded by 16 bytes, which makes
// the 16-byte fragment reads of 16 consecutive rows bank-conflict-free. The MFMA takes
// the weight fragment as its first operand, so each lane's four accumulators are four
// consecutive output columns of one row (16-byte float32 stores).
// For the expansion, a wave's weight rows are half gate and half up for the same columns,
// so gate and up values of an output element sit in the same lane and register slot.
//
// Work decomposition: the grid is (upper bound of M tiles) x (N tiles). Each workgroup
// finds its group (expert) and row range from the group offsets with one wave-wide scan
// of per-group tile counts; workgroups past the last tile exit.
#include <stdlib.h>
#include <string.h>

#include "internal.h"

namespace pcm {
namespace {

constexpr int BK = 64;

template <int BM_, int BNB_, int WM_, int WN_, int AK_>
struct Cfg {
    static constexpr int BM = BM_, BNB = BNB_, WM = WM_, WN = WN_;
    static constexpr int AK = AK_;                 // A columns staged per K step (64, or 128 = hi|lo)
    static constexpr int NT = WM * WN * 64;
    static constexpr int WTM = BM / WM, WTN = BNB / WN;
    static constexpr int MB = WTM / 16, NBK = WTN / 16;
    static constexpr int A_STRIDE = AK + 8, B_STRIDE = BK + 8;  // bf16 elements per LDS row
    static constexpr int A_CPR = AK / 8, B_CPR = BK / 8;       // 16-byte chunks per row
    static constexpr int A_CHUNKS = BM * A_CPR, B_CHUNKS = BNB * B_CPR;
    static constexpr int A_PER_T = (A_CHUNKS + NT - 1) / NT, B_PER_T = (B_CHUNKS + NT - 1) / NT;
    static constexpr int LDS_A = BM * A_STRIDE, LDS_B = BNB * B_STRIDE;
    static constexpr int LDS_BYTES = 2 * (LDS_A + LDS_B) * 2;
    static_assert(WTM % 16 == 0 && WTN % 16 == 0, "wave tile must hold whole MFMA blocks");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
};

// expansion tiles (A = x rows, 64 K per stage)
using ExpL = Cfg<256, 256, 2, 4, 64>;
using ExpM = Cfg<128, 128, 2, 2, 64>;
using ExpS = Cfg<16, 256, 1, 4, 64>;
// projection tiles (A = split z rows: 64 hi + 64 lo per stage)
using DownL = Cfg<128, 256, 2, 4, 128>;
using DownM = Cfg<64, 128, 1, 4, 128>;
using DownS = Cfg<16, 128, 1, 4, 128>;

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
        int incl = local;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int v = __shfl_up(incl, d);
            if (lane >= d) incl += v;
        }
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

__device__ inline uint32_t pack_bf16x2(float a, float b) {
    return (uint32_t)f32_to_bf16_rne(a) | ((uint32_t)f32_to_bf16_rne(b) << 16);
}

template <class C, int MODE>
__global__ __launch_bounds__(C::NT) void gemm_bf16_kernel(GemmArgs g, int64_t mt_upper) {
    extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
    __shared__ int s_tile[3];
    constexpr bool kSplitA = C::AK == 2 * BK;
    static_assert(MODE == kExpand ? !kSplitA : kSplitA, "expand reads x, down reads split z");
    const int64_t mt = blockIdx.x % mt_upper;
    const int ntile = (int)(blockIdx.x / mt_upper);
    if (!find_tile<C::BM>(g.offsets, g.n, g.a_rows, mt, s_tile)) return;
    const int e = s_tile[0], row0 = s_tile[1], row1 = s_tile[2];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / C::WN, wn = wave % C::WN;
    const int K = g.K, N = g.N;
    const int64_t a_row_elems = kSplitA ? 2 * (int64_t)K : K;      // bf16 elements per A row
    constexpr int kOutCols = (MODE == kExpand) ? C::BNB / 2 : C::BNB;  // output columns per tile

    // Global source of each 16-byte chunk this thread stages.
    const uint16_t* aptr[C::A_PER_T];
    const uint16_t* bptr[C::B_PER_T];
    const uint16_t* A = (const uint16_t*)g.a;
#pragma unroll
    for (int i = 0; i < C::A_PER_T; ++i) {
        const int c = tid + i * C::NT;
        const int row = c / C::A_CPR, kc = c % C::A_CPR;
        const int r = row0 + row;
        aptr[i] = nullptr;
        if (c < C::A_CHUNKS && r < row1) {
            int64_t src = r;
            if (g.gather) {
                src = g.gather[r];
                src = src < 0 ? 0 : (src >= g.a_rows ? g.a_rows - 1 : src);
            }
            aptr[i] = A + src * a_row_elems + kc * 8;
        }
    }
#pragma unroll
    for (int i = 0; i < C::B_PER_T; ++i) {
        const int c = tid + i * C::NT;
        const int j = c / C::B_CPR, kc = c % C::B_CPR;
        bptr[i] = nullptr;
        if (c < C::B_CHUNKS) {
            if (MODE == kExpand) {
                const int grp = j / C::WTN, jj = j % C::WTN, half = jj / (C::WTN / 2);
                const int f = ntile * kOutCols + grp * (C::WTN / 2) + jj % (C::WTN / 2);
                if (f < N)
                    bptr[i] = (const uint16_t*)(half ? g.b1 : g.b0) + ((int64_t)e * N + f) * K + kc * 8;
            } else {
                const int h = ntile * kOutCols + j;
                if (h < N) bptr[i] = (const uint16_t*)g.b0 + ((int64_t)e * N + h) * K + kc * 8;
            }
        }
    }

    uint4 ra[C::A_PER_T], rb[C::B_PER_T];
    auto gload = [&](int kt) {
#pragma unroll
        for (int i = 0; i < C::A_PER_T; ++i)
            ra[i] = aptr[i] ? *(const uint4*)(aptr[i] + (int64_t)kt * C::AK) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < C::B_PER_T; ++i)
            rb[i] = bptr[i] ? *(const uint4*)(bptr[i] + (int64_t)kt * BK) : make_uint4(0, 0, 0, 0);
    };
    auto lstore = [&](int buf) {
        uint16_t* As = lds + buf * (C::LDS_A + C::LDS_B);
        uint16_t* Bs = As + C::LDS_A;
#pragma unroll
        for (int i = 0; i < C::A_PER_T; ++i) {
            const int c = tid + i * C::NT;
            if (c < C::A_CHUNKS) *(uint4*)(As + (c / C::A_CPR) * C::A_STRIDE + (c % C::A_CPR) * 8) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < C::B_PER_T; ++i) {
            const int c = tid + i * C::NT;
            if (c < C::B_CHUNKS) *(uint4*)(Bs + (c / C::B_CPR) * C::B_STRIDE + (c % C::B_CPR) * 8) = rb[i];
        }
    };

    floatx4 acc[C::NBK][C::MB];
#pragma unroll
    for (int nb = 0; nb < C::NBK; ++nb)
#pragma unroll
        for (int mb = 0; mb < C::MB; ++mb) acc[nb][mb] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int KT = K / BK;
    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < KT; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < KT) gload(kt + 1);
        const uint16_t* As = lds + cur * (C::LDS_A + C::LDS_B);
        const uint16_t* Bs = As + C::LDS_A;
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            bf16x8 bfr[C::NBK], afr[C::MB];
            const int koff = ks * 32 + (lane >> 4) * 8;
#pragma unroll
            for (int nb = 0; nb < C::NBK; ++nb)
                bfr[nb] = *(const bf16x8*)(Bs + (wn * C::WTN + nb * 16 + (lane & 15)) * C::B_STRIDE + koff);
#pragma unroll
            for (int mb = 0; mb < C::MB; ++mb)
                afr[mb] = *(const bf16x8*)(As + (wm * C::WTM + mb * 16 + (lane & 15)) * C::A_STRIDE + koff);
#pragma unroll
            for (int nb = 0; nb < C::NBK; ++nb)
#pragma unroll
                for (int mb = 0; mb < C::MB; ++mb)
                    acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[nb], afr[mb], acc[nb][mb], 0, 0, 0);
            if (kSplitA) {  // the low halves, same weight fragments
#pragma unroll
                for (int mb = 0; mb < C::MB; ++mb)
                    afr[mb] = *(const bf16x8*)(As + (wm * C::WTM + mb * 16 + (lane & 15)) * C::A_STRIDE + BK + koff);
#pragma unroll
                for (int nb = 0; nb < C::NBK; ++nb)
#pragma unroll
                    for (int mb = 0; mb < C::MB; ++mb)
                        acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[nb], afr[mb], acc[nb][mb], 0, 0, 0);
            }
        }
        if (kt + 1 < KT) lstore(cur ^ 1);
        __syncthreads();
    }

    // Epilogue: lane holds columns c0..c0+3 of row (lane & 15) of each 16x16 block.
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) {
        const int r = row0 + wm * C::WTM + mb * 16 + (lane & 15);
        if (r >= row1) continue;
        if (MODE == kExpand) {
#pragma unroll
            for (int nb = 0; nb < C::NBK / 2; ++nb) {
                const int f = ntile * kOutCols + wn * (C::WTN / 2) + nb * 16 + (lane >> 4) * 4;
                if (f >= N) continue;
                const floatx4 gt = acc[nb][mb], up = acc[nb + C::NBK / 2][mb];
                float v[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = gt[i] / (1.0f + __expf(-gt[i])) * up[i];
                if (g.split_out) {
                    // hi at [blk][0..63], lo at [blk][64..127] of the row's split layout
                    uint16_t* U = (uint16_t*)g.out + (int64_t)r * 2 * N + (f / kSplitBlock) * 2 * kSplitBlock
                                  + f % kSplitBlock;
                    float lo[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) lo[i] = v[i] - bf16_bits_to_f32(f32_to_bf16_rne(v[i]));
                    *(uint2*)U = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
                    *(uint2*)(U + kSplitBlock) = make_uint2(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]));
                } else {
                    *(float4*)((float*)g.out + (int64_t)r * N + f) = make_float4(v[0], v[1], v[2], v[3]);
                }
            }
        } else {
            float* O = (float*)g.out;
#pragma unroll
            for (int nb = 0; nb < C::NBK; ++nb) {
                const int h = ntile * kOutCols + wn * C::WTN + nb * 16 + (lane >> 4) * 4;
                if (h >= N) continue;
                float4 v = make_float4(acc[nb][mb][0], acc[nb][mb][1], acc[nb][mb][2], acc[nb][mb][3]);
                float4* dst = (float4*)(O + (int64_t)r * N + h);
                if (MODE == kDownAccum && g.accumulate) {
                    const float4 o = *dst;
                    v.x += o.x; v.y += o.y; v.z += o.z; v.w += o.w;
                }
                *dst = v;
            }
        }
    }
}

template <class C, int MODE>
hipError_t launch_cfg(const GemmArgs& g, int64_t R, hipStream_t s) {
    static bool attr_set = false;  // idempotent; a race only repeats the same call
    if (!attr_set) {
        hipError_t err = hipFuncSetAttribute((const void*)gemm_bf16_kernel<C, MODE>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES);
        if (err != hipSuccess) return err;
        attr_set = true;
    }
    const int64_t mt_upper = g.offsets ? ceil_div(R, C::BM) + g.n : ceil_div(R, C::BM);
    constexpr int kOutCols = (MODE == kExpand) ? C::BNB / 2 : C::BNB;
    const int64_t nt = ceil_div(g.N, kOutCols);
    const int64_t grid = mt_upper * nt;
    if (grid <= 0) return hipSuccess;
    gemm_bf16_kernel<C, MODE><<<dim3((unsigned)grid), dim3(C::NT), C::LDS_BYTES, s>>>(g, mt_upper);
    return hipGetLastError();
}

// Tile shape: an environment override (PCM_GEMM_TILE = S | M | L) for tests and tuning,
// otherwise by the mean rows per group.
char pick_tile(int64_t R, int groups) {
    const char* env = getenv("PCM_GEMM_TILE");
    if (env && (env[0] == 'S' || env[0] == 'M' || env[0] == 'L')) return env[0];
    const int64_t mean = R / (groups > 0 ? groups : 1);
    if (mean <= 48) return 'S';
    if (mean < 512) return 'M';
    return 'L';
}

}  // namespace

hipError_t launch_gemm_bf16(GemmMode mode, const GemmArgs& g, int64_t R, hipStream_t s) {
    const char t = pick_tile(R, g.offsets ? g.n : 1);
    if (mode == kExpand) {
        if (t == 'S') return launch_cfg<ExpS, kExpand>(g, R, s);
        if (t == 'M') return launch_cfg<ExpM, kExpand>(g, R, s);
        return launch_cfg<ExpL, kExpand>(g, R, s);
    }
    if (mode == kDownStore) {
        if (t == 'S') return launch_cfg<DownS, kDownStore>(g, R, s);
        if (t == 'M') return launch_cfg<DownM, kDownStore>(g, R, s);
        return launch_cfg<DownL, kDownStore>(g, R, s);
    }
    if (t == 'S') return launch_cfg<DownS, kDownAccum>(g, R, s);
    if (t == 'M') return launch_cfg<DownM, kDownAccum>(g, R, s);
    return launch_cfg<DownL, kDownAccum>(g, R, s);
}

}  // namespace pcm
