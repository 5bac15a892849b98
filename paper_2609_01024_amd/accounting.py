"""Algorithmic work of the path-compositional MoE layer: FLOPs and bytes.

Only work the method must do is counted: the expansion of each (token, source)
pair once (Section 4.3's source-grouped reuse), one projection per (token,
target) pair after mixing the sources bound for that target (the projection is
linear, Section 4.1), and the mix itself. Padding rows, dense n x n work and
per-path projections that the rewrite avoids are never counted.
"""
from __future__ import annotations

BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3    # MI355X fp32 vector
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E


def expansion_flops_per_row(H: int, F: int) -> int:
    """Gate and up projections of one expert for one token (2 flops per MAC)."""
    return 2 * 2 * H * F


def projection_flops_per_row(H: int, F: int) -> int:
    """Down projection of one expert for one token."""
    return 2 * H * F


def expert_flops(H: int, F: int) -> int:
    return expansion_flops_per_row(H, F) + projection_flops_per_row(H, F)


def gemm_flops(R: int, H: int, F: int, T: int = 0, shared_F: int = 0, R_tgt: int = None) -> dict:
    """Executed MFMA work of the grouped GEMMs for R expansion rows and R_tgt projection rows
    (both T*k for the top-k router; the distinct sources and targets for the scored router),
    plus a shared expert."""
    R_tgt = R if R_tgt is None else R_tgt
    exp = R * expansion_flops_per_row(H, F)
    proj = R_tgt * projection_flops_per_row(H, F)
    sh_exp = T * expansion_flops_per_row(H, shared_F) if shared_F else 0
    sh_proj = T * projection_flops_per_row(H, shared_F) if shared_F else 0
    return {"expand": exp, "project": proj, "shared_expand": sh_exp, "shared_project": sh_proj,
            "total": exp + proj + sh_exp + sh_proj}


def mix_flops(F: int, n_paths: int) -> int:
    """z_(t,b) = sum_a beta_ab U_(t,a): one multiply-add per path and column."""
    return 2 * F * n_paths


def expanded_bytes(R: int, F: int, elem: int) -> int:
    return R * F * elem


def decode_weight_bytes(touched_experts: int, H: int, F: int, elem: int,
                        shared_F: int = 0) -> int:
    """Weight bytes a layer must stream when each touched expert is read once."""
    return touched_experts * 3 * H * F * elem + (3 * H * shared_F * elem if shared_F else 0)


# ------------------------------------------------------------ bytes of the memory-bound stages
def route_bytes(T: int, n: int, k: int) -> int:
    """Top-k of T logit rows: the logits in, ids and weights out."""
    return T * n * 4 + T * k * 8


def paths_bytes(T: int, n: int, k: int) -> int:
    """Path table and dispatch layout: ids and weights in (and the n x n mask once); path bits,
    weights beta, row_token / row_slot / row_of and the offsets out."""
    return T * k * 8 + n * n + T * 8 + T * k * k * 4 + T * k * 12 + (n + 1) * 4


def route_paths_bytes(T: int, n: int, k: int) -> int:
    """The fused indexing operation: the logits and the packed mask in; ids and weights, path
    bits, weights beta, row_token / row_slot / row_of and the offsets out."""
    return (T * n * 4 + n * ((n + 63) // 64) * 8 + T * k * 8 + T * 8 + T * k * k * 4
            + T * k * 12 + (n + 1) * 4)


def mix_bytes(R_src: int, R_tgt: int, F: int, T: int, K: int, u_elem: int = 4,
              z_elem: int = 2) -> int:
    """z_(t,b) = sum_a beta_ab u_(t,a): every U row in, every z row (and its scale) out, plus
    the per-token bits, weights and row indices."""
    return (R_src * F * u_elem + R_tgt * F * z_elem + (R_tgt * 4 if z_elem == 2 else 0)
            + T * 8 + T * K * K * 4 + 2 * T * K * 4)


def combine_bytes(R_tgt: int, H: int, T: int, K: int, ksplit: int = 1,
                  accumulate: bool = False) -> int:
    """y_t = [y_t] + sum_b o_(t,b): every o row of every K slice in, y out (and in when
    accumulating), plus the row indices."""
    return ksplit * R_tgt * H * 4 + T * H * 4 * (2 if accumulate else 1) + T * K * 4
