"""Seeded input generation.

Every tensor is drawn from ``numpy.random.default_rng([seed, tensor_id, chunk])``
in float32 and, for bf16 layers, rounded to bfloat16 (round to nearest even) by
torch. Per-expert chunks are drawn on a thread pool; the values do not depend on
the pool size.

Distributions ("N(0, s)" means standard deviation s):
  x            N(0, x_std)                                   [T, H]
  W_gate/W_up  N(0, w_std), expert e from chunk e             [n, F, H]
  W_down       N(0, w_std)                                    [n, H, F]
  shared       N(0, w_std)                                    [F_s, H], [F_s, H], [H, F_s]
  logits       router:      x @ W_r^T, W_r ~ N(0, w_std), float64 product rounded to float32
               normal:      N(0, 1)
               normal_bias: N(0, 1) + b_e, b_e ~ N(0, bias_std)
               zipf:        N(0, 1) - s * ln(rank_e), rank a seeded permutation of 1..n
               +ties:       rounded to multiples of 0.25 (exact ties are common)
               +one_expert: expert 0's logit raised by 100 for every token
  mask         each off-diagonal entry 1 with probability `density`, diagonal 1, uint8 [n, n]
               (row = expansion source i, column = projection target j)

Scored compositional routing (make_scored_inputs) adds:
  g_tgt        N(0, 1)                                        [T, n] (target-side prior)
  bias         compatibility bias B: 0 on the diagonal, c + U(-a, a) off it with
               c = -1, a = 0.5 (the negative-offset, bounded-noise initialisation)   [n, n]
  lambda       0.5 (weight of the target prior)
The base routing signal g_base is the layer's logits.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from .configs import LayerConfig

TID_X, TID_LOGITS, TID_ROUTER, TID_BIAS, TID_RANK, TID_MASK = 0, 1, 2, 3, 4, 5
TID_WG, TID_WU, TID_WD = 10, 11, 12
TID_SWG, TID_SWU, TID_SWD = 20, 21, 22
TID_GTGT, TID_COMPAT = 6, 7

SCORED_LAMBDA = 0.5
COMPAT_C, COMPAT_NOISE = -1.0, 0.5


def _rng(seed: int, tid: int, chunk: int = 0) -> np.random.Generator:
    return np.random.default_rng([seed, tid, chunk])


def _normal(seed: int, tid: int, shape, std: float, chunk: int = 0) -> np.ndarray:
    a = _rng(seed, tid, chunk).standard_normal(shape, dtype=np.float32)
    a *= np.float32(std)
    return a


def _to_dtype(a: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(a)
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def _stacked_normal(seed, tid, n, shape, std, dtype, workers) -> torch.Tensor:
    out = torch.empty((n,) + tuple(shape), dtype=torch.bfloat16 if dtype == "bf16" else torch.float32)

    def one(e):
        out[e].copy_(_to_dtype(_normal(seed, tid, shape, std, chunk=e), dtype))

    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(one, range(n)))
    return out


def quantise_logits(logits: np.ndarray, step: float = 0.25) -> np.ndarray:
    return (np.round(logits / step) * step).astype(np.float32)


@dataclass
class LayerInputs:
    cfg: LayerConfig
    seed: int
    x: torch.Tensor                 # [T, H]    f32 or bf16 (CPU)
    logits: np.ndarray              # [T, n]    f32
    mask: np.ndarray                # [n, n]    u8
    w_gate: torch.Tensor            # [n, F, H]
    w_up: torch.Tensor              # [n, F, H]
    w_down: torch.Tensor            # [n, H, F]
    s_gate: Optional[torch.Tensor] = None   # [F_s, H]
    s_up: Optional[torch.Tensor] = None     # [F_s, H]
    s_down: Optional[torch.Tensor] = None   # [H, F_s]


def _logits(cfg: LayerConfig, seed: int, x: torch.Tensor) -> np.ndarray:
    kind = cfg.logits.split("+")
    base, extra = kind[0], kind[1:]
    T, n = cfg.T, cfg.n
    if base == "router":
        wr = _normal(seed, TID_ROUTER, (n, cfg.H), cfg.w_std).astype(np.float64)
        l = (x.to(torch.float64).numpy() @ wr.T).astype(np.float32)
    elif base == "normal":
        l = _normal(seed, TID_LOGITS, (T, n), 1.0)
    elif base == "normal_bias":
        l = _normal(seed, TID_LOGITS, (T, n), 1.0) + _normal(seed, TID_BIAS, (n,), cfg.bias_std)[None, :]
    elif base == "zipf":
        rank = _rng(seed, TID_RANK).permutation(n) + 1
        prior = (-cfg.zipf_s * np.log(rank.astype(np.float64))).astype(np.float32)
        l = _normal(seed, TID_LOGITS, (T, n), 1.0) + prior[None, :]
    else:
        raise ValueError(cfg.logits)
    l = np.ascontiguousarray(l, dtype=np.float32)
    if "ties" in extra:
        l = quantise_logits(l)
    if "one_expert" in extra:
        l[:, 0] += np.float32(100.0)
    return l


def make_mask(n: int, density: float, seed: int) -> np.ndarray:
    m = (_rng(seed, TID_MASK).random((n, n)) < density).astype(np.uint8)
    np.fill_diagonal(m, 1)
    return m


def make_inputs(cfg: LayerConfig, seed: int = 0, workers: Optional[int] = None,
                with_weights: bool = True) -> LayerInputs:
    """Draw every tensor of one layer; all on the host."""
    workers = workers or min(16, os.cpu_count() or 1)
    x = _to_dtype(_normal(seed, TID_X, (cfg.T, cfg.H), cfg.x_std), cfg.dtype)
    logits = _logits(cfg, seed, x)
    mask = make_mask(cfg.n, cfg.density, seed)
    inp = LayerInputs(cfg, seed, x, logits, mask, None, None, None)
    if not with_weights:
        return inp
    inp.w_gate = _stacked_normal(seed, TID_WG, cfg.n, (cfg.F, cfg.H), cfg.w_std, cfg.dtype, workers)
    inp.w_up = _stacked_normal(seed, TID_WU, cfg.n, (cfg.F, cfg.H), cfg.w_std, cfg.dtype, workers)
    inp.w_down = _stacked_normal(seed, TID_WD, cfg.n, (cfg.H, cfg.F), cfg.w_std, cfg.dtype, workers)
    if cfg.shared_F:
        Fs = cfg.shared_F
        inp.s_gate = _to_dtype(_normal(seed, TID_SWG, (Fs, cfg.H), cfg.w_std), cfg.dtype)
        inp.s_up = _to_dtype(_normal(seed, TID_SWU, (Fs, cfg.H), cfg.w_std), cfg.dtype)
        inp.s_down = _to_dtype(_normal(seed, TID_SWD, (cfg.H, Fs), cfg.w_std), cfg.dtype)
    return inp


@dataclass
class ScoredInputs:
    g_tgt: np.ndarray               # [T, n]    f32
    bias: np.ndarray                # [n, n]    f32
    lam: float


def make_scored_inputs(cfg: LayerConfig, seed: int = 0) -> ScoredInputs:
    """Target prior and compatibility bias of the scored router (host arrays)."""
    g_tgt = _normal(seed, TID_GTGT, (cfg.T, cfg.n), 1.0)
    b = _rng(seed, TID_COMPAT).uniform(-COMPAT_NOISE, COMPAT_NOISE, (cfg.n, cfg.n))
    bias = (np.float64(COMPAT_C) + b).astype(np.float32)
    np.fill_diagonal(bias, 0.0)
    return ScoredInputs(np.ascontiguousarray(g_tgt), np.ascontiguousarray(bias), SCORED_LAMBDA)


def make_router_weights(cfg: LayerConfig, seed: int = 0) -> torch.Tensor:
    """Router matrix W_r [n, H], N(0, w_std), in the layer's dtype (the tiny workload's
    logits are x W_r^T of this same matrix)."""
    return _to_dtype(_normal(seed, TID_ROUTER, (cfg.n, cfg.H), cfg.w_std), cfg.dtype)
