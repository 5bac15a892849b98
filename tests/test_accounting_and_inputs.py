"""FLOP accounting against the paper's cost split, and the seeded input generator."""
import hashlib
import os
from fractions import Fraction

import numpy as np
import pytest

from paper_2609_01024_amd import accounting as acc
from workloads import CONFIGS, make_inputs, scaled, stress_config

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_flop_fractions.txt")


def _golden():
    out = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, num, den = line.split()
        out[name] = Fraction(int(num), int(den))
    return out


def test_flop_split_matches_paper():
    g = _golden()
    H, F = 4096, 14336                      # a Mixtral-8x7B expert
    e = acc.expert_flops(H, F)
    assert Fraction(acc.expansion_flops_per_row(H, F), e) == g["expansion_fraction"]
    top2 = 2 * e                             # two experts per token
    assert Fraction(acc.expansion_flops_per_row(H, F), top2) == g["top2_expansion_reuse_saving"]
    assert Fraction(acc.projection_flops_per_row(H, F), top2) == g["top2_projection_reuse_saving"]


def test_gemm_flops_counts_rows_once():
    f = acc.gemm_flops(R=8192, H=4096, F=14336)
    assert f["total"] == 6 * 8192 * 4096 * 14336
    f = acc.gemm_flops(R=65536, H=2048, F=1408, T=16384, shared_F=5632)
    assert f["shared_expand"] == 4 * 16384 * 2048 * 5632


def _digest(inp):
    h = hashlib.sha256()
    for t in (inp.x, inp.w_gate, inp.w_up, inp.w_down):
        h.update(t.contiguous().float().numpy().tobytes())
    h.update(inp.logits.tobytes())
    h.update(inp.mask.tobytes())
    return h.hexdigest()


def test_generator_is_deterministic_and_worker_independent():
    cfg = scaled(CONFIGS["olmoe"], T=64, H=128, F=64)
    a = make_inputs(cfg, seed=3, workers=1)
    b = make_inputs(cfg, seed=3, workers=4)
    c = make_inputs(cfg, seed=4, workers=4)
    assert _digest(a) == _digest(b)
    assert _digest(a) != _digest(c)


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_generator_shapes_and_structure(name):
    cfg = CONFIGS[name]
    small = scaled(cfg, T=min(cfg.T, 256), H=128, F=64, shared_F=64 if cfg.shared_F else 0)
    inp = make_inputs(small, seed=0)
    assert inp.x.shape == (small.T, small.H)
    assert inp.w_gate.shape == (small.n, small.F, small.H)
    assert inp.w_down.shape == (small.n, small.H, small.F)
    assert inp.logits.shape == (small.T, small.n) and inp.logits.dtype == np.float32
    assert np.all(np.diag(inp.mask) == 1)
    off = inp.mask[~np.eye(small.n, dtype=bool)]
    if small.n >= 8:
        assert abs(off.mean() - small.density) < 0.2
    w = inp.w_gate.float().numpy()
    assert abs(w.std() - small.w_std) < 0.1 * small.w_std
    assert str(inp.x.dtype) == ("torch.bfloat16" if cfg.dtype == "bf16" else "torch.float32")


def test_stress_inputs():
    base = scaled(CONFIGS["olmoe"], T=128, H=64, F=64)
    ties = make_inputs(stress_config("ties", base), with_weights=False)
    assert np.all(np.round(ties.logits * 4) == ties.logits * 4)
    one = make_inputs(stress_config("one_expert", base), with_weights=False)
    assert np.all(np.argmax(one.logits, axis=1) == 0)
