"""Projection weights widened once to float16 (PCM_BF16_F16DOWN, pcm_widen_f16) against
the bf16 weights they come from, through the C ABI (needs an MI355X).

pcm_widen_f16 must give, bit for bit, the float16 rounding (to nearest even) of every bf16
value, which numpy's float32 -> float16 conversion defines independently. The projection
kernels widen each bf16 fragment with the same rounding, so every call that takes projection
weights must give the same output bits with the widened copy as with the bf16 weights: the
large tiles (with and without the K split, every work order), the medium tiles, the
streaming kernels at every ring depth, the shared expert's accumulating projection, the
per-path baseline, the scored router's projection and the allocation-free call.
"""
import sys

import numpy as np
import pytest
import torch

import paper_2609_01024_amd as pcm
from workloads import make_inputs

from test_gpu_parity import SMALL, dev, poison
from test_gpu_scored import run_layer as run_scored_layer, scored_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def f16_reference(bits_bf16: np.ndarray) -> np.ndarray:
    """float16 bits of each bf16 value, rounded to nearest even (numpy's conversion)."""
    f32 = (bits_bf16.astype(np.uint32) << 16).view(np.float32)
    with np.errstate(over="ignore"):
        return f32.astype(np.float16).view(np.uint16)


def special_bf16(rng, count):
    """bf16 bit patterns over the whole finite range, denser where float16 rounds: float16's
    subnormal range, its smallest normals, its largest values and past them, signed zeros."""
    mags = np.concatenate([
        rng.uniform(-30, -14, count // 4),     # float16 subnormals and below
        rng.uniform(-14, 15.9999, count // 4),  # float16 normals
        rng.uniform(15.9, 16.1, count // 8),    # around 65504 and the overflow to inf
        rng.uniform(-126, 127, count // 8),     # the rest of bf16's range
    ])
    v = (2.0 ** mags) * rng.choice([-1.0, 1.0], mags.size)
    bits = (v.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    extra = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x387F, 0x3880, 0x477F, 0x4780,
                      0x7F7F, 0xFF7F, 0x3380, 0x3381, 0x33C0, 0x33C1], np.uint16)
    out = np.concatenate([bits, extra])
    rng.shuffle(out)
    return out


@pytest.mark.parametrize("count", [1, 7, 8, 9, 64, 1000, 4099, 1 << 20])
def test_widen_f16_rounds_to_nearest_even(count):
    rng = np.random.default_rng(count)
    bits = special_bf16(rng, 2 * count + 64)[:count]
    src = torch.from_numpy(bits.view(np.int16)).to(DEV).view(torch.bfloat16)
    out = torch.full((count,), -1, dtype=torch.int16, device=DEV).view(torch.float16)
    pcm.pcm_widen_f16(src, out=out)
    torch.cuda.synchronize()
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    ref = f16_reference(bits)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, [(hex(bits[i]), hex(got[i]), hex(ref[i])) for i in bad[:8]]


def test_widen_f16_zero_count_and_validation():
    w = torch.zeros((0,), dtype=torch.bfloat16, device=DEV)
    assert pcm.pcm_widen_f16(w).numel() == 0
    with pytest.raises(TypeError):
        pcm.pcm_widen_f16(torch.zeros((8,), dtype=torch.float32, device=DEV))


def widened(d):
    """The inputs of dev() with every projection weight widened to float16."""
    h = dict(d)
    h["w_down"] = pcm.pcm_widen_f16(d["w_down"])
    if "shared" in d:
        g, u, dn = d["shared"]
        h["shared"] = (g, u, pcm.pcm_widen_f16(dn))
    return h


def layer_bits(cfg, d, tuning=None):
    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, torch.bfloat16, DEV, cfg.shared_F)
    poison(plan)
    y = plan.forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"],
                     d.get("shared"), tuning=tuning)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("name,tuning", [
    ("mixtral_s", None), ("olmoe_s", None), ("fine_s", None), ("decode_s", None),
    ("splitk_s", None), ("shortk_s", None),
    ("olmoe_s", dict(tile="M")), ("fine_s", dict(tile="M")),
    ("mixtral_s", dict(tile="L", order_down=0)), ("fine_s", dict(tile="L", order_down=1)),
    ("splitk_s", dict(tile="L", order_down=2, em_window=3)),
    ("decode_s", dict(tile="S", stream_depth=0)), ("decode_s", dict(tile="S", stream_depth=3)),
    ("olmoe_s", dict(tile="S", stream_depth=2)), ("fine_s", dict(tile="S", stream_depth=6)),
])
def test_layer_with_widened_weights_is_bit_identical(name, tuning):
    cfg = SMALL[name]
    say(f"widened projection weights: {name} {tuning}")
    d = dev(make_inputs(cfg, seed=31))
    t = pcm.Tuning(**tuning) if tuning else None
    base = layer_bits(cfg, d, t)
    assert np.isfinite(base).all()
    y = layer_bits(cfg, widened(d), t)
    assert np.array_equal(y.view(np.uint32), base.view(np.uint32)), f"{name} {tuning}"


def test_dense_swiglu_accumulate_with_widened_weights():
    cfg = SMALL["fine_s"]
    d = dev(make_inputs(cfg, seed=32))
    g, u, dn = d["shared"]
    base = torch.randn((cfg.T, cfg.H), device=DEV)
    for tile in ("L", "M", "S"):
        t = pcm.Tuning(tile=tile)
        a = pcm.pcm_dense_swiglu(d["x"], g, u, dn, y=base.clone(), accumulate=True, tuning=t)
        b = pcm.pcm_dense_swiglu(d["x"], g, u, pcm.pcm_widen_f16(dn), y=base.clone(),
                                 accumulate=True, tuning=t)
        torch.cuda.synchronize()
        assert torch.equal(a.view(torch.int32), b.view(torch.int32)), tile


@pytest.mark.parametrize("reuse", [True, False])
def test_per_path_baseline_with_widened_weights(reuse):
    cfg = SMALL["olmoe_s"]
    d = dev(make_inputs(cfg, seed=33))
    ids, w = pcm.pcm_route(d["logits"], cfg.k)
    paths = pcm.pcm_build_paths(ids, w, d["mask"])
    a = pcm.pcm_layer_per_path(d["x"], d["w_gate"], d["w_up"], d["w_down"], paths, reuse=reuse)
    b = pcm.pcm_layer_per_path(d["x"], d["w_gate"], d["w_up"], pcm.pcm_widen_f16(d["w_down"]),
                               paths, reuse=reuse)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


@pytest.mark.parametrize("name", ["olmoe_s", "fine_s", "decode_s"])
def test_scored_layer_with_widened_weights(name):
    cfg = SMALL[name]
    inp, s = scored_inputs(cfg, 34)
    d = dev(inp)
    a = run_scored_layer(d, s.g_tgt, s.lam, s.bias, cfg.k)
    b = run_scored_layer(widened(d), s.g_tgt, s.lam, s.bias, cfg.k)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_noalloc_with_widened_weights():
    cfg = SMALL["decode_s"]
    d = dev(make_inputs(cfg, seed=35))
    ids, w = pcm.pcm_route(d["logits"], cfg.k)
    paths = pcm.pcm_build_paths(ids, w, d["mask"])
    u = pcm.pcm_expand(d["x"], d["w_gate"], d["w_up"], paths)
    a = pcm.pcm_project_combine(u, d["w_down"], paths)
    b = pcm.pcm_project_combine_noalloc(u, pcm.pcm_widen_f16(d["w_down"]), paths)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
