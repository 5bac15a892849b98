"""Scored compositional routing on the HIP path against the CPU oracle, through the C ABI
(needs an MI355X).

Integers (active-pair layout, selected paths, source / target groups, path bits, both
dispatch layouts) must match bit for bit, and so must the float32 path scores (both sides
form them with one fused multiply-add). Path weights: 1e-5 relative (absolute FLT_MIN).
Layer outputs: the same contract as the vanilla-compatible layer.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_01024_amd as pcm
from paper_2609_01024_amd import binding
from workloads import CONFIGS, make_inputs, make_scored_inputs, scaled, stress_config

from test_gpu_parity import SMALL, assert_y_close, block_tokens, dev, poison

pytestmark = pytest.mark.gpu
DEV = "cuda"
FLT_MIN = float(np.finfo(np.float32).tiny)


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def run_route(gb, gt, lam, bias, mask, K):
    layout = pcm.pcm_path_layout_build(t(mask), t(bias))
    p = pcm.pcm_route_scored(t(gb), t(gt), lam, layout, K)
    torch.cuda.synchronize()
    return layout, p


def check_route(gb, gt, lam, bias, mask, K, what=""):
    """Every integer output bit-exact against the oracle; weights to 1e-5."""
    n = mask.shape[0]
    layout, p = run_route(gb, gt, lam, bias, mask, K)
    src, tgt, sc, beta = oracle.route_scored(gb, gt, lam, bias, mask, K)
    sel = p.sel_pair.cpu().numpy()
    assert np.array_equal(sel, src * n + tgt), f"selected paths {what}"
    pos0 = lambda a: (a + np.float32(0.0)).view(np.uint32)   # -0 and +0 are the same score
    assert np.array_equal(pos0(p.sel_score.cpu().numpy()), pos0(sc)), f"scores {what}"
    n_src, srcs, n_tgt, tgts, bits, bg = oracle.group_scored(src, tgt, beta)
    assert np.array_equal(p.n_src.cpu().numpy(), n_src), f"n_src {what}"
    assert np.array_equal(p.src_expert.cpu().numpy(), srcs), f"src_expert {what}"
    assert np.array_equal(p.n_tgt.cpu().numpy(), n_tgt), f"n_tgt {what}"
    assert np.array_equal(p.tgt_expert.cpu().numpy(), tgts), f"tgt_expert {what}"
    assert np.array_equal(p.path_bits.cpu().numpy().view(np.uint64), bits), f"path bits {what}"
    np.testing.assert_allclose(p.beta.cpu().numpy(), bg, rtol=1e-5, atol=FLT_MIN, err_msg=what)
    for side, ids, cnt in (("src", srcs, n_src), ("tgt", tgts, n_tgt)):
        off, rt, rs, ro = oracle.permute_var(ids, cnt, n)
        R = int(cnt.sum())
        assert np.array_equal(getattr(p, f"{side}_offsets").cpu().numpy(), off), f"{side} offsets {what}"
        assert np.array_equal(getattr(p, f"{side}_row_token").cpu().numpy()[:R], rt), f"{side} row_token"
        assert np.array_equal(getattr(p, f"{side}_row_slot").cpu().numpy()[:R], rs), f"{side} row_slot"
        assert np.array_equal(getattr(p, f"{side}_row_of").cpu().numpy(), ro), f"{side} row_of {what}"
    return layout, p


def scored_inputs(cfg, seed):
    inp = make_inputs(cfg, seed=seed)
    s = make_scored_inputs(cfg, seed=seed)
    return inp, s


def run_layer(d, g_tgt, lam, bias, K, tuning=None, plan_out=None):
    T, H = d["x"].shape
    n, F, _ = d["w_gate"].shape
    plan = pcm.ScoredLayerPlan(T, H, F, n, K, d["x"].dtype, DEV,
                               d["shared"][0].shape[0] if "shared" in d else 0)
    poison(plan)
    plan.build_layout(d["mask"], t(bias))
    y = plan.forward(d["x"], d["logits"], t(g_tgt), lam, d["w_gate"], d["w_up"], d["w_down"],
                     d.get("shared"), tuning=tuning)
    torch.cuda.synchronize()
    if plan_out is not None:
        plan_out.append(plan)
    return y.cpu().numpy()


def oracle_layer(inp, s, tokens=None):
    c = inp.cfg
    y = oracle.layer_scored(inp.x, inp.logits, s.g_tgt, s.lam, s.bias, inp.mask, inp.w_gate,
                            inp.w_up, inp.w_down, c.k, tokens=tokens)
    if inp.s_gate is not None:
        y = y + oracle.dense_swiglu(inp.x, inp.s_gate, inp.s_up, inp.s_down, tokens=tokens)
    return y


# ------------------------------------------------------------------ layout, route
@pytest.mark.parametrize("n,d", [(1, 0.0), (3, 1.0), (8, 0.5), (64, 0.25), (256, 0.2), (256, 0.0)])
def test_layout(n, d):
    rng = np.random.default_rng(n)
    mask = (rng.random((n, n)) < d).astype(np.uint8)
    mask[np.arange(n), np.arange(n)] = 0        # the diagonal is active regardless
    bias = rng.standard_normal((n, n)).astype(np.float32)
    lay = pcm.pcm_path_layout_build(t(mask), t(bias))
    torch.cuda.synchronize()
    act = (mask != 0) | np.eye(n, dtype=bool)
    flat = np.flatnonzero(act)
    cnt = int(lay.count.cpu()[0])
    assert cnt == flat.size
    pr = lay.pair.cpu().numpy()[:cnt].view(np.uint32)
    assert np.array_equal((pr >> 16) * n + (pr & 0xFFFF), flat)
    assert np.array_equal(lay.bias.cpu().numpy()[:cnt], bias.ravel()[flat])


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_route_scored_full_size(name):
    cfg = CONFIGS[name]
    say(f"scored route {name}")
    inp, s = scored_inputs(cfg, 0)
    check_route(inp.logits, s.g_tgt, s.lam, s.bias, inp.mask, cfg.k, name)


@pytest.mark.parametrize("T,n,K,d,lam", [(1, 1, 1, 0.0, 0.5), (5, 4, 4, 1.0, 2.0), (256, 8, 2, 0.5, 0.5),
                                         (257, 64, 8, 0.25, 0.0), (1025, 64, 8, 0.3, 1.0),
                                         (700, 256, 8, 0.2, 0.5), (64, 8, 8, 1.0, 64.0),
                                         # weights that are not powers of two: lambda * g_tgt is
                                         # rounded inside the fused multiply-add
                                         (513, 64, 8, 0.3, 0.3), (300, 16, 6, 0.6, 0.7),
                                         (1100, 60, 4, 0.3, -1.25)])
def test_route_scored_shapes(T, n, K, d, lam):
    rng = np.random.default_rng(T + n)
    gb = rng.standard_normal((T, n)).astype(np.float32)
    gt = rng.standard_normal((T, n)).astype(np.float32)
    mask = (rng.random((n, n)) < d).astype(np.uint8)
    bias = (-1.0 + rng.uniform(-0.5, 0.5, (n, n))).astype(np.float32)
    np.fill_diagonal(bias, 0.0)
    check_route(gb, gt, lam, bias, mask, K, f"T={T} n={n} K={K}")


def test_route_scored_ties_and_signed_zeros():
    """Quantised inputs make exact score ties common; equal scores go to the lower
    flattened index, and -0 equals +0."""
    rng = np.random.default_rng(5)
    T, n, K = 300, 16, 6
    q = lambda a: (np.round(a * 2) / 2).astype(np.float32)
    gb, gt = q(rng.standard_normal((T, n))), q(rng.standard_normal((T, n)))
    bias = q(-1.0 + rng.uniform(-1, 1, (n, n)))
    np.fill_diagonal(bias, 0.0)
    mask = (rng.random((n, n)) < 0.6).astype(np.uint8)
    check_route(gb, gt, 0.5, bias, mask, K, "ties")
    z = np.zeros((2, 4), np.float32)
    z[0] = [-0.0, 0.0, -0.0, 0.0]
    zb = np.zeros((4, 4), np.float32)
    zb[0, 1] = -0.0
    _, p = check_route(z, -z, 1.0, zb, np.ones((4, 4), np.uint8), 4, "signed zeros")
    assert list(p.sel_pair.cpu().numpy()[0]) == [0, 1, 2, 3]


def test_route_scored_diagonal_is_vanilla_topk():
    """mask = I and no target prior: the selection is the vanilla top-K and the weights
    its renormalised softmax (the vanilla-compatible router's output)."""
    cfg = CONFIGS["olmoe"]
    inp, s = scored_inputs(cfg, 1)
    eye = np.eye(cfg.n, dtype=np.uint8)
    _, p = check_route(inp.logits, s.g_tgt, 0.0, s.bias, eye, cfg.k, "diag")
    ids, w = pcm.pcm_route(t(inp.logits), cfg.k)
    torch.cuda.synchronize()
    ids = ids.cpu().numpy()
    assert np.array_equal(p.sel_pair.cpu().numpy(), ids * cfg.n + ids)


# ------------------------------------------------------------------ whole layer
@pytest.mark.parametrize("tile", ["auto", "S", "M", "L"])
@pytest.mark.parametrize("name", sorted(SMALL))
def test_scored_layer_small(name, tile):
    tuning = pcm.Tuning(tile=tile) if tile != "auto" else None
    cfg = SMALL[name]
    say(f"scored layer {name} tile {tile}")
    inp, s = scored_inputs(cfg, 1)
    d = dev(inp)
    y = run_layer(d, s.g_tgt, s.lam, s.bias, cfg.k, tuning=tuning)
    assert_y_close(y, oracle_layer(inp, s), cfg.dtype, f"scored {name}/{tile}")


@pytest.mark.parametrize("lam", [0.3, 0.7, -1.25])
def test_scored_layer_general_lambda(lam):
    """The whole scored layer at target-prior weights that are not powers of two."""
    cfg = SMALL["olmoe_s"]
    inp, s = scored_inputs(cfg, 4)
    d = dev(inp)
    check_route(inp.logits, s.g_tgt, lam, s.bias, inp.mask, cfg.k, f"lambda {lam}")
    y = run_layer(d, s.g_tgt, lam, s.bias, cfg.k)
    ref = oracle.layer_scored(inp.x, inp.logits, s.g_tgt, lam, s.bias, inp.mask, inp.w_gate,
                              inp.w_up, inp.w_down, cfg.k)
    assert_y_close(y, ref, cfg.dtype, f"scored lambda {lam}")


def test_scored_layer_single_source_paths():
    """Zero bias, full mask, no target prior: one source feeds K targets per token."""
    cfg = scaled(SMALL["olmoe_s"], density=1.0, T=400, name="single_source")
    inp, s = scored_inputs(cfg, 2)
    zero = np.zeros((cfg.n, cfg.n), np.float32)
    d = dev(inp)
    y = run_layer(d, s.g_tgt, 0.0, zero, cfg.k)
    ref = oracle.layer_scored(inp.x, inp.logits, s.g_tgt, 0.0, zero, inp.mask, inp.w_gate, inp.w_up,
                              inp.w_down, cfg.k)
    assert_y_close(y, ref, cfg.dtype, "single source")


def test_scored_layer_edge_cases():
    for cfg in (scaled(SMALL["olmoe_s"], n=8, k=8, density=1.0, T=300, name="K_eq_n"),
                scaled(SMALL["olmoe_s"], n=1, k=1, T=333, name="n1"),
                scaled(SMALL["olmoe_s"], k=1, T=500, name="K1"),
                stress_config("one_expert", scaled(SMALL["olmoe_s"], T=700, name="one"))):
        inp, s = scored_inputs(cfg, 5)
        y = run_layer(dev(inp), s.g_tgt, s.lam, s.bias, cfg.k)
        assert_y_close(y, oracle_layer(inp, s), cfg.dtype, cfg.name)


def test_scored_layer_diagonal_equals_vanilla_layer():
    """mask = I and lambda = 0: the scored layer's output equals the vanilla-compatible
    layer's on the same inputs (same kernels, same rows, same order)."""
    cfg = scaled(SMALL["mixtral_s"], density=0.0, name="diag")
    inp, s = scored_inputs(cfg, 3)
    d = dev(inp)
    y_s = run_layer(d, s.g_tgt, 0.0, s.bias, cfg.k)
    y_v = pcm.layer_forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"],
                            cfg.k)
    torch.cuda.synchronize()
    y_v = y_v.cpu().numpy()
    # the two routers' weights may differ in the last bit (their own softmax code), which
    # can move a float16 rounding of z; the combine also sums targets in another order
    assert np.abs(y_s - y_v).max() <= 1e-3 * np.abs(y_v).max()


def test_scored_layer_is_deterministic():
    cfg = SMALL["olmoe_s"]
    inp, s = scored_inputs(cfg, 7)
    d = dev(inp)
    a = run_layer(d, s.g_tgt, s.lam, s.bias, cfg.k)
    b = run_layer(d, s.g_tgt, s.lam, s.bias, cfg.k)
    assert np.array_equal(a, b)


@pytest.mark.slow
@pytest.mark.parametrize("name", ["tiny", "mixtral", "olmoe", "finegrained_shared", "decode"])
def test_scored_layer_full_size(name):
    """The scored layer at the workload's size with every buffer NaN first; y against the
    oracle on the tokens of the first and last row of every 256-row block of both dispatch
    layouts (the expansion's and the projection's M tiles) plus a random sample."""
    cfg = CONFIGS[name]
    say(f"scored full-size {name}: inputs")
    inp, s = scored_inputs(cfg, 0)
    d = dev(inp)
    say(f"scored full-size {name}: layer")
    plans = []
    y = run_layer(d, s.g_tgt, s.lam, s.bias, cfg.k, plan_out=plans)
    assert np.isfinite(y).all(), f"{name}: unwritten or non-finite outputs"
    p = plans[0].paths
    rng = np.random.default_rng(12)
    nsample = cfg.T if cfg.T <= 64 else 24
    tokens = np.unique(np.concatenate([
        [0, cfg.T - 1], rng.choice(cfg.T, nsample, replace=False),
        block_tokens(p.src_offsets.cpu().numpy(), p.src_row_token.cpu().numpy()),
        block_tokens(p.tgt_offsets.cpu().numpy(), p.tgt_row_token.cpu().numpy())]))
    say(f"scored full-size {name}: oracle on {tokens.size} tokens")
    assert_y_close(y[tokens], oracle_layer(inp, s, tokens), cfg.dtype, name)


