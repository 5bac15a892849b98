"""HIP path against the CPU oracle, through the C ABI (needs an MI355X).

Integers (top-k ids, path bits, the dispatch layout) must match bit for bit.
Floating point: router weights and path weights to 1e-5 relative (absolute
FLT_MIN below float32's normal range); layer outputs
elementwise within |d| <= 1e-2 + 2e-2 |ref| and, tighter, a relative Frobenius
error <= 5e-3 for bfloat16 layers (two roundings to bfloat16, of U and of the
mixed z, each <= 2^-9 relative) and max |d| <= 1e-4 max |ref| for float32 layers.
"""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_01024_amd as pcm
from workloads import CONFIGS, make_inputs, scaled, stress_config

pytestmark = pytest.mark.gpu
DEV = "cuda"
FLT_MIN = float(np.finfo(np.float32).tiny)


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


# ---------------------------------------------------------------------- helpers
def dev(inp):
    d = dict(x=inp.x.to(DEV), logits=torch.from_numpy(inp.logits).to(DEV),
             mask=torch.from_numpy(inp.mask).to(DEV))
    if inp.w_gate is not None:
        d.update(w_gate=inp.w_gate.to(DEV), w_up=inp.w_up.to(DEV), w_down=inp.w_down.to(DEV))
    if inp.s_gate is not None:
        d["shared"] = (inp.s_gate.to(DEV), inp.s_up.to(DEV), inp.s_down.to(DEV))
    return d


def assert_y_close(y, ref, dtype, what=""):
    y = np.asarray(y, np.float64)
    d = np.abs(y - ref)
    bound = 1e-2 + 2e-2 * np.abs(ref)
    bad = d > bound
    assert not bad.any(), f"{what}: {bad.sum()} elements outside |d| <= 1e-2 + 2e-2|ref| (max d {d.max():.3e})"
    if dtype == "bf16":
        rel = np.linalg.norm(d) / max(np.linalg.norm(ref), 1e-30)
        assert rel <= 5e-3, f"{what}: relative Frobenius error {rel:.3e} > 5e-3"
    else:
        m = d.max() / max(np.abs(ref).max(), 1e-30)
        assert m <= 1e-4, f"{what}: max |d| / max |ref| = {m:.3e} > 1e-4"
    return d


def check_route(logits_np, k):
    ids_ref, w_ref = oracle.route(logits_np, k)
    ids, w = pcm.pcm_route(torch.from_numpy(logits_np).to(DEV), k)
    torch.cuda.synchronize()
    assert np.array_equal(ids.cpu().numpy(), ids_ref), "top-k ids differ"
    # float32 carries no relative precision below its smallest normal number
    np.testing.assert_allclose(w.cpu().numpy(), w_ref, rtol=1e-5, atol=FLT_MIN)
    return ids, w


def check_paths(ids, w, mask_np, n, beta_mode=0):
    """GPU path table from the GPU route outputs vs the oracle on the same inputs."""
    ids_np = ids.cpu().numpy()
    w_np = w.cpu().numpy().astype(np.float64)
    bits_ref, beta_ref = oracle.paths(ids_np, w_np, mask_np, beta_mode)
    off_ref, rt_ref, rs_ref, ro_ref = oracle.permute(ids_np, n)
    p = pcm.pcm_build_paths(ids, w, torch.from_numpy(mask_np).to(DEV), beta_mode)
    torch.cuda.synchronize()
    assert np.array_equal(p.path_bits.cpu().numpy().view(np.uint64), bits_ref), "path bits differ"
    np.testing.assert_allclose(p.beta.cpu().numpy(), beta_ref, rtol=1e-5, atol=FLT_MIN)
    assert np.array_equal(p.expert_offsets.cpu().numpy(), off_ref), "expert offsets differ"
    assert np.array_equal(p.row_token.cpu().numpy(), rt_ref), "row_token differs"
    assert np.array_equal(p.row_slot.cpu().numpy(), rs_ref), "row_slot differs"
    assert np.array_equal(p.row_of.cpu().numpy(), ro_ref), "row_of differs"
    return p


def run_layer(d, k, beta_mode=0):
    y = pcm.layer_forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"], k,
                          beta_mode=beta_mode, shared=d.get("shared"))
    torch.cuda.synchronize()
    return y.cpu().numpy()


# ------------------------------------------------------------------------ route
@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_route_full_size(name):
    cfg = CONFIGS[name]
    say(f"route {name}")
    inp = make_inputs(cfg, with_weights=False)
    check_route(inp.logits, cfg.k)


@pytest.mark.parametrize("kind", ["ties", "one_expert"])
def test_route_stress(kind):
    cfg = stress_config(kind, CONFIGS["olmoe"])
    inp = make_inputs(cfg, with_weights=False)
    check_route(inp.logits, cfg.k)


def test_route_shapes_and_signed_zeros():
    rng = np.random.default_rng(5)
    for n in (1, 2, 3, 63, 64, 65, 128, 130, 200, 256):
        for k in sorted({1, min(n, 2), min(n, 5), min(n, 8)}):
            l = rng.standard_normal((77, n)).astype(np.float32)
            check_route(l, k)
            check_route((np.round(l) / 2).astype(np.float32), k)   # heavy ties
    l = np.array([[-0.0, 0.0, 0.0, -0.0, -1.0, 2.0, 2.0]], np.float32)
    ids, _ = check_route(l, 6)
    assert list(ids.cpu().numpy()[0]) == [5, 6, 0, 1, 2, 3]


# ------------------------------------------------------------------ path table
@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_build_paths_full_size(name):
    cfg = CONFIGS[name]
    say(f"paths {name}")
    inp = make_inputs(cfg, with_weights=False)
    ids, w = pcm.pcm_route(torch.from_numpy(inp.logits).to(DEV), cfg.k)
    p1 = check_paths(ids, w, inp.mask, cfg.n)
    p2 = pcm.pcm_build_paths(ids, w, torch.from_numpy(inp.mask).to(DEV))
    torch.cuda.synchronize()
    for f in ("path_bits", "beta", "expert_offsets", "row_token", "row_slot", "row_of"):
        assert torch.equal(getattr(p1, f), getattr(p2, f)), f"{f} differs between runs"


@pytest.mark.parametrize("beta_mode", [0, 1, 2])
@pytest.mark.parametrize("T,n,k", [(1, 1, 1), (5, 4, 4), (256, 8, 2), (257, 64, 8), (1025, 64, 8),
                                   (3000, 256, 8), (4097, 60, 4)])
def test_build_paths_shapes(T, n, k, beta_mode):
    rng = np.random.default_rng(T + n)
    l = rng.standard_normal((T, n)).astype(np.float32)
    mask = (rng.random((n, n)) < 0.4).astype(np.uint8)
    if n > 1:
        mask[0, 0] = 0  # a zero diagonal entry is treated as 1
    ids, w = pcm.pcm_route(torch.from_numpy(l).to(DEV), k)
    check_paths(ids, w, mask, n, beta_mode)


def test_build_paths_all_on_one_expert():
    cfg = stress_config("one_expert", scaled(CONFIGS["olmoe"], T=2500))
    inp = make_inputs(cfg, with_weights=False)
    ids, w = pcm.pcm_route(torch.from_numpy(inp.logits).to(DEV), cfg.k)
    p = check_paths(ids, w, inp.mask, cfg.n)
    assert int(p.expert_offsets[1] - p.expert_offsets[0]) == cfg.T


# ------------------------------------------------------------------ whole layer
SMALL = {
    "tiny": CONFIGS["tiny"],
    "mixtral_s": scaled(CONFIGS["mixtral"], T=1500, H=320, F=448, name="mixtral_s"),
    "olmoe_s": scaled(CONFIGS["olmoe"], T=1100, H=256, F=192, name="olmoe_s"),
    "fine_s": scaled(CONFIGS["finegrained_shared"], T=1200, H=192, F=320, shared_F=448,
                     name="fine_s"),
    "decode_s": scaled(CONFIGS["decode"], H=512, F=256, name="decode_s"),
    # long F and few output tiles: the large-tile projection splits K in two slices
    "splitk_s": scaled(CONFIGS["mixtral"], T=300, H=256, F=4096, n=4, name="splitk_s"),
    # one and two 64-wide K stages (H = 64, F = 128): the pipelines' start-up loads past the
    # last stage are clamped re-reads
    "shortk_s": scaled(CONFIGS["mixtral"], T=700, H=64, F=128, n=4, name="shortk_s"),
}


@pytest.mark.parametrize("tile", ["auto", "S", "M", "L"])
@pytest.mark.parametrize("name", sorted(SMALL))
def test_layer_small(name, tile, monkeypatch):
    if tile != "auto":
        monkeypatch.setenv("PCM_GEMM_TILE", tile)
    cfg = SMALL[name]
    say(f"layer {name} tile {tile}")
    inp = make_inputs(cfg, seed=1)
    d = dev(inp)
    y = run_layer(d, cfg.k)
    ref = oracle.layer_inputs(inp)
    assert_y_close(y, ref, cfg.dtype, f"{name}/{tile}")


@pytest.mark.parametrize("T", [60, 64, 68])
def test_layer_tile_policy_boundary(T):
    """Mean expansion rows per expert of 15, 16 and 17 (n = 8, k = 2): the default choice moves
    from the streaming kernel to the large tiles at 16 rows, and the projection (fewer rows after
    the target mix) may take the other kernel in the same layer; every side matches the
    oracle."""
    cfg = scaled(SMALL["mixtral_s"], T=T, name=f"boundary{T}")
    assert (cfg.n, cfg.k) == (8, 2)
    say(f"tile policy boundary T={T} mean rows {T * cfg.k // cfg.n}")
    inp = make_inputs(cfg, seed=29)
    y = run_layer(dev(inp), cfg.k)
    assert_y_close(y, oracle.layer_inputs(inp), cfg.dtype, cfg.name)


@pytest.mark.parametrize("beta_mode", [1, 2])
def test_layer_beta_modes(beta_mode):
    cfg = SMALL["olmoe_s"]
    inp = make_inputs(cfg, seed=2)
    y = run_layer(dev(inp), cfg.k, beta_mode)
    assert_y_close(y, oracle.layer_inputs(inp, beta_mode=beta_mode), cfg.dtype, f"beta {beta_mode}")


def test_expand_rows_against_oracle():
    cfg = SMALL["mixtral_s"]
    inp = make_inputs(cfg, seed=3)
    d = dev(inp)
    ids, w = pcm.pcm_route(d["logits"], cfg.k)
    p = pcm.pcm_build_paths(ids, w, d["mask"])
    u = pcm.pcm_expand(d["x"], d["w_gate"], d["w_up"], p)
    torch.cuda.synchronize()
    rows = np.random.default_rng(0).choice(cfg.R, 64, replace=False)
    tok = p.row_token.cpu().numpy()[rows]
    ex = ids.cpu().numpy()[tok, p.row_slot.cpu().numpy()[rows]]
    ref = oracle.expansion_rows(inp.x, inp.w_gate, inp.w_up, tok, ex)
    got = u.cpu().numpy()[rows]
    scale = np.sqrt((ref ** 2).mean())
    # float32 accumulation of exact bf16 products over H terms
    assert np.all(np.abs(got - ref) <= 1e-5 * np.abs(ref) + 1e-5 * scale)


def test_layer_diagonal_mask_is_vanilla():
    """Only diagonal paths: the GPU layer equals the vanilla top-k MoE of the oracle."""
    cfg = scaled(SMALL["olmoe_s"], density=0.0, name="olmoe_diag")
    inp = make_inputs(cfg, seed=4)
    y = run_layer(dev(inp), cfg.k)
    assert_y_close(y, oracle.layer_inputs(inp), cfg.dtype, "diagonal only")


def test_layer_edge_cases():
    # k = n = 8 with a full mask; n = 1, k = 1; every token on one expert
    for cfg in (scaled(SMALL["olmoe_s"], n=8, k=8, density=1.0, T=300, name="k_eq_n"),
                scaled(SMALL["olmoe_s"], n=1, k=1, T=333, name="n1"),
                stress_config("one_expert", scaled(SMALL["olmoe_s"], T=700, name="one"))):
        inp = make_inputs(cfg, seed=5)
        y = run_layer(dev(inp), cfg.k)
        assert_y_close(y, oracle.layer_inputs(inp), cfg.dtype, cfg.name)


def test_zero_tokens_is_noop():
    cfg = SMALL["olmoe_s"]
    inp = make_inputs(scaled(cfg, T=4, name="t4"), seed=0)
    d = dev(inp)
    empty = d["x"][:0]
    y = pcm.layer_forward(empty, d["logits"][:0], d["mask"], d["w_gate"], d["w_up"], d["w_down"], cfg.k)
    torch.cuda.synchronize()
    assert y.shape == (0, cfg.H)


def test_dense_swiglu_accumulate():
    cfg = SMALL["fine_s"]
    inp = make_inputs(cfg, seed=6)
    d = dev(inp)
    base = torch.randn((cfg.T, cfg.H), device=DEV)
    y = pcm.pcm_dense_swiglu(d["x"], *d["shared"], y=base.clone(), accumulate=True)
    y0 = pcm.pcm_dense_swiglu(d["x"], *d["shared"])
    torch.cuda.synchronize()
    ref = oracle.dense_swiglu(inp.x, inp.s_gate, inp.s_up, inp.s_down)
    assert_y_close(y0.cpu().numpy(), ref, cfg.dtype, "dense")
    assert torch.equal(y, base + y0), "accumulate must add the same values"


@pytest.mark.parametrize("T", [513, 640, 641, 767, 768])
def test_dense_swiglu_large_tile_tails(T, monkeypatch):
    """One group of T rows on the 256 x 256 tiles: the last tile holds T mod 256 rows, and
    runs on the 128-row tail shape when that remainder is at most 128."""
    monkeypatch.setenv("PCM_GEMM_TILE", "L")
    cfg = scaled(CONFIGS["finegrained_shared"], T=T, H=256, F=64, shared_F=512, name=f"dense{T}")
    say(f"dense swiglu T={T}")
    inp = make_inputs(cfg, seed=8)
    d = dev(inp)
    y = pcm.pcm_dense_swiglu(d["x"], *d["shared"])
    torch.cuda.synchronize()
    ref = oracle.dense_swiglu(inp.x, inp.s_gate, inp.s_up, inp.s_down)
    assert_y_close(y.cpu().numpy(), ref, cfg.dtype, f"dense T={T}")


@pytest.mark.parametrize("name", ["mixtral_s", "olmoe_s", "fine_s", "splitk_s"])
def test_large_tile_work_orders_bit_identical(name, monkeypatch):
    """The work order of the large tiles (grouped, longest first, expert-major with several
    windows) decides only which workgroup computes which tile: the layer output must be the
    same bits under every order, and within tolerance of the oracle. Every intermediate
    buffer is filled with NaN before each run, so a tile that no workgroup computes shows."""
    monkeypatch.setenv("PCM_GEMM_TILE", "L")
    cfg = SMALL[name]
    inp = make_inputs(cfg, seed=21)
    d = dev(inp)
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, dtype, DEV, cfg.shared_F)

    def run():
        plan.u.fill_(float("nan"))
        plan.y.fill_(float("nan"))
        for ws in (plan.ws_proj, plan.ws_shared):
            if ws is not None:
                ws.fill_(0xFF)   # NaN in float16 and float32 alike
        y = plan.forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"],
                         d.get("shared"))
        torch.cuda.synchronize()
        return y.cpu().numpy()

    base = run()
    assert np.isfinite(base).all()
    assert_y_close(base, oracle.layer_inputs(inp), cfg.dtype, f"{name}/default order")
    for order, window in [(0, None), (1, None), (2, "1"), (2, "5"), (2, "12"), (2, "64")]:
        say(f"work order {order} window {window} on {name}")
        monkeypatch.setenv("PCM_GEMM_ORDER_EXPAND", str(order))
        monkeypatch.setenv("PCM_GEMM_ORDER_DOWN", str(order))
        if window is not None:
            monkeypatch.setenv("PCM_GEMM_EM_WINDOW", window)
        y = run()
        assert np.array_equal(y, base), f"{name}: order {order} window {window} changed the output"


@pytest.mark.parametrize("name", ["decode_s", "olmoe_s", "fine_s"])
def test_stream_kernels_bit_identical(name, monkeypatch):
    """The streaming GEMMs of few-row groups: the LDS-ring kernel (whole-line weight loads) at
    every ring depth and the register-ring kernel (depth 0; otherwise run only where buffer
    offsets would pass 4 GiB) feed the same operands to the same MFMAs, so the layer output must
    be the same bits under each, and within tolerance of the oracle."""
    monkeypatch.setenv("PCM_GEMM_TILE", "S")
    cfg = SMALL[name]
    inp = make_inputs(cfg, seed=23)
    d = dev(inp)
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, dtype, DEV, cfg.shared_F)

    def run():
        plan.u.fill_(float("nan"))
        plan.y.fill_(float("nan"))
        for ws in (plan.ws_proj, plan.ws_shared):
            if ws is not None:
                ws.fill_(0xFF)
        y = plan.forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"],
                         d.get("shared"))
        torch.cuda.synchronize()
        return y.cpu().numpy()

    base = run()
    assert np.isfinite(base).all()
    assert_y_close(base, oracle.layer_inputs(inp), cfg.dtype, f"{name}/default stream kernel")
    for depth in ["0", "2", "3", "4", "6"]:
        say(f"stream kernel depth {depth} on {name}")
        monkeypatch.setenv("PCM_LSTREAM_D", depth)
        y = run()
        assert np.array_equal(y, base), f"{name}: ring depth {depth} changed the output"


def test_layer_is_deterministic():
    cfg = SMALL["olmoe_s"]
    d = dev(make_inputs(cfg, seed=7))
    a = run_layer(d, cfg.k)
    b = run_layer(d, cfg.k)
    assert np.array_equal(a, b)


# ---------------------------------------------- full-size workloads, sampled tokens
@pytest.mark.slow
@pytest.mark.parametrize("name", ["tiny", "mixtral", "olmoe", "finegrained_shared", "decode"])
def test_layer_full_size(name):
    cfg = CONFIGS[name]
    say(f"full-size {name}: generating inputs")
    inp = make_inputs(cfg, seed=0)
    d = dev(inp)
    say(f"full-size {name}: running the layer")
    y = run_layer(d, cfg.k)
    ids, w = check_route(inp.logits, cfg.k)
    check_paths(ids, w, inp.mask, cfg.n)
    rng = np.random.default_rng(11)
    nsample = cfg.T if cfg.T <= 64 else 24
    tokens = np.unique(np.concatenate([[0, cfg.T - 1], rng.choice(cfg.T, nsample, replace=False)]))
    say(f"full-size {name}: oracle on {tokens.size} tokens")
    ref = oracle.layer_inputs(inp, tokens=tokens)
    assert_y_close(y[tokens], ref, cfg.dtype, name)
    assert np.isfinite(y).all()


def test_layer_split_k_projection_at_scale():
    """Few output tiles per row block and a long F: the large-tile projection splits K in two
    slices over hundreds of tiles. Sampled tokens against the oracle, bit-identical reruns."""
    cfg = scaled(CONFIGS["mixtral"], T=8192, H=1024, F=4096, name="split_k")
    say("split-K projection at scale: generating inputs")
    inp = make_inputs(cfg, seed=12)
    d = dev(inp)
    y = run_layer(d, cfg.k)
    y2 = run_layer(d, cfg.k)
    assert np.array_equal(y, y2), "the K slices must give the same sums every run"
    rng = np.random.default_rng(13)
    tokens = np.unique(np.concatenate([[0, cfg.T - 1], rng.choice(cfg.T, 96, replace=False)]))
    say(f"split-K projection at scale: oracle on {tokens.size} tokens")
    ref = oracle.layer_inputs(inp, tokens=tokens)
    assert_y_close(y[tokens], ref, cfg.dtype, "split-K at scale")


# ------------------------------------------- per-path execution (ablation baselines)
@pytest.mark.parametrize("reuse", [1, 0])
@pytest.mark.parametrize("name", ["tiny", "mixtral_s", "olmoe_s", "fine_s", "decode_s"])
def test_layer_per_path(name, reuse):
    """One projection per path (and, without reuse, one expansion per path): the same layer
    as the target-mixed path, against the oracle."""
    cfg = SMALL[name]
    say(f"per-path {name} reuse {reuse}")
    inp = make_inputs(cfg, seed=8)
    d = dev(inp)
    ids, w = pcm.pcm_route(d["logits"], cfg.k)
    p = pcm.pcm_build_paths(ids, w, d["mask"])
    y = pcm.pcm_layer_per_path(d["x"], d["w_gate"], d["w_up"], d["w_down"], p, reuse=bool(reuse))
    if "shared" in d:
        pcm.pcm_dense_swiglu(d["x"], *d["shared"], y=y, accumulate=True)
    torch.cuda.synchronize()
    assert_y_close(y.cpu().numpy(), oracle.layer_inputs(inp), cfg.dtype, f"per-path {name}")


def test_layer_per_path_reuse_is_bit_identical():
    """Recomputing U per path gives the same U rows, hence the same output bits."""
    cfg = SMALL["olmoe_s"]
    d = dev(make_inputs(cfg, seed=9))
    ids, w = pcm.pcm_route(d["logits"], cfg.k)
    p = pcm.pcm_build_paths(ids, w, d["mask"])
    a = pcm.pcm_layer_per_path(d["x"], d["w_gate"], d["w_up"], d["w_down"], p, reuse=True)
    b = pcm.pcm_layer_per_path(d["x"], d["w_gate"], d["w_up"], d["w_down"], p, reuse=False)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# ------------------------------------------------------- router GEMM fused with top-k
def check_route_logits(x, wr, k, what):
    ids, w, lg = pcm.pcm_route_logits(x.to(DEV), wr.to(DEV), k, want_logits=True)
    torch.cuda.synchronize()
    lg = lg.cpu().numpy()
    ref = oracle.router_logits(x, wr)
    xa = np.abs(x.float().numpy().astype(np.float64))
    wa = np.abs(wr.float().numpy().astype(np.float64))
    bound = 1e-5 * (xa @ wa.T) + FLT_MIN          # float32 accumulation of exact products
    assert np.all(np.abs(lg - ref) <= bound), f"router logits {what}"
    # the top-k decision is taken on the kernel's own float32 logits
    ids_ref, w_ref = oracle.route(lg, k)
    assert np.array_equal(ids.cpu().numpy(), ids_ref), f"router ids {what}"
    np.testing.assert_allclose(w.cpu().numpy(), w_ref, rtol=1e-5, atol=FLT_MIN, err_msg=what)
    return lg


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_route_logits_full_size(name):
    from workloads import make_router_weights
    cfg = CONFIGS[name]
    inp = make_inputs(cfg, seed=0, with_weights=False)
    wr = make_router_weights(cfg, seed=0)
    lg = check_route_logits(inp.x, wr, cfg.k, name)
    if name == "tiny":   # the tiny workload's logits are x W_r^T of the same matrix
        np.testing.assert_allclose(lg, inp.logits, rtol=1e-4, atol=1e-6)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("T,H,n,k", [(1, 64, 1, 1), (63, 128, 8, 2), (64, 256, 60, 4),
                                     (65, 192, 64, 8), (1000, 512, 256, 8), (130, 64, 17, 3)])
def test_route_logits_shapes(T, H, n, k, dtype):
    g = torch.Generator().manual_seed(T * 7 + n)
    x = torch.randn((T, H), generator=g)
    wr = torch.randn((n, H), generator=g) * 0.1
    if dtype == "bf16":
        x, wr = x.to(torch.bfloat16), wr.to(torch.bfloat16)
    check_route_logits(x, wr, k, f"T={T} H={H} n={n} k={k} {dtype}")
