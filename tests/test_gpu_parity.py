"""HIP path against the CPU oracle, through the C ABI (needs an MI355X).

Integers (top-k ids, path bits, the dispatch layout) must match bit for bit.
Floating point: router weights and path weights to 1e-5 relative (absolute
FLT_MIN below float32's normal range). Layer outputs: elementwise within
|d| <= 1e-2 + 2e-2 |ref| (the contract), and tighter, a relative Frobenius error
<= 1e-3 for bfloat16 layers and max |d| <= 1e-4 max |ref| for float32 layers.
In a bfloat16 layer U stays float32, the mixed z is rounded once to float16 (11
significant bits, after a power-of-two row scale) and the products accumulate in
float32, so the expected relative error is about 2^-12, near 2e-4.
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
        assert rel <= 1e-3, f"{what}: relative Frobenius error {rel:.3e} > 1e-3"
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


def run_layer(d, k, beta_mode=0, tuning=None):
    y = pcm.layer_forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"], k,
                          beta_mode=beta_mode, shared=d.get("shared"), tuning=tuning)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def poison(plan):
    """Fill every output, intermediate and workspace of a layer plan with NaN (or all-ones
    bits for integers), so that an element no kernel writes shows in the results."""
    nan = float("nan")
    for t in (plan.u, plan.y):
        t.fill_(nan)
    for ws in (getattr(plan, "ws_proj", None), getattr(plan, "ws_shared", None),
               getattr(plan, "ws_paths", None), getattr(plan, "ws_route", None)):
        if ws is not None:
            ws.fill_(0xFF)   # NaN in float16 and float32 alike, -1 in integers
    for name in getattr(plan.paths, "__dataclass_fields__", {}):
        t = getattr(plan.paths, name)
        if isinstance(t, torch.Tensor):
            t.view(torch.uint8).fill_(0xFF)
    for name in ("ids", "w"):
        if hasattr(plan, name):
            getattr(plan, name).view(torch.uint8).fill_(0xFF)


def block_tokens(offsets, row_token, bm=256):
    """The tokens of the first and the last row of every bm-row block of every expert's rows
    (the M tiles of the large-tile GEMMs), so that every tile has a row compared."""
    toks = []
    for e in range(len(offsets) - 1):
        for r0 in range(int(offsets[e]), int(offsets[e + 1]), bm):
            r1 = min(r0 + bm, int(offsets[e + 1])) - 1
            toks += [int(row_token[r0]), int(row_token[r1])]
    return np.array(toks, dtype=np.int64)


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
    # 16 N tiles per group in the expansion: the expert-major order deals each group's windows
    # over the 8 XCDs (window-interleaved), with one to four 256-row tiles per expert
    "wide_s": scaled(CONFIGS["mixtral"], T=1500, H=256, F=2048, name="wide_s"),
    # 24 N tiles per group, three per XCD: windows of one or three N tiles, and experts whose
    # last row block takes the tail tile (run after the full row blocks' windows) next to
    # experts with only a tail row block
    "wide3_s": scaled(CONFIGS["mixtral"], T=1200, H=192, F=3072, name="wide3_s"),
}


@pytest.mark.parametrize("tile", ["auto", "S", "M", "L", "W"])
@pytest.mark.parametrize("name", sorted(SMALL))
def test_layer_small(name, tile):
    tuning = pcm.Tuning(tile=tile) if tile != "auto" else None
    cfg = SMALL[name]
    say(f"layer {name} tile {tile}")
    inp = make_inputs(cfg, seed=1)
    d = dev(inp)
    y = run_layer(d, cfg.k, tuning=tuning)
    ref = oracle.layer_inputs(inp)
    assert_y_close(y, ref, cfg.dtype, f"{name}/{tile}")


@pytest.mark.parametrize("T,F", [(60, 448), (64, 448), (68, 448), (60, 4096), (64, 4096),
                                 (256, 4096), (512, 4096)])
def test_layer_tile_policy_boundary(T, F):
    """Mean rows per expert of 15, 16 and 17 (n = 8, k = 2), and with F = 4096 (the large-tile
    projection then splits K in two slices) of 15, 16, 64 and 128. Both GEMMs of a layer see
    the same rows (T * k, one per (token, slot) pair, sorted by expert), so both take the same
    kernel: the streaming kernel below 16 rows per expert, the large tiles from 16 on. The
    default output must be the same bits as a run with that kernel forced, and match the
    oracle."""
    cfg = scaled(SMALL["mixtral_s"], T=T, F=F, H=256 if F == 4096 else SMALL["mixtral_s"].H,
                 name=f"boundary{T}_{F}")
    assert (cfg.n, cfg.k) == (8, 2)
    rows = T * cfg.k // cfg.n
    say(f"tile policy boundary T={T} F={F} mean rows {rows}")
    inp = make_inputs(cfg, seed=29)
    d = dev(inp)
    y = run_layer(d, cfg.k)
    forced = run_layer(d, cfg.k, tuning=pcm.Tuning(tile="S" if rows < 16 else "L"))
    assert np.array_equal(y, forced), f"{cfg.name}: default differs from the forced kernel"
    if F == 4096 and rows >= 16:
        lay = pcm.project_workspace_layout(T, cfg.H, F, cfg.n, cfg.k, pcm.PCM_BF16)
        assert lay["ksplit"] == 2, "the projection splits K at this shape"
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


@pytest.mark.parametrize("name", ["mixtral_s", "olmoe_s", "decode_s", "wide_s", "wide3_s"])
def test_expand_output_bits_across_kernels(name):
    """Every expansion kernel (streaming at each ring depth and the register ring, medium
    tiles, large tiles in every work order) writes the same U bits: the same MFMA products in
    the same order and the same SwiGLU epilogue. U starts as NaN, so an element that no kernel
    writes shows. mixtral_s has a half-filled last N tile (F = 448)."""
    cfg = SMALL[name]
    d = dev(make_inputs(cfg, seed=24))
    ids, w = pcm.pcm_route(d["logits"], cfg.k)
    p = pcm.pcm_build_paths(ids, w, d["mask"])
    u = torch.empty((cfg.T * cfg.k, cfg.F), dtype=torch.float32, device=DEV)

    def run(tuning):
        u.fill_(float("nan"))
        pcm.pcm_expand(d["x"], d["w_gate"], d["w_up"], p, u=u, tuning=tuning)
        torch.cuda.synchronize()
        return u.cpu().numpy().copy()

    base = run(None)
    assert np.isfinite(base).all()
    for t in [dict(tile="S", stream_depth=0), dict(tile="S", stream_depth=2),
              dict(tile="S", stream_depth=6), dict(tile="M"), dict(tile="L", order_expand=0),
              dict(tile="L", order_expand=1), dict(tile="L", order_expand=2, em_window=1),
              dict(tile="L", order_expand=2, em_window=12), dict(tile="W", order_expand=0),
              dict(tile="W", order_expand=1), dict(tile="W", order_expand=2, em_window=1),
              dict(tile="W", order_expand=2, em_window=12)]:
        say(f"expansion kernels {name} {t}")
        got = run(pcm.Tuning(**t))
        assert np.array_equal(got.view(np.uint32), base.view(np.uint32)), f"{name} {t}"


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
@pytest.mark.parametrize("tile", ["L", "W"])
def test_dense_swiglu_large_tile_tails(T, tile):
    """One group of T rows on the 256 x 256 tiles (four or eight waves): the last tile holds
    T mod 256 rows, and runs on the 128-row tail shape when that remainder is at most 128."""
    cfg = scaled(CONFIGS["finegrained_shared"], T=T, H=256, F=64, shared_F=512, name=f"dense{T}")
    say(f"dense swiglu T={T} tile {tile}")
    inp = make_inputs(cfg, seed=8)
    d = dev(inp)
    y = pcm.pcm_dense_swiglu(d["x"], *d["shared"], tuning=pcm.Tuning(tile=tile))
    torch.cuda.synchronize()
    ref = oracle.dense_swiglu(inp.x, inp.s_gate, inp.s_up, inp.s_down)
    assert_y_close(y.cpu().numpy(), ref, cfg.dtype, f"dense T={T}")


@pytest.mark.parametrize("name", ["mixtral_s", "olmoe_s", "fine_s", "splitk_s", "wide_s", "wide3_s"])
def test_large_tile_work_orders_bit_identical(name):
    """The work order of the large tiles (grouped, longest first, expert-major with several
    windows) decides only which workgroup computes which tile: the layer output must be the
    same bits under every order, and within tolerance of the oracle. Every intermediate
    buffer is filled with NaN before each run, so a tile that no workgroup computes shows."""
    cfg = SMALL[name]
    inp = make_inputs(cfg, seed=21)
    d = dev(inp)
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, dtype, DEV, cfg.shared_F)

    def run(tuning):
        poison(plan)
        y = plan.forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"],
                         d.get("shared"), tuning=tuning)
        torch.cuda.synchronize()
        return y.cpu().numpy()

    base = run(pcm.Tuning(tile="L"))
    assert np.isfinite(base).all()
    assert_y_close(base, oracle.layer_inputs(inp), cfg.dtype, f"{name}/default order")
    for tile in ("L", "W"):      # the large tiles on four and on eight waves
        for order, window in [(0, 0), (1, 0), (2, 1), (2, 5), (2, 12), (2, 64)]:
            say(f"work order {order} window {window} tile {tile} on {name}")
            y = run(pcm.Tuning(tile=tile, order_expand=order, order_down=order, em_window=window))
            assert np.array_equal(y, base), \
                f"{name}: tile {tile} order {order} window {window} changed the output"


@pytest.mark.parametrize("name", ["mixtral_s", "olmoe_s", "fine_s", "decode_s", "wide_s", "wide3_s"])
def test_tile_families_bit_identical(name):
    """Where the projection does not split K, every tile family (streaming, medium, large tiles
    on four and on eight waves) accumulates each output over K in the same order, so the layer
    output is the same bits under each, the default choice included."""
    cfg = SMALL[name]
    inp = make_inputs(cfg, seed=25)
    d = dev(inp)
    for tile in ("L", "W"):
        assert pcm.project_workspace_layout(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, pcm.PCM_BF16,
                                            pcm.Tuning(tile=tile))["ksplit"] == 1, tile
    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, torch.bfloat16, DEV, cfg.shared_F)

    def run(tuning):
        poison(plan)
        y = plan.forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"],
                         d.get("shared"), tuning=tuning)
        torch.cuda.synchronize()
        return y.cpu().numpy()

    base = run(None)
    assert np.isfinite(base).all()
    assert_y_close(base, oracle.layer_inputs(inp), cfg.dtype, f"{name}/default")
    for tile in ("S", "M", "L", "W"):
        say(f"tile family {tile} on {name}")
        y = run(pcm.Tuning(tile=tile))
        assert np.array_equal(y.view(np.uint32), base.view(np.uint32)), f"{name}: tile {tile}"


@pytest.mark.parametrize("name", ["decode_s", "olmoe_s", "fine_s"])
def test_stream_kernels_bit_identical(name):
    """The streaming GEMMs of few-row groups: the LDS-ring kernel (whole-line weight loads) at
    every ring depth and the register-ring kernel (depth 0; otherwise run only where buffer
    offsets would pass 4 GiB) feed the same operands to the same MFMAs, so the layer output must
    be the same bits under each, and within tolerance of the oracle."""
    cfg = SMALL[name]
    inp = make_inputs(cfg, seed=23)
    d = dev(inp)
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, dtype, DEV, cfg.shared_F)

    def run(tuning):
        poison(plan)
        y = plan.forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"],
                         d.get("shared"), tuning=tuning)
        torch.cuda.synchronize()
        return y.cpu().numpy()

    base = run(pcm.Tuning(tile="S"))
    assert np.isfinite(base).all()
    assert_y_close(base, oracle.layer_inputs(inp), cfg.dtype, f"{name}/default stream kernel")
    for depth in [0, 2, 3, 4, 6]:
        say(f"stream kernel depth {depth} on {name}")
        y = run(pcm.Tuning(tile="S", stream_depth=depth))
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
    """The whole layer at the workload's size, in the launch configuration the benchmark
    times. Every buffer starts as NaN, so an element that no kernel writes shows; y is then
    compared with the oracle on the tokens of the first and last row of every 256-row block of
    every expert (every M tile of both GEMMs; all of y's columns cover every projection N
    tile, and every U column feeds every y column) plus a random sample."""
    cfg = CONFIGS[name]
    say(f"full-size {name}: generating inputs")
    inp = make_inputs(cfg, seed=0)
    d = dev(inp)
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, dtype, DEV, cfg.shared_F)
    poison(plan)
    say(f"full-size {name}: running the layer")
    y = plan.forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"],
                     d.get("shared"))
    torch.cuda.synchronize()
    y = y.cpu().numpy()
    assert np.isfinite(y).all(), f"{name}: unwritten or non-finite outputs"
    ids, w = check_route(inp.logits, cfg.k)
    assert torch.equal(ids, plan.ids) and torch.equal(w, plan.w)
    check_paths(ids, w, inp.mask, cfg.n)
    off = plan.paths.expert_offsets.cpu().numpy()
    rt = plan.paths.row_token.cpu().numpy()
    rng = np.random.default_rng(11)
    nsample = cfg.T if cfg.T <= 64 else 24
    tokens = np.unique(np.concatenate([[0, cfg.T - 1], rng.choice(cfg.T, nsample, replace=False),
                                       block_tokens(off, rt)]))
    say(f"full-size {name}: oracle on {tokens.size} tokens")
    ref = oracle.layer_inputs(inp, tokens=tokens)
    assert_y_close(y[tokens], ref, cfg.dtype, name)


@pytest.mark.slow
def test_projection_full_k_stage_mixtral():
    """The projection alone at the Mixtral shape (K = F = 14336): o read back
    from the workspace against float64 W_down z on the GPU's own z (float16 rows and their
    power-of-two scales), on the first and last row of every 256-row block of every expert,
    all H columns. A dropped 64-wide K stage changes o by about 7% (Frobenius); the bound is
    float32 accumulation."""
    cfg = CONFIGS["mixtral"]
    say("projection stage: generating inputs")
    inp = make_inputs(cfg, seed=0)
    d = dev(inp)
    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, torch.bfloat16, DEV)
    poison(plan)
    plan.forward(d["x"], d["logits"], d["mask"], d["w_gate"], d["w_up"], d["w_down"])
    torch.cuda.synchronize()
    R, H, F = cfg.R, cfg.H, cfg.F
    lay = pcm.project_workspace_layout(cfg.T, H, F, cfg.n, cfg.k, pcm.PCM_BF16)
    ks = lay["ksplit"]
    ws = plan.ws_proj
    z = ws[lay["z"]:lay["z"] + R * F * 2].view(torch.float16).view(R, F)
    zs = ws[lay["zscale"]:lay["zscale"] + R * 4].view(torch.float32)
    o = ws[lay["o"]:lay["o"] + ks * R * H * 4].view(torch.float32).view(ks, R, H)
    off = plan.paths.expert_offsets.cpu().numpy()
    rows = []
    for e in range(cfg.n):
        for r0 in range(int(off[e]), int(off[e + 1]), 256):
            rows += [r0, min(r0 + 256, int(off[e + 1])) - 1]
    rows = np.array(sorted(set(rows)))
    got = o.sum(dim=0).cpu().numpy()[rows].astype(np.float64)   # the combine's sum of slices
    assert np.isfinite(got).all()
    zr = z.cpu().numpy()[rows].astype(np.float64)
    sc = zs.cpu().numpy()[rows].astype(np.float64)
    expert = np.searchsorted(off, rows, side="right") - 1
    ref = np.empty_like(got)
    mag = np.empty_like(got)
    for e in np.unique(expert):
        sel = expert == e
        wd = inp.w_down[e].float().numpy().astype(np.float64)            # [H, F]
        ref[sel] = (zr[sel] @ wd.T) * sc[sel, None]
        mag[sel] = (np.abs(zr[sel]) @ np.abs(wd).T) * np.abs(sc[sel, None])
    err = np.abs(got - ref)
    assert np.all(err <= 1e-4 * mag + 1e-30), f"max err / bound {np.max(err / (1e-4 * mag)):.3f}"
    rel = np.linalg.norm(err) / np.linalg.norm(ref)
    assert rel <= 1e-4, f"relative Frobenius error of o {rel:.2e}"


def test_projection_weight_range():
    """Projection weights far from the workloads' N(0, 0.02): scaled by 1e-3 (many then fall
    below 2^-17, where the widening to float16 rounds to a multiple of 2^-24) and a few entries
    near 1e4 (exact in float16). The layer stays inside the contract and the tight gate."""
    cfg = SMALL["mixtral_s"]
    inp = make_inputs(cfg, seed=31)
    wd = inp.w_down.float() * 1e-3
    rng = np.random.default_rng(31)
    idx = [tuple(int(rng.integers(0, s)) for s in wd.shape) for _ in range(12)]
    for i, ix in enumerate(idx):
        wd[ix] = (1.0 if i % 2 else -1.0) * float(rng.uniform(8e3, 1.2e4))
    inp.w_down = wd.to(torch.bfloat16)
    frac = float((inp.w_down.float().abs() < 2 ** -17).float().mean())
    say(f"weight range: {frac:.2%} of W_down below 2^-17")
    assert frac > 0.1
    y = run_layer(dev(inp), cfg.k)
    assert_y_close(y, oracle.layer_inputs(inp), cfg.dtype, "projection weight range")


def test_layer_split_k_projection_at_scale():
    """Fewer output tiles than one round of the chip and a long F: the large-tile projection
    splits K in two slices (320 items). Sampled tokens against the oracle, bit-identical reruns."""
    cfg = scaled(CONFIGS["mixtral"], T=4096, H=1024, F=4096, name="split_k")
    assert pcm.project_workspace_layout(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, pcm.PCM_BF16)["ksplit"] == 2
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
