"""The fused indexing operation (Section 4.3: route, path filter, path weights and the
dispatch layout in one operation over a per-layer packed mask) against the oracle and
against the separate route and path-build calls, through the C ABI (needs an MI355X).

Integers (top-k ids, path bits, the dispatch layout) must match the oracle bit for bit;
router and path weights to 1e-5 relative (absolute FLT_MIN below float32's normal range).
Against pcm_route followed by pcm_build_paths every output, floats included, must be
bit-identical: both take the same float32 steps in the same order.
"""
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
FIELDS = ("path_bits", "beta", "expert_offsets", "row_token", "row_slot", "row_of")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def packed_reference(mask):
    """The packed layout by its definition: bit j % 64 of word [i][j // 64] is mask[i][j] != 0
    or i == j."""
    n = mask.shape[0]
    W = (n + 63) // 64
    out = np.zeros((n, W), np.uint64)
    for i in range(n):
        for j in range(n):
            if mask[i, j] or i == j:
                out[i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    return out


def fused(logits, packed, k, beta_mode=0):
    """The fused call with every output poisoned first (an element it does not write shows)."""
    T, n = logits.shape
    ids = torch.full((T, k), -1, dtype=torch.int32, device=DEV)
    w = torch.full((T, k), float("nan"), dtype=torch.float32, device=DEV)
    out = pcm.PathTable.empty(T, n, k, DEV)
    for f in FIELDS:
        getattr(out, f).view(torch.uint8).fill_(0xFF)
    ws_bytes = pcm.workspace_bytes(pcm.binding.OP_ROUTE_PATHS, T, 0, 0, n, k, 0)
    ws = torch.full((ws_bytes,), 0xFF, dtype=torch.uint8, device=DEV)
    ws[:256].zero_()   # the completion counter starts at zero; the rest is scratch
    r = pcm.pcm_route_paths(logits, packed, k, beta_mode, ids, w, out=out, ws=ws)
    torch.cuda.synchronize()
    assert not ws[:256].any(), "the call left its completion counter nonzero"
    return r


def check_fused(logits_np, mask_np, k, beta_mode=0, what=""):
    T, n = logits_np.shape
    logits = torch.from_numpy(logits_np).to(DEV)
    mask = torch.from_numpy(mask_np).to(DEV)
    packed = pcm.pcm_mask_pack(mask)
    ids, w, p = fused(logits, packed, k, beta_mode)
    torch.cuda.synchronize()
    # against the oracle
    ids_ref, w_ref = oracle.route(logits_np, k)
    assert np.array_equal(ids.cpu().numpy(), ids_ref), f"{what}: top-k ids differ"
    np.testing.assert_allclose(w.cpu().numpy(), w_ref, rtol=1e-5, atol=FLT_MIN)
    ids_np, w_np = ids.cpu().numpy(), w.cpu().numpy().astype(np.float64)
    bits_ref, beta_ref = oracle.paths(ids_np, w_np, mask_np, beta_mode)
    off_ref, rt_ref, rs_ref, ro_ref = oracle.permute(ids_np, n)
    assert np.array_equal(p.path_bits.cpu().numpy().view(np.uint64), bits_ref), f"{what}: path bits"
    np.testing.assert_allclose(p.beta.cpu().numpy(), beta_ref, rtol=1e-5, atol=FLT_MIN)
    assert np.array_equal(p.expert_offsets.cpu().numpy(), off_ref), f"{what}: expert offsets"
    assert np.array_equal(p.row_token.cpu().numpy(), rt_ref), f"{what}: row_token"
    assert np.array_equal(p.row_slot.cpu().numpy(), rs_ref), f"{what}: row_slot"
    assert np.array_equal(p.row_of.cpu().numpy(), ro_ref), f"{what}: row_of"
    # against the separate calls
    ids2, w2 = pcm.pcm_route(logits, k)
    p2 = pcm.pcm_build_paths(ids2, w2, mask, beta_mode)
    torch.cuda.synchronize()
    assert torch.equal(ids, ids2) and torch.equal(w.view(torch.int32), w2.view(torch.int32)), what
    for f in FIELDS:
        a, b = getattr(p, f), getattr(p2, f)
        if a.dtype == torch.float32:
            a, b = a.view(torch.int32), b.view(torch.int32)
        assert torch.equal(a, b), f"{what}: {f} differs from the separate calls"
    return ids, w, p


@pytest.mark.parametrize("n", [1, 5, 64, 65, 130, 256])
def test_mask_pack(n):
    rng = np.random.default_rng(n)
    mask = (rng.random((n, n)) < 0.3).astype(np.uint8) * rng.integers(1, 256, (n, n)).astype(np.uint8)
    np.fill_diagonal(mask, 0)   # the diagonal is set whatever the mask holds
    packed = torch.full((n, (n + 63) // 64), -1, dtype=torch.int64, device=DEV)
    pcm.pcm_mask_pack(torch.from_numpy(mask).to(DEV), packed)
    torch.cuda.synchronize()
    assert np.array_equal(packed.cpu().numpy().view(np.uint64), packed_reference(mask))


@pytest.mark.parametrize("name", sorted(CONFIGS))
def test_route_paths_full_size(name):
    cfg = CONFIGS[name]
    say(f"route_paths {name}")
    inp = make_inputs(cfg, with_weights=False)
    _, _, p1 = check_fused(inp.logits, inp.mask, cfg.k, what=name)
    _, _, p2 = fused(torch.from_numpy(inp.logits).to(DEV),
                     pcm.pcm_mask_pack(torch.from_numpy(inp.mask).to(DEV)), cfg.k)
    torch.cuda.synchronize()
    for f in FIELDS:
        assert torch.equal(getattr(p1, f).view(torch.uint8), getattr(p2, f).view(torch.uint8)), \
            f"{f} differs between runs"


@pytest.mark.parametrize("beta_mode", [0, 1, 2])
@pytest.mark.parametrize("T,n,k", [(1, 1, 1), (5, 4, 4), (63, 256, 8), (64, 8, 2), (65, 8, 2),
                                   (127, 64, 8), (128, 130, 5), (129, 200, 3), (1000, 65, 8),
                                   (4097, 60, 4), (3000, 256, 8)])
def test_route_paths_shapes(T, n, k, beta_mode):
    rng = np.random.default_rng(T * 7 + n)
    l = rng.standard_normal((T, n)).astype(np.float32)
    mask = (rng.random((n, n)) < 0.4).astype(np.uint8)
    if n > 1:
        mask[0, 0] = 0  # a zero diagonal entry is treated as 1
    check_fused(l, mask, k, beta_mode, what=f"T={T} n={n} k={k} beta={beta_mode}")


@pytest.mark.parametrize("kind", ["ties", "one_expert"])
def test_route_paths_stress(kind):
    cfg = stress_config(kind, scaled(CONFIGS["olmoe"], T=2500))
    inp = make_inputs(cfg, with_weights=False)
    _, _, p = check_fused(inp.logits, inp.mask, cfg.k, what=kind)
    if kind == "one_expert":
        assert int(p.expert_offsets[1] - p.expert_offsets[0]) == cfg.T


def test_route_paths_heavy_ties_and_signed_zeros():
    rng = np.random.default_rng(11)
    for n in (3, 64, 65, 256):
        l = (np.round(rng.standard_normal((200, n))) / 2).astype(np.float32)
        l[::7] = -0.0
        l[1::7] = 0.0
        mask = (rng.random((n, n)) < 0.5).astype(np.uint8)
        check_fused(l, mask, min(n, 8), what=f"ties n={n}")


@pytest.mark.parametrize("T,n,k", [(1, 8, 2), (3, 256, 8), (32, 256, 8), (61, 64, 8), (64, 60, 4),
                                   (65, 64, 8)])
def test_route_paths_reused_workspace(T, n, k):
    """Back-to-back calls on one workspace (the single-launch case's completion counter must
    come back to zero after each), alternating two inputs, each checked against the oracle."""
    rng = np.random.default_rng(T + 31 * n)
    ls = [rng.standard_normal((T, n)).astype(np.float32) for _ in range(2)]
    mask = (rng.random((n, n)) < 0.3).astype(np.uint8)
    packed = pcm.pcm_mask_pack(torch.from_numpy(mask).to(DEV))
    ws = pcm.binding.route_paths_workspace(T, n, k, DEV)
    outs = []
    for r in range(6):
        lg = torch.from_numpy(ls[r % 2]).to(DEV)
        ids, w, p = pcm.pcm_route_paths(lg, packed, k, ws=ws)
        outs.append((ids.clone(), p.row_token.clone(), p.row_of.clone(), p.expert_offsets.clone()))
    torch.cuda.synchronize()
    assert not ws[:256].any()
    for r in range(6):
        ids_ref, _ = oracle.route(ls[r % 2], k)
        off_ref, rt_ref, _, ro_ref = oracle.permute(ids_ref, n)
        ids, rt, ro, off = (t.cpu().numpy() for t in outs[r])
        assert np.array_equal(ids, ids_ref) and np.array_equal(off, off_ref), r
        assert np.array_equal(rt, rt_ref) and np.array_equal(ro, ro_ref), r


def test_layer_plan_with_packed_mask_is_bit_identical():
    cfg = scaled(CONFIGS["olmoe"], T=300, H=256, F=128)
    inp = make_inputs(cfg)
    x, logits = inp.x.to(DEV), torch.from_numpy(inp.logits).to(DEV)
    mask = torch.from_numpy(inp.mask).to(DEV)
    wg, wu, wd = inp.w_gate.to(DEV), inp.w_up.to(DEV), inp.w_down.to(DEV)
    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, x.dtype, DEV)
    y1 = plan.forward(x, logits, mask, wg, wu, wd).clone()
    y2 = plan.forward(x, logits, pcm.pcm_mask_pack(mask), wg, wu, wd).clone()
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int32), y2.view(torch.int32))
