"""Pins of the CPU oracle: checks against things other than the oracle itself.

Each ``pin_*`` function takes a loaded oracle library handle ``L`` and raises
AssertionError if the oracle disagrees with
  * brute force (stable sort of all logits, enumeration of all n x n paths,
    dense per-token evaluation of every U_i and every P_ij),
  * closed forms (the vanilla top-k MoE when only diagonal paths are allowed;
    the all-pairs closed form; k = 1; n = 1 as a dense SwiGLU FFN),
  * invariants (weight sums, expert relabelling, exact bfloat16 widening,
    reuse of expansion outputs not changing results).
The same functions run against deliberately broken builds of the oracle in
test_oracle_mutants.py, which shows that a plausible mistake fails a pin.
"""
from __future__ import annotations

import numpy as np

import oracle

RNG = np.random.default_rng(20260901)


# ----------------------------------------------------------------- references
def softmax_renorm_topk(l: np.ndarray, k: int):
    """Top-k by stable sort of all logits (ties to lower id) and the full softmax
    renormalised over the selected experts."""
    order = np.argsort(-l.astype(np.float64), axis=1, kind="stable")[:, :k]
    full = np.exp(l.astype(np.float64) - l.max(axis=1, keepdims=True))
    full /= full.sum(axis=1, keepdims=True)
    sel = np.take_along_axis(full, order, axis=1)
    return order.astype(np.int32), sel / sel.sum(axis=1, keepdims=True)


def textbook_swiglu(x, wg, wu, wd):
    """F(x) = W_down (SiLU(W_gate x) * (W_up x)) for rows of x (float64)."""
    g = x @ wg.T
    u = x @ wu.T
    return (g / (1.0 + np.exp(-g)) * u) @ wd.T


def dense_bruteforce_layer(x, logits, wg, wu, wd, mask, k, beta_mode=oracle.BETA_SRC_COND):
    """Every token: all n expansions U_i, all n^2 paths P_ij = W_down_j U_i, then the
    allowed ones among the token's selected experts, weighted by their path weight."""
    x = np.asarray(x, np.float64)
    T = x.shape[0]
    n = wg.shape[0]
    G = np.einsum("th,nfh->tnf", x, wg)
    Uall = G / (1.0 + np.exp(-G)) * np.einsum("th,nfh->tnf", x, wu)       # [T, n, F]
    P = np.einsum("jhf,tif->tijh", wd, Uall)                               # [T, n, n, H]
    ids, p = softmax_renorm_topk(logits, k)
    y = np.zeros((T, wd.shape[1]))
    for t in range(T):
        E = list(ids[t])
        prob = {e: p[t, a] for a, e in enumerate(E)}
        allowed = [(i, j) for i in range(n) for j in range(n)
                   if i in prob and j in prob and (i == j or mask[i, j])]
        tot = sum(prob[i] * prob[j] for i, j in allowed)
        for i, j in allowed:
            w = prob[i] * prob[j]
            if beta_mode == oracle.BETA_SRC_COND:
                w /= sum(prob[jj] for ii, jj in allowed if ii == i)
            elif beta_mode == oracle.BETA_GLOBAL:
                w /= tot
            y[t] += w * P[t, i, j]
    return y


def rand_layer(T, H, F, n, k, density, x_std=1.0, w_std=0.1, ties=False):
    x = RNG.standard_normal((T, H)) * x_std
    wg = RNG.standard_normal((n, F, H)) * w_std
    wu = RNG.standard_normal((n, F, H)) * w_std
    wd = RNG.standard_normal((n, H, F)) * w_std
    l = RNG.standard_normal((T, n)).astype(np.float32)
    if ties:
        l = (np.round(l * 2) / 2).astype(np.float32)
    mask = (RNG.random((n, n)) < density).astype(np.uint8)
    np.fill_diagonal(mask, 1)
    f32 = lambda a: np.ascontiguousarray(a, dtype=np.float32)
    return f32(x), l, f32(wg), f32(wu), f32(wd), mask


def _close(a, b, rel=1e-12, what=""):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    scale = max(np.abs(b).max(), 1e-300)
    err = np.abs(a - b).max() / scale
    assert err <= rel, f"{what}: max rel err {err:.3e} > {rel:.1e}"


# ----------------------------------------------------------------------- pins
def pin_topk_bruteforce(L):
    for n in (1, 2, 3, 8, 16, 64, 256):
        for k in sorted({1, min(n, 2), min(n, 4), min(n, 8)}):
            for ties in (False, True):
                l = RNG.standard_normal((97, n)).astype(np.float32)
                if ties:
                    l = (np.round(l * 2) / 2).astype(np.float32)
                ids, w = oracle.route(l, k, L=L)
                ref_ids, ref_w = softmax_renorm_topk(l, k)
                assert np.array_equal(ids, ref_ids), f"top-k ids n={n} k={k} ties={ties}"
                _close(w, ref_w, 1e-12, f"top-k weights n={n} k={k}")
                _close(w.sum(axis=1), np.ones(97), 1e-14, "weights sum to 1")
    # signed zeros are equal logits: the lower id wins
    l = np.array([[-0.0, 0.0, 0.0, -0.0, -1.0]], np.float32)
    ids, _ = oracle.route(l, 4, L=L)
    assert list(ids[0]) == [0, 1, 2, 3], ids


def pin_path_bits_bruteforce(L):
    for n, k, d in ((8, 2, 0.5), (16, 4, 0.3), (64, 8, 0.25), (3, 3, 0.5), (256, 8, 0.2)):
        l = RNG.standard_normal((50, n)).astype(np.float32)
        mask = (RNG.random((n, n)) < d).astype(np.uint8)
        mask[RNG.random(n) < 0.5, :] = 0  # some sources with no off-diagonal targets
        ids, w = oracle.route(l, k, L=L)
        m0 = mask.copy()
        np.fill_diagonal(m0, 0)  # a zero diagonal must be ignored (m_ii = 1 forced)
        bits, beta = oracle.paths(ids, w, m0, L=L)
        for t in range(50):
            slot = {int(e): a for a, e in enumerate(ids[t])}
            ref = 0
            for i in range(n):
                for j in range(n):
                    if i in slot and j in slot and (i == j or m0[i, j]):
                        ref |= 1 << (slot[i] * k + slot[j])
            assert int(bits[t]) == ref, f"path bits n={n} k={k} t={t}"
            off = [(a, b) for a in range(k) for b in range(k) if not (ref >> (a * k + b)) & 1]
            assert all(beta[t, a, b] == 0.0 for a, b in off), "beta must be 0 off-path"


def pin_beta_closed_forms(L):
    n, k = 16, 4
    l = RNG.standard_normal((200, n)).astype(np.float32)
    mask = (RNG.random((n, n)) < 0.4).astype(np.uint8)
    ids, p = oracle.route(l, k, L=L)
    bits, b_src = oracle.paths(ids, p, mask, oracle.BETA_SRC_COND, L=L)
    _, b_prod = oracle.paths(ids, p, mask, oracle.BETA_PRODUCT, L=L)
    _, b_glob = oracle.paths(ids, p, mask, oracle.BETA_GLOBAL, L=L)
    on = np.array([[[(int(bits[t]) >> (a * k + b)) & 1 for b in range(k)] for a in range(k)]
                   for t in range(200)], np.float64)
    prod = p[:, :, None] * p[:, None, :] * on
    _close(b_prod, prod, 1e-15, "PRODUCT = p_a p_b on paths")
    _close(b_glob, prod / prod.sum(axis=(1, 2), keepdims=True), 1e-14, "GLOBAL")
    _close(b_glob.sum(axis=(1, 2)), np.ones(200), 1e-14, "GLOBAL sums to 1")
    _close(b_src.sum(axis=(1, 2)), np.ones(200), 1e-14, "SRC_COND sums to 1")
    _close(b_src.sum(axis=2), p, 1e-14, "SRC_COND source row sums to p_a")
    srcsum = (p[:, None, :] * on).sum(axis=2)                      # sum_{b in T_a} p_b
    _close(b_src, prod / srcsum[:, :, None], 1e-14, "SRC_COND closed form")
    # every pair allowed: the three readings coincide and equal the product
    full = np.ones((n, n), np.uint8)
    for mode in (0, 1, 2):
        _, b = oracle.paths(ids, p, full, mode, L=L)
        _close(b, p[:, :, None] * p[:, None, :], 1e-14, f"full mask mode {mode}")
    # diagonal only: SRC_COND gives beta_aa = p_a, i.e. the vanilla weights alpha_e
    eye = np.eye(n, dtype=np.uint8)
    _, b = oracle.paths(ids, p, eye, oracle.BETA_SRC_COND, L=L)
    _close(np.einsum("taa->ta", b), p, 1e-15, "diagonal-only beta_aa = p_a")


def pin_permutation_bruteforce(L):
    for T, n, k in ((0, 4, 2), (1, 1, 1), (37, 8, 2), (300, 64, 8), (129, 256, 8), (64, 5, 5)):
        ids = np.array([RNG.permutation(n)[:k] for _ in range(T)], np.int32).reshape(T, k)
        off, rt, rs, ro = oracle.permute(ids, n, L=L)
        pairs = sorted((int(ids[t, a]), t, a) for t in range(T) for a in range(k))
        assert list(rt) == [t for _, t, _ in pairs], "row_token"
        assert list(rs) == [a for _, _, a in pairs], "row_slot"
        counts = np.bincount(ids.ravel(), minlength=n) if T else np.zeros(n, int)
        assert list(off) == [0] + list(np.cumsum(counts)), "expert_offsets"
        for r, (_, t, a) in enumerate(pairs):
            assert ro[t, a] == r, "row_of inverse"


def pin_layer_bruteforce(L):
    cases = [(6, 16, 8, 8, 2, 0.5), (5, 8, 16, 16, 4, 0.4), (4, 16, 8, 3, 3, 0.7),
             (7, 64, 16, 12, 8, 0.3), (3, 8, 8, 2, 1, 1.0)]
    for T, H, F, n, k, d in cases:
        for ties in (False, True):
            x, l, wg, wu, wd, mask = rand_layer(T, H, F, n, k, d, ties=ties)
            for mode in (0, 1, 2):
                y = oracle.layer(x, l, wg, wu, wd, mask, k, beta_mode=mode, L=L)
                ref = dense_bruteforce_layer(x, l, wg, wu, wd, mask, k, mode)
                _close(y, ref, 1e-12, f"layer vs brute force T={T} n={n} k={k} mode={mode}")


def pin_diagonal_is_vanilla_moe(L):
    """Only diagonal paths allowed: the layer is the standard top-k MoE (Section 4.1)."""
    T, H, F, n, k = 9, 32, 16, 8, 3
    x, l, wg, wu, wd, _ = rand_layer(T, H, F, n, k, 0.0)
    mask = np.eye(n, dtype=np.uint8)
    y = oracle.layer(x, l, wg, wu, wd, mask, k, L=L)
    ids, p = softmax_renorm_topk(l, k)
    ref = np.zeros((T, H))
    for t in range(T):
        for a in range(k):
            e = ids[t, a]
            ref[t] += p[t, a] * textbook_swiglu(x[t:t + 1].astype(np.float64), wg[e].astype(np.float64),
                                                wu[e].astype(np.float64), wd[e].astype(np.float64))[0]
    _close(y, ref, 1e-12, "diagonal-only = vanilla top-k MoE")


def pin_full_mask_closed_form(L):
    """Every pair allowed: y = sum_b p_b W_down_b (sum_a p_a U_a) by linearity of D."""
    T, H, F, n, k = 8, 16, 24, 6, 4
    x, l, wg, wu, wd, _ = rand_layer(T, H, F, n, k, 1.0)
    y = oracle.layer(x, l, wg, wu, wd, np.ones((n, n), np.uint8), k, L=L)
    ids, p = softmax_renorm_topk(l, k)
    ref = np.zeros((T, H))
    for t in range(T):
        xt = x[t].astype(np.float64)
        U = [(lambda g, u: g / (1 + np.exp(-g)) * u)(wg[e].astype(np.float64) @ xt,
                                                     wu[e].astype(np.float64) @ xt) for e in ids[t]]
        mix = sum(p[t, a] * U[a] for a in range(k))
        ref[t] = sum(p[t, b] * (wd[ids[t, b]].astype(np.float64) @ mix) for b in range(k))
    _close(y, ref, 1e-12, "full mask closed form")


def pin_k1_and_n1(L):
    T, H, F = 7, 16, 32
    x, l, wg, wu, wd, mask = rand_layer(T, H, F, 5, 1, 0.8)
    y = oracle.layer(x, l, wg, wu, wd, mask, 1, L=L)
    top = np.argmax(l, axis=1)
    f64 = lambda a: a.astype(np.float64)
    ref = np.stack([textbook_swiglu(f64(x[t:t + 1]), f64(wg[e]), f64(wu[e]), f64(wd[e]))[0]
                    for t, e in enumerate(top)])
    _close(y, ref, 1e-12, "k = 1 is the single selected expert")
    x, l, wg, wu, wd, mask = rand_layer(T, H, F, 1, 1, 0.0)
    y = oracle.layer(x, l, wg, wu, wd, mask, 1, L=L)
    _close(y, textbook_swiglu(f64(x), f64(wg[0]), f64(wu[0]), f64(wd[0])), 1e-12, "n = 1 dense FFN")
    ys = oracle.dense_swiglu(x, wg[0], wu[0], wd[0], L=L)
    _close(ys, textbook_swiglu(f64(x), f64(wg[0]), f64(wu[0]), f64(wd[0])), 1e-12, "shared expert")


def pin_reuse_and_target_mix(L):
    """Reusing U_i per source (Section 4.3) changes nothing; mixing per target before the
    linear D_j agrees to rounding."""
    T, H, F, n, k = 6, 16, 16, 8, 4
    x, l, wg, wu, wd, mask = rand_layer(T, H, F, n, k, 0.5)
    y_lit = oracle.layer(x, l, wg, wu, wd, mask, k, reuse=False, L=L)
    y_re = oracle.layer(x, l, wg, wu, wd, mask, k, reuse=True, L=L)
    assert np.array_equal(y_lit, y_re), "reuse must be bit-identical to per-path evaluation"
    ids, p = oracle.route(l, k, L=L)
    bits, beta = oracle.paths(ids, p, mask, L=L)
    U = oracle.expansion_rows(x, wg, wu, np.repeat(np.arange(T), k), ids.ravel(), L=L).reshape(T, k, F)
    Z = np.einsum("tab,taf->tbf", beta, U)
    y_mix = np.stack([sum(wd[ids[t, b]].astype(np.float64) @ Z[t, b] for b in range(k)) for t in range(T)])
    _close(y_re, y_mix, 1e-12, "target-mixed rewrite")


def pin_expansion_rows(L):
    T, H, F, n = 5, 32, 8, 4
    x, _, wg, wu, _, _ = rand_layer(T, H, F, n, 1, 0.0)
    tok = np.array([0, 4, 2, 2]); ex = np.array([3, 0, 1, 3], np.int32)
    U = oracle.expansion_rows(x, wg, wu, tok, ex, L=L)
    for i, (t, e) in enumerate(zip(tok, ex)):
        g = wg[e].astype(np.float64) @ x[t].astype(np.float64)
        u = wu[e].astype(np.float64) @ x[t].astype(np.float64)
        _close(U[i], g / (1 + np.exp(-g)) * u, 1e-13, "expansion row")


def pin_relabel_invariance(L):
    T, H, F, n, k = 6, 16, 8, 10, 3
    x, l, wg, wu, wd, mask = rand_layer(T, H, F, n, k, 0.5)
    y = oracle.layer(x, l, wg, wu, wd, mask, k, L=L)
    perm = RNG.permutation(n)            # old expert e becomes perm[e]
    inv = np.argsort(perm)
    y2 = oracle.layer(x, np.ascontiguousarray(l[:, inv]), np.ascontiguousarray(wg[inv]),
                      np.ascontiguousarray(wu[inv]), np.ascontiguousarray(wd[inv]),
                      np.ascontiguousarray(mask[np.ix_(inv, inv)]), k, L=L)
    _close(y2, y, 1e-14, "expert relabelling")
    ids, _ = oracle.route(l, k, L=L)
    ids2, _ = oracle.route(np.ascontiguousarray(l[:, inv]), k, L=L)
    assert np.array_equal(ids2, perm[ids]), "ids follow the relabelling"


def pin_bf16_widening(L):
    """bfloat16 inputs are widened exactly: same result as their float32 values."""
    import torch
    T, H, F, n, k = 4, 64, 64, 8, 2
    x, l, wg, wu, wd, mask = rand_layer(T, H, F, n, k, 0.5)
    tb = [torch.from_numpy(a).to(torch.bfloat16) for a in (x, wg, wu, wd)]
    y_b = oracle.layer(*tb[:1], l, *tb[1:], mask, k, L=L)
    y_f = oracle.layer(*[t.float() for t in tb[:1]], l, *[t.float() for t in tb[1:]], mask, k, L=L)
    assert np.array_equal(y_b, y_f), "bf16 widening must be exact"


def pin_edge_cases(L):
    # T = 0: nothing to do, success
    ids, w = oracle.route(np.zeros((0, 4), np.float32), 2, L=L)
    assert ids.shape == (0, 2)
    # k = n: every expert selected, every allowed pair is a path
    T, H, F, n = 3, 8, 8, 4
    x, l, wg, wu, wd, mask = rand_layer(T, H, F, n, n, 0.5)
    _close(oracle.layer(x, l, wg, wu, wd, mask, n, L=L),
           dense_bruteforce_layer(x, l, wg, wu, wd, mask, n), 1e-12, "k = n")
    # invalid arguments are rejected
    L2 = L
    st = L2.pcmo_route(0, 1, 4, 5, 0, 0)
    assert st != 0, "k > n must be rejected"
    st = L2.pcmo_route(0, 1, 16, 9, 0, 0)
    assert st != 0, "k > 8 must be rejected"


# ------------------------------------------------------------ scored routing
def eq9_bias(n, c=-1.0, noise=0.5, quant=None):
    """Compatibility bias of Section 4.2's initialisation: b_ii = 0, b_ij = c + eps with
    bounded uniform noise; quant rounds to a grid (exact float32 ties)."""
    b = (c + RNG.uniform(-noise, noise, (n, n))).astype(np.float32)
    if quant:
        b = (np.round(b / quant) * quant).astype(np.float32)
    np.fill_diagonal(b, 0.0)
    return b


def bruteforce_scored(gb, gt, lam, bias, mask, K):
    """Every token: the full n x n score matrix (float32; lam is a power of two so
    lam * g_tgt is exact and the sum is a single float32 rounding, as in fmaf), inactive
    pairs at -inf, then a stable sort of the flattened matrix by descending score: the
    first K entries, ties to the lower i*n + j. Returns src, tgt, score, beta."""
    T, n = gb.shape
    active = (mask != 0) | np.eye(n, dtype=bool)
    src = np.empty((T, K), np.int32); tgt = np.empty((T, K), np.int32)
    sc = np.empty((T, K), np.float32); beta = np.empty((T, K))
    for t in range(T):
        s = (gb[t][:, None] + bias).astype(np.float32) + np.float32(lam) * gt[t][None, :]
        s = s.astype(np.float32)
        flat = np.where(active, s, -np.inf).ravel()
        order = np.argsort(-flat.astype(np.float64), kind="stable")[:K]
        src[t], tgt[t] = order // n, order % n
        sc[t] = flat[order]
        e = np.exp(sc[t].astype(np.float64) - sc[t, 0])
        beta[t] = e / e.sum()
    return src, tgt, sc, beta


def dense_scored_layer(x, wg, wu, wd, src, tgt, beta):
    """All U_i and all P_ij per token, then y = sum over the selected paths of beta P_ij."""
    x = np.asarray(x, np.float64)
    G = np.einsum("th,nfh->tnf", x, wg)
    Uall = G / (1.0 + np.exp(-G)) * np.einsum("th,nfh->tnf", x, wu)
    P = np.einsum("jhf,tif->tijh", wd, Uall)
    T = x.shape[0]
    return np.stack([sum(beta[t, r] * P[t, src[t, r], tgt[t, r]] for r in range(src.shape[1]))
                     for t in range(T)])


def pin_scored_bruteforce(L):
    cases = [(7, 16, 8, 8, 2, 0.5, 0.5), (5, 8, 8, 16, 4, 0.3, 2.0), (6, 8, 16, 6, 6, 0.7, 0.0),
             (4, 8, 8, 64, 8, 0.25, 0.5), (3, 8, 8, 3, 3, 1.0, 1.0)]
    for T, H, F, n, K, d, lam in cases:
        for quant in (None, 0.25):
            x, _, wg, wu, wd, mask = rand_layer(T, H, F, n, K, d)
            gb = RNG.standard_normal((T, n)).astype(np.float32)
            gt = RNG.standard_normal((T, n)).astype(np.float32)
            if quant:
                gb = (np.round(gb / quant) * quant).astype(np.float32)
                gt = (np.round(gt / quant) * quant).astype(np.float32)
            bias = eq9_bias(n, quant=quant)
            m0 = mask.copy(); np.fill_diagonal(m0, 0)      # a zero diagonal is overridden
            src, tgt, sc, beta = oracle.route_scored(gb, gt, lam, bias, m0, K, L=L)
            rs, rt, rsc, rb = bruteforce_scored(gb, gt, lam, bias, m0, K)
            what = f"T={T} n={n} K={K} lam={lam} quant={quant}"
            assert np.array_equal(src, rs) and np.array_equal(tgt, rt), f"selected paths {what}"
            assert np.array_equal(sc, rsc), f"scores {what}"
            _close(beta, rb, 1e-14, f"beta {what}")
            y = oracle.layer_scored(x, gb, gt, lam, bias, m0, wg, wu, wd, K, L=L)
            ref = dense_scored_layer(x, wg, wu, wd, rs, rt, rb)
            _close(y, ref, 1e-12, f"layer vs brute force {what}")


def pin_scored_reduces_to_vanilla(L):
    """Only diagonal paths, no target prior: the router is the vanilla top-K with the
    renormalised softmax, and the layer is the standard top-k MoE (Section 4.1)."""
    T, H, F, n, K = 9, 32, 16, 8, 3
    x, l, wg, wu, wd, _ = rand_layer(T, H, F, n, K, 0.0)
    eye = np.eye(n, dtype=np.uint8)
    gt = RNG.standard_normal((T, n)).astype(np.float32)
    bias = eq9_bias(n)
    src, tgt, _, beta = oracle.route_scored(l, gt, 0.0, bias, eye, K, L=L)
    ids, p = softmax_renorm_topk(l, K)
    assert np.array_equal(src, ids) and np.array_equal(tgt, ids), "diagonal top-K"
    _close(beta, p, 1e-14, "beta = renormalised softmax")
    y = oracle.layer_scored(x, l, gt, 0.0, bias, eye, wg, wu, wd, K, L=L)
    f64 = lambda a: a.astype(np.float64)
    ref = np.stack([sum(p[t, a] * textbook_swiglu(f64(x[t:t + 1]), f64(wg[e]), f64(wu[e]), f64(wd[e]))[0]
                        for a, e in enumerate(ids[t])) for t in range(T)])
    _close(y, ref, 1e-12, "scored routing with mask = I is the vanilla MoE")
    # a very negative off-diagonal bias prunes like the mask
    full = np.ones((n, n), np.uint8)
    b2 = np.full((n, n), -1e4, np.float32); np.fill_diagonal(b2, 0.0)
    src2, tgt2, _, beta2 = oracle.route_scored(l, gt, 0.0, b2, full, K, L=L)
    assert np.array_equal(src2, ids) and np.array_equal(tgt2, ids), "bias pruning"
    _close(beta2, p, 1e-14, "bias pruning beta")


def pin_scored_single_source(L):
    """All pairs active, zero bias, no target prior: s_ij = g_i, so the K paths are
    (i*, 0), ..., (i*, K-1) of the top source, each with weight 1/K:
    y = (1/K) sum_{j<K} W_down_j U_{i*}."""
    T, H, F, n, K = 6, 16, 24, 8, 4
    x, l, wg, wu, wd, _ = rand_layer(T, H, F, n, K, 1.0)
    full = np.ones((n, n), np.uint8)
    gt = RNG.standard_normal((T, n)).astype(np.float32)
    zero = np.zeros((n, n), np.float32)
    src, tgt, _, beta = oracle.route_scored(l, gt, 0.0, zero, full, K, L=L)
    top = np.argmax(l, axis=1)
    assert np.array_equal(src, np.repeat(top[:, None], K, 1)), "single source"
    assert np.array_equal(tgt, np.tile(np.arange(K, dtype=np.int32), (T, 1))), "targets 0..K-1"
    _close(beta, np.full((T, K), 1.0 / K), 1e-15, "uniform weights")
    y = oracle.layer_scored(x, l, gt, 0.0, zero, full, wg, wu, wd, K, L=L)
    ref = np.zeros((T, H))
    for t in range(T):
        xt, i = x[t].astype(np.float64), top[t]
        g, u = wg[i].astype(np.float64) @ xt, wu[i].astype(np.float64) @ xt
        U = g / (1 + np.exp(-g)) * u
        ref[t] = sum(wd[j].astype(np.float64) @ U for j in range(K)) / K
    _close(y, ref, 1e-12, "single-source closed form")


def pin_scored_target_prior(L):
    """A dominant target prior sends every selected path to its unique best target j*;
    the sources are then the top-K of g_base_i + b_ij* (ties to the lower id)."""
    T, n, K = 40, 16, 5
    gb = RNG.standard_normal((T, n)).astype(np.float32)
    gt = RNG.standard_normal((T, n)).astype(np.float32)
    jstar = RNG.integers(0, n, T)
    gt[np.arange(T), jstar] = 8.0
    bias = eq9_bias(n)
    full = np.ones((n, n), np.uint8)
    src, tgt, _, _ = oracle.route_scored(gb, gt, 64.0, bias, full, K, L=L)
    assert np.array_equal(tgt, np.repeat(jstar[:, None].astype(np.int32), K, 1)), "one target"
    for t in range(T):
        col = (gb[t] + bias[:, jstar[t]]).astype(np.float32)
        assert list(src[t]) == list(np.argsort(-col.astype(np.float64), kind="stable")[:K]), "sources"


def pin_scored_groups_and_dispatch(L):
    for T, n, K, d in ((50, 8, 2, 0.5), (40, 64, 8, 0.25), (30, 256, 8, 0.2), (20, 6, 6, 1.0)):
        gb = RNG.standard_normal((T, n)).astype(np.float32)
        gt = RNG.standard_normal((T, n)).astype(np.float32)
        mask = (RNG.random((n, n)) < d).astype(np.uint8)
        bias = eq9_bias(n, noise=1.5)
        src, tgt, _, beta = oracle.route_scored(gb, gt, 0.5, bias, mask, K, L=L)
        _close(beta.sum(axis=1), np.ones(T), 1e-14, "weights sum to 1")
        assert np.all(np.diff(beta, axis=1) <= 0), "weights follow the selection order"
        n_src, srcs, n_tgt, tgts, bits, bg = oracle.group_scored(src, tgt, beta, L=L)
        for t in range(T):
            pairs = list(zip(src[t], tgt[t]))
            assert len(set(pairs)) == K, "distinct paths"
            assert all(i == j or mask[i, j] for i, j in pairs), "paths inside A"
            S, G = sorted(set(src[t])), sorted(set(tgt[t]))
            assert n_src[t] == len(S) and list(srcs[t, :len(S)]) == S, "sources"
            assert n_tgt[t] == len(G) and list(tgts[t, :len(G)]) == G, "targets"
            ref = 0
            for r, (i, j) in enumerate(pairs):
                a, b = S.index(i), G.index(j)
                ref |= 1 << (a * K + b)
                assert bg[t, a, b] == beta[t, r], "grouped weight"
            assert int(bits[t]) == ref, "grouped bits"
            assert abs(bg[t].sum() - 1.0) < 1e-14, "grouped weights sum to 1"
        for ids, cnt in ((srcs, n_src), (tgts, n_tgt)):
            off, rt, rs, ro = oracle.permute_var(ids, cnt, n, L=L)
            entries = sorted((int(ids[t, a]), t, a) for t in range(T) for a in range(cnt[t]))
            assert list(rt) == [t for _, t, _ in entries] and list(rs) == [a for _, _, a in entries]
            counts = np.bincount([e for e, _, _ in entries], minlength=n)
            assert list(off) == [0] + list(np.cumsum(counts)), "offsets"
            for r, (_, t, a) in enumerate(entries):
                assert ro[t, a] == r, "row_of"
            assert all(ro[t, a] == -1 for t in range(T) for a in range(cnt[t], K)), "unused slots"
    # reuse of U per source changes nothing
    T, H, F, n, K = 5, 16, 16, 8, 4
    x, _, wg, wu, wd, mask = rand_layer(T, H, F, n, K, 0.6)
    gb = RNG.standard_normal((T, n)).astype(np.float32)
    gt = RNG.standard_normal((T, n)).astype(np.float32)
    bias = eq9_bias(n, noise=1.0)
    y1 = oracle.layer_scored(x, gb, gt, 1.0, bias, mask, wg, wu, wd, K, reuse=True, L=L)
    y0 = oracle.layer_scored(x, gb, gt, 1.0, bias, mask, wg, wu, wd, K, reuse=False, L=L)
    assert np.array_equal(y0, y1), "reuse must be bit-identical"


def pin_scored_relabel_and_edges(L):
    T, H, F, n, K = 6, 16, 8, 10, 3
    x, _, wg, wu, wd, mask = rand_layer(T, H, F, n, K, 0.5)
    gb = RNG.standard_normal((T, n)).astype(np.float32)
    gt = RNG.standard_normal((T, n)).astype(np.float32)
    bias = eq9_bias(n, noise=1.0)
    y = oracle.layer_scored(x, gb, gt, 0.5, bias, mask, wg, wu, wd, K, L=L)
    perm = RNG.permutation(n)
    inv = np.argsort(perm)
    c = np.ascontiguousarray
    y2 = oracle.layer_scored(x, c(gb[:, inv]), c(gt[:, inv]), 0.5, c(bias[np.ix_(inv, inv)]),
                             c(mask[np.ix_(inv, inv)]), c(wg[inv]), c(wu[inv]), c(wd[inv]), K, L=L)
    _close(y2, y, 1e-14, "expert relabelling")
    src, _, _, _ = oracle.route_scored(np.zeros((0, n), np.float32), np.zeros((0, n), np.float32),
                                       0.5, bias, mask, K, L=L)
    assert src.shape == (0, K)
    assert L.pcmo_route_scored(0, 0, 0.5, 0, 0, 1, 4, 5, 0, 0, 0, 0) != 0, "K > n must be rejected"
    assert L.pcmo_route_scored(0, 0, 0.5, 0, 0, 1, 16, 9, 0, 0, 0, 0) != 0, "K > 8 must be rejected"


def fp32_nearest(q) -> np.float32:
    """The float32 nearest to the exact rational q, ties to the even significand (IEEE
    round-to-nearest-even), from integer arithmetic on q's numerator and denominator."""
    from fractions import Fraction
    q = Fraction(q)
    if q == 0:
        return np.float32(0.0)
    sign, a = (-1, -q) if q < 0 else (1, q)
    e = a.numerator.bit_length() - a.denominator.bit_length()   # 2^e <= a < 2^(e+2)
    if a < Fraction(2) ** e:
        e -= 1
    elif a >= Fraction(2) ** (e + 1):
        e += 1
    quantum = max(e - 23, -149)                                  # 24 significant bits; subnormals
    m = a / Fraction(2) ** quantum
    fl = m.numerator // m.denominator
    rem = m - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    v = Fraction(fl) * Fraction(2) ** quantum
    assert v <= Fraction(float(np.finfo(np.float32).max)), "overflow"
    return np.float32(sign * float(v))                           # exact: v has <= 24 bits


def fma_f32(a, b, c) -> np.float32:
    """a * b + c for float32 operands, rounded once to float32 (exact rational arithmetic)."""
    from fractions import Fraction
    return fp32_nearest(Fraction(float(a)) * Fraction(float(b)) + Fraction(float(c)))


def pin_scored_general_lambda(L):
    """The path score at a weight lambda that is not a power of two (so lambda * g_tgt is not
    exact in float32): every score equals g_base_i + b_ij (one float32 addition) plus
    lambda * g_tgt_j, the sum rounded once, computed here in exact rational arithmetic; the
    selection is the stable descending sort of those scores and the weights their softmax."""
    for lam, (T, n, K, d) in ((0.3, (12, 16, 8, 0.4)), (0.7, (10, 8, 4, 0.6)),
                              (-1.25, (10, 12, 6, 0.5))):
        gb = RNG.standard_normal((T, n)).astype(np.float32)
        gt = RNG.standard_normal((T, n)).astype(np.float32)
        mask = (RNG.random((n, n)) < d).astype(np.uint8)
        bias = eq9_bias(n)
        lam32 = np.float32(lam)
        src, tgt, sc, beta = oracle.route_scored(gb, gt, lam, bias, mask, K, L=L)
        active = (mask != 0) | np.eye(n, dtype=bool)
        rounded_twice = 0
        for t in range(T):
            s = np.full((n, n), -np.inf)
            for i in range(n):
                for j in range(n):
                    if active[i, j]:
                        c = gb[t, i] + bias[i, j]          # float32 + float32: one rounding
                        s[i, j] = fma_f32(lam32, gt[t, j], c)
                        rounded_twice += s[i, j] != np.float32(np.float32(lam32 * gt[t, j]) + c)
            order = np.argsort(-s.ravel(), kind="stable")[:K]
            what = f"lambda={lam} token {t}"
            assert list(src[t]) == list(order // n) and list(tgt[t]) == list(order % n), what
            assert np.array_equal(sc[t], s.ravel()[order].astype(np.float32)), f"scores {what}"
            e = np.exp(s.ravel()[order] - s.ravel()[order[0]])
            _close(beta[t], e / e.sum(), 1e-14, f"weights {what}")
        # the case is informative: rounding the product separately changes some scores
        assert rounded_twice > 0, f"lambda={lam}: no score tells one rounding from two"


def pin_router_logits(L):
    """Router scores: one-hot router rows read single features; a scaled row scales its
    score; a brute-force sum over h on small integers is exact; bf16 widening is exact."""
    T, H, n = 9, 64, 6
    x = RNG.standard_normal((T, H)).astype(np.float32)
    hsel = RNG.choice(H, n, replace=False)
    onehot = np.zeros((n, H), np.float32)
    onehot[np.arange(n), hsel] = 1.0
    _close(oracle.router_logits(x, onehot, L=L), x[:, hsel].astype(np.float64), 0.0, "one-hot rows")
    onehot[2] *= 3.0
    _close(oracle.router_logits(x, onehot, L=L)[:, 2], 3.0 * x[:, hsel[2]].astype(np.float64), 1e-15,
           "scaled row")
    xi = RNG.integers(-8, 9, (T, H)).astype(np.float32)
    wi = RNG.integers(-8, 9, (n, H)).astype(np.float32)
    ref = np.array([[sum(int(xi[t, h]) * int(wi[e, h]) for h in range(H)) for e in range(n)]
                    for t in range(T)], np.float64)
    assert np.array_equal(oracle.router_logits(xi, wi, L=L), ref), "integer brute force"
    import torch
    xb, wb = torch.from_numpy(x).to(torch.bfloat16), torch.from_numpy(wi).to(torch.bfloat16)
    assert np.array_equal(oracle.router_logits(xb, wb, L=L),
                          oracle.router_logits(xb.float(), wb.float(), L=L)), "bf16 widening"


ALL_PINS = [pin_topk_bruteforce, pin_path_bits_bruteforce, pin_beta_closed_forms,
            pin_permutation_bruteforce, pin_layer_bruteforce, pin_diagonal_is_vanilla_moe,
            pin_full_mask_closed_form, pin_k1_and_n1, pin_reuse_and_target_mix,
            pin_expansion_rows, pin_relabel_invariance, pin_bf16_widening, pin_edge_cases,
            pin_scored_bruteforce, pin_scored_reduces_to_vanilla, pin_scored_single_source,
            pin_scored_target_prior, pin_scored_groups_and_dispatch, pin_scored_relabel_and_edges,
            pin_scored_general_lambda, pin_router_logits]
