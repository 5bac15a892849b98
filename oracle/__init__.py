"""CPU oracle of the path-compositional MoE layer: ctypes wrapper around
``pcomoe_oracle.c`` (plain C, float64, OpenMP over tokens).

TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import this package. It shares no code with the
GPU library and never imports it.

The wrapper marshals arguments only: every step of the computation happens in
the C file. Inputs are host arrays (numpy, or CPU torch tensors for bfloat16,
passed as their raw 16-bit patterns).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pcomoe_oracle.c")
_LIB = os.path.join(_HERE, "libpcomoe_oracle.so")

F32, BF16 = 0, 1
BETA_SRC_COND, BETA_PRODUCT, BETA_GLOBAL = 0, 1, 2


def build(extra_flags: Optional[list] = None, out: str = _LIB) -> str:
    """Compile the oracle with gcc (-O2, no fast-math, OpenMP)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall", "-Wextra",
           "-o", out + ".tmp", _SRC, "-lm"] + list(extra_flags or [])
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_lib = None


def lib(path: str = _LIB) -> ctypes.CDLL:
    global _lib
    if _lib is not None and path == _LIB:
        return _lib
    if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(_SRC):
        build(out=path)
    L = ctypes.CDLL(path)
    P, I64, I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    L.pcmo_route.argtypes = [P, I64, I, I, P, P]
    L.pcmo_paths.argtypes = [P, P, P, I64, I, I, I, P, P]
    L.pcmo_permute.argtypes = [P, I64, I, I, P, P, P, P]
    L.pcmo_layer_tokens.argtypes = [I, P, P, P, P, P, P, I64, I, I, I, I, I, I, P, I64, P]
    L.pcmo_expansion_rows.argtypes = [I, P, P, P, I64, I, I, I, P, P, I64, P]
    L.pcmo_dense_swiglu_tokens.argtypes = [I, P, P, P, P, I64, I, I, P, I64, P]
    L.pcmo_set_num_threads.argtypes = [I]
    Fl = ctypes.c_float
    L.pcmo_route_scored.argtypes = [P, P, Fl, P, P, I64, I, I, P, P, P, P]
    L.pcmo_group_scored.argtypes = [P, P, P, I64, I, P, P, P, P, P, P]
    L.pcmo_permute_var.argtypes = [P, P, I64, I, I, P, P, P, P]
    L.pcmo_layer_scored_tokens.argtypes = [I, P, P, P, Fl, P, P, P, P, P, I64, I, I, I, I, I, P,
                                           I64, P]
    L.pcmo_router_logits.argtypes = [I, P, P, I64, I, I, P]
    for name in ("pcmo_route", "pcmo_paths", "pcmo_permute", "pcmo_layer_tokens", "pcmo_router_logits",
                 "pcmo_expansion_rows", "pcmo_dense_swiglu_tokens", "pcmo_num_threads",
                 "pcmo_route_scored", "pcmo_group_scored", "pcmo_permute_var",
                 "pcmo_layer_scored_tokens"):
        getattr(L, name).restype = I
    if path == _LIB:
        _lib = L
    return L


def _ptr(a) -> int:
    return a.ctypes.data if isinstance(a, np.ndarray) else a.data_ptr()


def _host(a, dtype_code=None):
    """Host array in the oracle's element format: numpy float32 or uint16 bit patterns."""
    try:
        import torch
        if isinstance(a, torch.Tensor):
            a = a.detach().cpu().contiguous()
            if a.dtype == torch.bfloat16:
                return a.view(torch.int16).numpy().view(np.uint16), BF16
            return np.ascontiguousarray(a.numpy(), dtype=np.float32), F32
    except ImportError:  # pragma: no cover
        pass
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return a, BF16
    return np.ascontiguousarray(a, dtype=np.float32), F32


def _check(st: int, what: str):
    if st != 0:
        raise ValueError(f"oracle {what} failed with status {st}")


def num_threads() -> int:
    return lib().pcmo_num_threads()


def set_num_threads(nt: int):
    lib().pcmo_set_num_threads(int(nt))


def route(logits: np.ndarray, k: int, L=None):
    L = L or lib()
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    T, n = logits.shape
    ids = np.empty((T, k), np.int32)
    w = np.empty((T, k), np.float64)
    _check(L.pcmo_route(_ptr(logits), T, n, k, _ptr(ids), _ptr(w)), "route")
    return ids, w


def paths(topk_ids, topk_w, mask, beta_mode: int = BETA_SRC_COND, L=None):
    L = L or lib()
    ids = np.ascontiguousarray(topk_ids, dtype=np.int32)
    w = np.ascontiguousarray(topk_w, dtype=np.float64)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    T, k = ids.shape
    n = mask.shape[0]
    bits = np.empty((T,), np.uint64)
    beta = np.empty((T, k, k), np.float64)
    _check(L.pcmo_paths(_ptr(ids), _ptr(w), _ptr(mask), T, n, k, beta_mode, _ptr(bits), _ptr(beta)),
           "paths")
    return bits, beta


def permute(topk_ids, n: int, L=None):
    L = L or lib()
    ids = np.ascontiguousarray(topk_ids, dtype=np.int32)
    T, k = ids.shape
    offsets = np.empty((n + 1,), np.int32)
    row_token = np.empty((T * k,), np.int32)
    row_slot = np.empty((T * k,), np.int32)
    row_of = np.empty((T * k,), np.int32)
    _check(L.pcmo_permute(_ptr(ids), T, n, k, _ptr(offsets), _ptr(row_token), _ptr(row_slot),
                          _ptr(row_of)), "permute")
    return offsets, row_token, row_slot, row_of.reshape(T, k)


def layer(x, logits, w_gate, w_up, w_down, mask, k: int, beta_mode: int = BETA_SRC_COND,
          reuse: bool = True, tokens=None, L=None) -> np.ndarray:
    """y[tokens] of the layer in float64; tokens=None means every token."""
    L = L or lib()
    xh, dt = _host(x)
    wg, dtg = _host(w_gate)
    wu, dtu = _host(w_up)
    wd, dtd = _host(w_down)
    if not (dt == dtg == dtu == dtd):
        raise ValueError("x and the weights must share one dtype")
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    T, H = xh.shape
    n, F, H2 = wg.shape
    if H2 != H or wd.shape != (n, H, F) or wu.shape != wg.shape or logits.shape != (T, n):
        raise ValueError("shape mismatch")
    tok = np.arange(T, dtype=np.int64) if tokens is None else np.ascontiguousarray(tokens, np.int64)
    y = np.empty((tok.size, H), np.float64)
    _check(L.pcmo_layer_tokens(dt, _ptr(xh), _ptr(logits), _ptr(wg), _ptr(wu), _ptr(wd), _ptr(mask),
                               T, H, F, n, k, beta_mode, int(bool(reuse)), _ptr(tok), tok.size,
                               _ptr(y)), "layer")
    return y


def expansion_rows(x, w_gate, w_up, tokens, experts, L=None) -> np.ndarray:
    L = L or lib()
    xh, dt = _host(x)
    wg, _ = _host(w_gate)
    wu, _ = _host(w_up)
    T, H = xh.shape
    n, F, _ = wg.shape
    tok = np.ascontiguousarray(tokens, np.int64)
    ex = np.ascontiguousarray(experts, np.int32)
    U = np.empty((tok.size, F), np.float64)
    _check(L.pcmo_expansion_rows(dt, _ptr(xh), _ptr(wg), _ptr(wu), T, H, F, n, _ptr(tok), _ptr(ex),
                                 tok.size, _ptr(U)), "expansion_rows")
    return U


def dense_swiglu(x, wg, wu, wd, tokens=None, L=None) -> np.ndarray:
    L = L or lib()
    xh, dt = _host(x)
    g, _ = _host(wg)
    u, _ = _host(wu)
    d, _ = _host(wd)
    T, H = xh.shape
    Fs = g.shape[0]
    tok = np.arange(T, dtype=np.int64) if tokens is None else np.ascontiguousarray(tokens, np.int64)
    y = np.empty((tok.size, H), np.float64)
    _check(L.pcmo_dense_swiglu_tokens(dt, _ptr(xh), _ptr(g), _ptr(u), _ptr(d), T, H, Fs, _ptr(tok),
                                      tok.size, _ptr(y)), "dense_swiglu")
    return y


def layer_inputs(inp, tokens=None, beta_mode: int = BETA_SRC_COND, reuse: bool = True) -> np.ndarray:
    """y[tokens] for a workloads.LayerInputs, including the shared expert if it has one."""
    c = inp.cfg
    y = layer(inp.x, inp.logits, inp.w_gate, inp.w_up, inp.w_down, inp.mask, c.k,
              beta_mode=beta_mode, reuse=reuse, tokens=tokens)
    if inp.s_gate is not None:
        y = y + dense_swiglu(inp.x, inp.s_gate, inp.s_up, inp.s_down, tokens=tokens)
    return y


# ------------------------------------------------------------- scored routing
def route_scored(g_base, g_tgt, lam: float, bias, mask, K: int, L=None):
    """Selected paths of every token in selection order: src[T,K], tgt[T,K],
    score[T,K] (float32) and beta[T,K] (float64, softmax of the selected scores)."""
    L = L or lib()
    gb = np.ascontiguousarray(g_base, dtype=np.float32)
    gt = np.ascontiguousarray(g_tgt, dtype=np.float32)
    b = np.ascontiguousarray(bias, dtype=np.float32)
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    T, n = gb.shape
    src = np.empty((T, K), np.int32)
    tgt = np.empty((T, K), np.int32)
    score = np.empty((T, K), np.float32)
    beta = np.empty((T, K), np.float64)
    _check(L.pcmo_route_scored(_ptr(gb), _ptr(gt), float(lam), _ptr(b), _ptr(m), T, n, K, _ptr(src),
                               _ptr(tgt), _ptr(score), _ptr(beta)), "route_scored")
    return src, tgt, score, beta


def group_scored(src, tgt, beta, L=None):
    """Source and target groups: n_src[T], srcs[T,K], n_tgt[T], tgts[T,K] (ascending,
    -1 padded), bits[T] (bit a*K+b: path srcs[a] -> tgts[b]) and beta_g[T,K,K]."""
    L = L or lib()
    src = np.ascontiguousarray(src, np.int32)
    tgt = np.ascontiguousarray(tgt, np.int32)
    beta = np.ascontiguousarray(beta, np.float64)
    T, K = src.shape
    n_src = np.empty((T,), np.int32)
    srcs = np.empty((T, K), np.int32)
    n_tgt = np.empty((T,), np.int32)
    tgts = np.empty((T, K), np.int32)
    bits = np.empty((T,), np.uint64)
    beta_g = np.empty((T, K, K), np.float64)
    _check(L.pcmo_group_scored(_ptr(src), _ptr(tgt), _ptr(beta), T, K, _ptr(n_src), _ptr(srcs),
                               _ptr(n_tgt), _ptr(tgts), _ptr(bits), _ptr(beta_g)), "group_scored")
    return n_src, srcs, n_tgt, tgts, bits, beta_g


def permute_var(ids, counts, n: int, L=None):
    """Dispatch layout for counts[t] <= K entries per token: expert_offsets[n+1],
    row_token[R], row_slot[R], row_of[T,K] (-1 for unused slots), R = sum(counts)."""
    L = L or lib()
    ids = np.ascontiguousarray(ids, np.int32)
    counts = np.ascontiguousarray(counts, np.int32)
    T, K = ids.shape
    R = int(counts.sum())
    offsets = np.empty((n + 1,), np.int32)
    row_token = np.empty((max(R, 1),), np.int32)
    row_slot = np.empty((max(R, 1),), np.int32)
    row_of = np.empty((T * K,), np.int32)
    _check(L.pcmo_permute_var(_ptr(ids), _ptr(counts), T, n, K, _ptr(offsets), _ptr(row_token),
                              _ptr(row_slot), _ptr(row_of)), "permute_var")
    return offsets, row_token[:R], row_slot[:R], row_of.reshape(T, K)


def layer_scored(x, g_base, g_tgt, lam: float, bias, mask, w_gate, w_up, w_down, K: int,
                 reuse: bool = True, tokens=None, L=None) -> np.ndarray:
    """y[tokens] of the layer under scored routing, float64; tokens=None: every token."""
    L = L or lib()
    xh, dt = _host(x)
    wg, dtg = _host(w_gate)
    wu, dtu = _host(w_up)
    wd, dtd = _host(w_down)
    if not (dt == dtg == dtu == dtd):
        raise ValueError("x and the weights must share one dtype")
    gb = np.ascontiguousarray(g_base, dtype=np.float32)
    gt = np.ascontiguousarray(g_tgt, dtype=np.float32)
    b = np.ascontiguousarray(bias, dtype=np.float32)
    m = np.ascontiguousarray(mask, dtype=np.uint8)
    T, H = xh.shape
    n, F, H2 = wg.shape
    if H2 != H or wd.shape != (n, H, F) or gb.shape != (T, n) or gt.shape != (T, n) \
            or b.shape != (n, n) or m.shape != (n, n):
        raise ValueError("shape mismatch")
    tok = np.arange(T, dtype=np.int64) if tokens is None else np.ascontiguousarray(tokens, np.int64)
    y = np.empty((tok.size, H), np.float64)
    _check(L.pcmo_layer_scored_tokens(dt, _ptr(xh), _ptr(gb), _ptr(gt), float(lam), _ptr(b), _ptr(m),
                                      _ptr(wg), _ptr(wu), _ptr(wd), T, H, F, n, K, int(bool(reuse)),
                                      _ptr(tok), tok.size, _ptr(y)), "layer_scored")
    return y


def router_logits(x, w_router, L=None) -> np.ndarray:
    """logits[t, e] = x_t . W_r[e] in float64."""
    L = L or lib()
    xh, dt = _host(x)
    wr, dtw = _host(w_router)
    if dt != dtw:
        raise ValueError("x and the router weights must share one dtype")
    T, H = xh.shape
    n = wr.shape[0]
    out = np.empty((T, n), np.float64)
    _check(L.pcmo_router_logits(dt, _ptr(xh), _ptr(wr), T, H, n, _ptr(out)), "router_logits")
    return out
