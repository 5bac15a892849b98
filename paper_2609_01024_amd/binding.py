"""ctypes binding of libpcomoe (include/pcomoe.h) for torch tensors on a ROCm device.

The functions carry the C entry points' names and only marshal arguments: they
check shapes and dtypes, allocate outputs with torch when the caller passes none,
and pass raw device pointers plus the current HIP stream. Every step of the layer
runs in the library's HIP kernels; there is no fallback path. If the library is
not built, the first call raises RuntimeError.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from dataclasses import dataclass, field
from typing import Optional, Sequence

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpcomoe.so")

PCM_F32, PCM_BF16, PCM_BF16_F16DOWN = 0, 1, 2
BETA_SRC_COND, BETA_PRODUCT, BETA_GLOBAL = 0, 1, 2
OP_BUILD_PATHS, OP_EXPAND, OP_PROJECT_COMBINE, OP_DENSE_SWIGLU, OP_ROUTE_SCORED = 0, 1, 2, 3, 4
OP_LAYER_PER_PATH, OP_ROUTE_LOGITS, OP_ROUTE_PATHS = 5, 6, 7

EXPORTS = ("pcm_route", "pcm_build_paths", "pcm_expand", "pcm_project_combine",
           "pcm_dense_swiglu", "pcm_workspace_bytes", "pcm_status_string", "pcm_abi_version",
           "pcm_path_layout_build", "pcm_route_scored", "pcm_expand_scored",
           "pcm_project_combine_scored", "pcm_layer_per_path", "pcm_route_logits",
           "pcm_residual_add", "pcm_expand_tuned", "pcm_project_combine_tuned",
           "pcm_dense_swiglu_tuned", "pcm_expand_scored_tuned", "pcm_project_combine_scored_tuned",
           "pcm_project_workspace_layout", "pcm_project_combine_noalloc", "pcm_mask_pack",
           "pcm_route_paths", "pcm_widen_f16")


class PcmTuning(ctypes.Structure):
    _fields_ = [("tile", ctypes.c_int), ("order_expand", ctypes.c_int), ("order_down", ctypes.c_int),
                ("em_window", ctypes.c_int), ("group_n", ctypes.c_int), ("stream_depth", ctypes.c_int),
                ("stage_events", ctypes.c_void_p * 4)]


@dataclass
class Tuning:
    """Kernel choices forced for tests and measurement (pcm_tuning); the defaults are the
    library's own choices. stage_events: four torch.cuda.Event (created by a first record)
    that the project-and-combine calls record before the mix, the projection GEMM, the combine
    and after it."""
    tile: str = ""              # "", "S", "M", "L" (four waves) or "W" (eight waves)
    order_expand: int = -1
    order_down: int = -1
    em_window: int = 0
    group_n: int = 0
    stream_depth: int = -1
    stage_events: Sequence = field(default_factory=tuple)

    def struct(self) -> PcmTuning:
        ev = [0, 0, 0, 0]
        for i, e in enumerate(self.stage_events):
            ev[i] = e.cuda_event
        return PcmTuning(ord(self.tile) if self.tile else 0, self.order_expand, self.order_down,
                         self.em_window, self.group_n, self.stream_depth, (ctypes.c_void_p * 4)(*ev))


class PcmPaths(ctypes.Structure):
    _fields_ = [("path_bits", ctypes.c_void_p), ("beta", ctypes.c_void_p),
                ("expert_offsets", ctypes.c_void_p), ("row_token", ctypes.c_void_p),
                ("row_slot", ctypes.c_void_p), ("row_of", ctypes.c_void_p)]


class PcmPathLayout(ctypes.Structure):
    _fields_ = [("count", ctypes.c_void_p), ("pair", ctypes.c_void_p), ("bias", ctypes.c_void_p)]


_SCORED_FIELDS = ("sel_pair", "sel_score", "n_src", "src_expert", "n_tgt", "tgt_expert",
                  "path_bits", "beta", "src_offsets", "src_row_token", "src_row_slot", "src_row_of",
                  "tgt_offsets", "tgt_row_token", "tgt_row_slot", "tgt_row_of")


class PcmScoredPaths(ctypes.Structure):
    _fields_ = [(f, ctypes.c_void_p) for f in _SCORED_FIELDS]


_lib = None


def lib(path: str = _LIB_PATH) -> ctypes.CDLL:
    """Load libpcomoe.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -c 'import __graft_entry__ as g; "
                           "g.build()'` (the layer has no fallback path)")
    L = ctypes.CDLL(path)
    P, I, I64, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    L.pcm_route.argtypes = [P, I64, I, I, P, P, P]
    L.pcm_build_paths.argtypes = [P, P, P, I64, I, I, I, ctypes.POINTER(PcmPaths), P, SZ, P]
    L.pcm_mask_pack.argtypes = [P, I, P, P]
    L.pcm_route_paths.argtypes = [P, P, I64, I, I, I, P, P, ctypes.POINTER(PcmPaths), P, SZ, P]
    L.pcm_expand.argtypes = [I, P, P, P, ctypes.POINTER(PcmPaths), I64, I, I, I, I, P, P, SZ, P]
    L.pcm_project_combine.argtypes = [I, P, P, ctypes.POINTER(PcmPaths), I64, I, I, I, I, P, I, P,
                                      SZ, P]
    L.pcm_dense_swiglu.argtypes = [I, P, P, P, P, I64, I, I, P, I, P, SZ, P]
    L.pcm_workspace_bytes.argtypes = [I, I64, I, I, I, I, I]
    L.pcm_workspace_bytes.restype = SZ
    L.pcm_status_string.argtypes = [I]
    L.pcm_status_string.restype = ctypes.c_char_p
    L.pcm_path_layout_build.argtypes = [P, P, I, ctypes.POINTER(PcmPathLayout), P]
    L.pcm_route_scored.argtypes = [P, P, ctypes.c_float, ctypes.POINTER(PcmPathLayout), I64, I, I,
                                   ctypes.POINTER(PcmScoredPaths), P, SZ, P]
    L.pcm_expand_scored.argtypes = [I, P, P, P, ctypes.POINTER(PcmScoredPaths), I64, I, I, I, I, P,
                                    P, SZ, P]
    L.pcm_project_combine_scored.argtypes = [I, P, P, ctypes.POINTER(PcmScoredPaths), I64, I, I, I,
                                             I, P, I, P, SZ, P]
    L.pcm_route_logits.argtypes = [I, P, P, I64, I, I, I, P, P, P, P, SZ, P]
    L.pcm_residual_add.argtypes = [I, P, P, I64, I, P]
    L.pcm_widen_f16.argtypes = [P, I64, P, P]
    L.pcm_layer_per_path.argtypes = [I, P, P, P, P, ctypes.POINTER(PcmPaths), I64, I, I, I, I, I, P,
                                     I, P, SZ, P]
    TP = ctypes.POINTER(PcmTuning)
    for name in ("pcm_expand", "pcm_project_combine", "pcm_dense_swiglu", "pcm_expand_scored",
                 "pcm_project_combine_scored"):
        getattr(L, name + "_tuned").argtypes = getattr(L, name).argtypes + [TP]
    L.pcm_project_combine_noalloc.argtypes = [I, P, P, ctypes.POINTER(PcmPaths), I64, I, I, I, I, P,
                                              I, P]
    SZP = ctypes.POINTER(SZ)
    L.pcm_project_workspace_layout.argtypes = [I, I64, I, I, I, I, TP, SZP, SZP, SZP,
                                               ctypes.POINTER(I)]
    for name in ("pcm_route", "pcm_build_paths", "pcm_expand", "pcm_project_combine",
                 "pcm_dense_swiglu", "pcm_abi_version", "pcm_path_layout_build",
                 "pcm_route_scored", "pcm_expand_scored", "pcm_project_combine_scored",
                 "pcm_layer_per_path", "pcm_route_logits", "pcm_residual_add",
                 "pcm_expand_tuned", "pcm_project_combine_tuned", "pcm_dense_swiglu_tuned",
                 "pcm_expand_scored_tuned", "pcm_project_combine_scored_tuned",
                 "pcm_project_workspace_layout", "pcm_project_combine_noalloc", "pcm_mask_pack",
                 "pcm_route_paths", "pcm_widen_f16"):
        getattr(L, name).restype = I
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise RuntimeError(lib().pcm_status_string(status).decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream: Optional[torch.cuda.Stream]):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _on(stream: Optional[torch.cuda.Stream]):
    """Context for allocating outputs and workspaces: on `stream` when one is given, so that the
    caching allocator orders their reuse after the kernels enqueued there."""
    return torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()


def _call(name: str, args: list, tuning):
    """The plain entry point, or its *_tuned form with the tuning (a Tuning, or a PcmTuning
    built beforehand) appended."""
    if tuning is None:
        return getattr(lib(), name)(*args)
    t = tuning if isinstance(tuning, PcmTuning) else tuning.struct()
    return getattr(lib(), name + "_tuned")(*args, ctypes.byref(t))


def project_workspace_layout(T: int, H: int, F: int, n: int, k: int, dtype: int,
                             tuning: Optional[Tuning] = None) -> dict:
    """Byte offsets of z, its row scales and o inside pcm_project_combine's workspace, and the
    number of K slices of o (pcm_project_workspace_layout)."""
    z, zs, o = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    ks = ctypes.c_int()
    t = tuning.struct() if tuning is not None else None
    _check(lib().pcm_project_workspace_layout(dtype, T, H, F, n, k,
                                              ctypes.byref(t) if t is not None else None,
                                              ctypes.byref(z), ctypes.byref(zs), ctypes.byref(o),
                                              ctypes.byref(ks)))
    return {"z": z.value, "zscale": zs.value, "o": o.value, "ksplit": ks.value}


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return PCM_BF16
    if t.dtype == torch.float32:
        return PCM_F32
    if t.dtype == torch.float16:   # projection weights widened once (pcm_widen_f16)
        return PCM_BF16_F16DOWN
    raise TypeError(f"unsupported dtype {t.dtype}")


def _layer_code(x: torch.Tensor, w_down: torch.Tensor) -> int:
    """Layer dtype of a call that takes both activations and projection weights."""
    if x.dtype == torch.bfloat16 and w_down.dtype == torch.float16:
        return PCM_BF16_F16DOWN
    return _dtype_code(x)


def _dev(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError("tensors must be contiguous device tensors")


def workspace_bytes(op: int, T: int, H: int, F: int, n: int, k: int, dtype: int) -> int:
    return int(lib().pcm_workspace_bytes(op, T, H, F, n, k, dtype))


def _workspace(nbytes: int, device) -> Optional[torch.Tensor]:
    return torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=device) if nbytes else None


# ------------------------------------------------------------------------ calls
def pcm_route(logits: torch.Tensor, k: int, topk_ids=None, topk_w=None, stream=None):
    _dev(logits)
    T, n = logits.shape
    with _on(stream):
        ids = topk_ids if topk_ids is not None else torch.empty((T, k), dtype=torch.int32, device=logits.device)
        w = topk_w if topk_w is not None else torch.empty((T, k), dtype=torch.float32, device=logits.device)
    _dev(ids, w)
    _check(lib().pcm_route(_ptr(logits), T, n, k, _ptr(ids), _ptr(w), _stream(stream)))
    return ids, w


def pcm_route_logits(x, w_router, k: int, logits=None, topk_ids=None, topk_w=None,
                     want_logits: bool = False, ws: torch.Tensor = None, stream=None):
    """Router GEMM fused with the top-k: returns (ids, w) or (ids, w, logits)."""
    _dev(x, w_router)
    T, H = x.shape
    n = w_router.shape[0]
    dev = x.device
    dt = _dtype_code(x)
    with _on(stream):
        ids = topk_ids if topk_ids is not None else torch.empty((T, k), dtype=torch.int32, device=dev)
        w = topk_w if topk_w is not None else torch.empty((T, k), dtype=torch.float32, device=dev)
        if want_logits and logits is None:
            logits = torch.empty((T, n), dtype=torch.float32, device=dev)
        if ws is None:
            ws = _workspace(workspace_bytes(OP_ROUTE_LOGITS, T, H, 0, n, k, dt), dev)
    _dev(ids, w, logits)
    _check(lib().pcm_route_logits(dt, _ptr(x), _ptr(w_router), T, H, n, k, _ptr(logits), _ptr(ids),
                                  _ptr(w), _ptr(ws), ws.numel() if ws is not None else 0,
                                  _stream(stream)))
    return (ids, w, logits) if want_logits else (ids, w)


def pcm_residual_add(h: torch.Tensor, y: torch.Tensor, stream=None) -> torch.Tensor:
    """h += y in place (rounded to h's dtype)."""
    _dev(h, y)
    T, H = h.shape
    _check(lib().pcm_residual_add(_dtype_code(h), _ptr(h), _ptr(y), T, H, _stream(stream)))
    return h


def pcm_widen_f16(w: torch.Tensor, out: torch.Tensor = None, stream=None) -> torch.Tensor:
    """Projection weights for PCM_BF16_F16DOWN: the bf16 tensor w rounded to float16 (to
    nearest even, as the projection kernels widen bf16 fragments). A layer passes the result
    as w_down; the projections then give the same bits as with w."""
    _dev(w, out)
    if w.dtype != torch.bfloat16 or not w.is_contiguous():
        raise TypeError("w must be a contiguous bfloat16 tensor")
    with _on(stream):
        out = out if out is not None else torch.empty(w.shape, dtype=torch.float16, device=w.device)
    if out.dtype != torch.float16 or out.shape != w.shape or not out.is_contiguous():
        raise TypeError("out must be a contiguous float16 tensor of w's shape")
    _check(lib().pcm_widen_f16(_ptr(w), w.numel(), _ptr(out), _stream(stream)))
    return out


@dataclass
class PathTable:
    """Device buffers of one pcm_paths layout for T tokens, n experts, top-k."""
    T: int
    n: int
    k: int
    path_bits: torch.Tensor
    beta: torch.Tensor
    expert_offsets: torch.Tensor
    row_token: torch.Tensor
    row_slot: torch.Tensor
    row_of: torch.Tensor

    @classmethod
    def empty(cls, T: int, n: int, k: int, device) -> "PathTable":
        i32 = dict(dtype=torch.int32, device=device)
        return cls(T, n, k, torch.empty((T,), dtype=torch.int64, device=device),
                   torch.empty((T, k, k), dtype=torch.float32, device=device),
                   torch.empty((n + 1,), **i32), torch.empty((T * k,), **i32),
                   torch.empty((T * k,), **i32), torch.empty((T, k), **i32))

    def struct(self) -> PcmPaths:
        return PcmPaths(self.path_bits.data_ptr(), self.beta.data_ptr(), self.expert_offsets.data_ptr(),
                        self.row_token.data_ptr(), self.row_slot.data_ptr(), self.row_of.data_ptr())


def pcm_build_paths(topk_ids, topk_w, mask, beta_mode: int = BETA_SRC_COND, out: PathTable = None,
                    ws: torch.Tensor = None, stream=None) -> PathTable:
    _dev(topk_ids, topk_w, mask)
    T, k = topk_ids.shape
    n = mask.shape[0]
    need = workspace_bytes(OP_BUILD_PATHS, T, 0, 0, n, k, 0)
    with _on(stream):
        out = out or PathTable.empty(T, n, k, topk_ids.device)
        if ws is None:
            ws = _workspace(need, topk_ids.device)
    st = out.struct()
    _check(lib().pcm_build_paths(_ptr(topk_ids), _ptr(topk_w), _ptr(mask), T, n, k, beta_mode,
                                 ctypes.byref(st), _ptr(ws), ws.numel() if ws is not None else 0,
                                 _stream(stream)))
    return out


def pcm_mask_pack(mask: torch.Tensor, packed: torch.Tensor = None, stream=None) -> torch.Tensor:
    """The layer's mask [n,n] u8 as the packed [n, ceil(n/64)] int64 bitset of pcm_route_paths
    (the diagonal set)."""
    _dev(mask)
    n = mask.shape[0]
    with _on(stream):
        packed = packed if packed is not None else torch.empty((n, (n + 63) // 64), dtype=torch.int64,
                                                               device=mask.device)
    _dev(packed)
    _check(lib().pcm_mask_pack(_ptr(mask), n, _ptr(packed), _stream(stream)))
    return packed


def route_paths_workspace(T: int, n: int, k: int, device) -> torch.Tensor:
    """A workspace for pcm_route_paths, zero-filled (its completion counter starts at zero and
    every call leaves it there, so the workspace can be reused as it is)."""
    return torch.zeros((workspace_bytes(OP_ROUTE_PATHS, T, 0, 0, n, k, 0),), dtype=torch.uint8,
                       device=device)


def pcm_route_paths(logits, packed_mask, k: int, beta_mode: int = BETA_SRC_COND, topk_ids=None,
                    topk_w=None, out: PathTable = None, ws: torch.Tensor = None, stream=None):
    """Fused indexing: (topk_ids, topk_w, PathTable) from the logits and a packed mask."""
    _dev(logits, packed_mask)
    T, n = logits.shape
    dev = logits.device
    need = workspace_bytes(OP_ROUTE_PATHS, T, 0, 0, n, k, 0)
    with _on(stream):
        ids = topk_ids if topk_ids is not None else torch.empty((T, k), dtype=torch.int32, device=dev)
        w = topk_w if topk_w is not None else torch.empty((T, k), dtype=torch.float32, device=dev)
        out = out or PathTable.empty(T, n, k, dev)
        if ws is None:
            ws = route_paths_workspace(T, n, k, dev)
    _dev(ids, w)
    st = out.struct()
    _check(lib().pcm_route_paths(_ptr(logits), _ptr(packed_mask), T, n, k, beta_mode, _ptr(ids),
                                 _ptr(w), ctypes.byref(st), _ptr(ws),
                                 ws.numel() if ws is not None else 0, _stream(stream)))
    return ids, w, out


def pcm_expand(x, w_gate, w_up, paths: PathTable, u=None, stream=None,
               tuning: Optional[Tuning] = None) -> torch.Tensor:
    _dev(x, w_gate, w_up, u)
    T, H = x.shape
    n, F, _ = w_gate.shape
    with _on(stream):
        u = u if u is not None else torch.empty((T * paths.k, F), dtype=torch.float32, device=x.device)
    st = paths.struct()
    _check(_call("pcm_expand", [_dtype_code(x), _ptr(x), _ptr(w_gate), _ptr(w_up), ctypes.byref(st),
                                T, H, F, n, paths.k, _ptr(u), None, 0, _stream(stream)], tuning))
    return u


def pcm_project_combine(u, w_down, paths: PathTable, y=None, accumulate: bool = False,
                        ws: torch.Tensor = None, stream=None,
                        tuning: Optional[Tuning] = None) -> torch.Tensor:
    _dev(u, w_down, y)
    n, H, F = w_down.shape
    T, k = paths.T, paths.k
    dt = _dtype_code(w_down)
    with _on(stream):
        y = y if y is not None else torch.empty((T, H), dtype=torch.float32, device=u.device)
        if ws is None:
            ws = _workspace(workspace_bytes(OP_PROJECT_COMBINE, T, H, F, n, k, dt), u.device)
    st = paths.struct()
    _check(_call("pcm_project_combine", [dt, _ptr(u), _ptr(w_down), ctypes.byref(st), T, H, F, n, k,
                                         _ptr(y), int(bool(accumulate)), _ptr(ws),
                                         ws.numel() if ws is not None else 0, _stream(stream)],
                 tuning))
    return y


def pcm_project_combine_noalloc(u, w_down, paths: PathTable, y=None, accumulate: bool = False,
                                stream=None) -> torch.Tensor:
    """pcm_project_combine with the library's own per-GPU scratch instead of a workspace."""
    _dev(u, w_down, y)
    n, H, F = w_down.shape
    T, k = paths.T, paths.k
    with _on(stream):
        y = y if y is not None else torch.empty((T, H), dtype=torch.float32, device=u.device)
    st = paths.struct()
    _check(lib().pcm_project_combine_noalloc(_dtype_code(w_down), _ptr(u), _ptr(w_down),
                                             ctypes.byref(st), T, H, F, n, k, _ptr(y),
                                             int(bool(accumulate)), _stream(stream)))
    return y


def pcm_dense_swiglu(x, w_gate, w_up, w_down, y=None, accumulate: bool = False,
                     ws: torch.Tensor = None, stream=None,
                     tuning: Optional[Tuning] = None) -> torch.Tensor:
    _dev(x, w_gate, w_up, w_down, y)
    T, H = x.shape
    Fs = w_gate.shape[0]
    dt = _layer_code(x, w_down)
    with _on(stream):
        y = y if y is not None else torch.empty((T, H), dtype=torch.float32, device=x.device)
        if ws is None:
            ws = _workspace(workspace_bytes(OP_DENSE_SWIGLU, T, H, Fs, 1, 1, dt), x.device)
    _check(_call("pcm_dense_swiglu", [dt, _ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(w_down), T, H, Fs,
                                      _ptr(y), int(bool(accumulate)), _ptr(ws),
                                      ws.numel() if ws is not None else 0, _stream(stream)], tuning))
    return y


def pcm_layer_per_path(x, w_gate, w_up, w_down, paths: PathTable, reuse: bool = True, y=None,
                       accumulate: bool = False, ws: torch.Tensor = None, stream=None) -> torch.Tensor:
    """Per-path execution (baseline): one projection per path; reuse=False also expands
    once per path."""
    _dev(x, w_gate, w_up, w_down, y)
    T, H = x.shape
    n, F, _ = w_gate.shape
    k = paths.k
    dt = _layer_code(x, w_down)
    with _on(stream):
        y = y if y is not None else torch.empty((T, H), dtype=torch.float32, device=x.device)
        if ws is None:
            ws = _workspace(workspace_bytes(OP_LAYER_PER_PATH, T, H, F, n, k, dt), x.device)
    st = paths.struct()
    _check(lib().pcm_layer_per_path(dt, _ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(w_down),
                                    ctypes.byref(st), T, H, F, n, k, int(bool(reuse)), _ptr(y),
                                    int(bool(accumulate)), _ptr(ws),
                                    ws.numel() if ws is not None else 0, _stream(stream)))
    return y


# --------------------------------------------------------------- scored routing
@dataclass
class PathLayout:
    """Device buffers of one layer's active-pair layout (n experts)."""
    n: int
    count: torch.Tensor
    pair: torch.Tensor
    bias: torch.Tensor

    @classmethod
    def empty(cls, n: int, device) -> "PathLayout":
        return cls(n, torch.empty((1,), dtype=torch.int32, device=device),
                   torch.empty((n * n,), dtype=torch.int32, device=device),
                   torch.empty((n * n,), dtype=torch.float32, device=device))

    def struct(self) -> PcmPathLayout:
        return PcmPathLayout(self.count.data_ptr(), self.pair.data_ptr(), self.bias.data_ptr())


def pcm_path_layout_build(mask, bias, out: PathLayout = None, stream=None) -> PathLayout:
    _dev(mask, bias)
    n = mask.shape[0]
    if bias.dtype != torch.float32 or bias.shape != (n, n) or mask.dtype != torch.uint8:
        raise TypeError("mask [n,n] uint8 and bias [n,n] float32")
    with _on(stream):
        out = out or PathLayout.empty(n, mask.device)
    st = out.struct()
    _check(lib().pcm_path_layout_build(_ptr(mask), _ptr(bias), n, ctypes.byref(st), _stream(stream)))
    return out


@dataclass
class ScoredPathTable:
    """Device buffers of one pcm_scored_paths for T tokens, n experts, K paths."""
    T: int
    n: int
    K: int
    sel_pair: torch.Tensor
    sel_score: torch.Tensor
    n_src: torch.Tensor
    src_expert: torch.Tensor
    n_tgt: torch.Tensor
    tgt_expert: torch.Tensor
    path_bits: torch.Tensor
    beta: torch.Tensor
    src_offsets: torch.Tensor
    src_row_token: torch.Tensor
    src_row_slot: torch.Tensor
    src_row_of: torch.Tensor
    tgt_offsets: torch.Tensor
    tgt_row_token: torch.Tensor
    tgt_row_slot: torch.Tensor
    tgt_row_of: torch.Tensor

    @classmethod
    def empty(cls, T: int, n: int, K: int, device) -> "ScoredPathTable":
        i32 = dict(dtype=torch.int32, device=device)
        e = lambda *shape, **kw: torch.empty(shape, **(kw or i32))
        return cls(T, n, K, e(T, K), e(T, K, dtype=torch.float32, device=device), e(T), e(T, K), e(T),
                   e(T, K), e(T, dtype=torch.int64, device=device),
                   e(T, K, K, dtype=torch.float32, device=device),
                   e(n + 1), e(T * K), e(T * K), e(T, K), e(n + 1), e(T * K), e(T * K), e(T, K))

    def struct(self) -> PcmScoredPaths:
        return PcmScoredPaths(*[getattr(self, f).data_ptr() for f in _SCORED_FIELDS])


def pcm_route_scored(g_base, g_tgt, lam: float, layout: PathLayout, K: int,
                     out: ScoredPathTable = None, ws: torch.Tensor = None,
                     stream=None) -> ScoredPathTable:
    _dev(g_base, g_tgt)
    T, n = g_base.shape
    with _on(stream):
        out = out or ScoredPathTable.empty(T, n, K, g_base.device)
        if ws is None:
            ws = _workspace(workspace_bytes(OP_ROUTE_SCORED, T, 0, 0, n, K, 0), g_base.device)
    lst, st = layout.struct(), out.struct()
    _check(lib().pcm_route_scored(_ptr(g_base), _ptr(g_tgt), float(lam), ctypes.byref(lst), T, n, K,
                                  ctypes.byref(st), _ptr(ws), ws.numel() if ws is not None else 0,
                                  _stream(stream)))
    return out


def pcm_expand_scored(x, w_gate, w_up, paths: ScoredPathTable, u=None, stream=None,
                      tuning: Optional[Tuning] = None) -> torch.Tensor:
    _dev(x, w_gate, w_up, u)
    T, H = x.shape
    n, F, _ = w_gate.shape
    with _on(stream):
        u = u if u is not None else torch.empty((T * paths.K, F), dtype=torch.float32, device=x.device)
    st = paths.struct()
    _check(_call("pcm_expand_scored", [_dtype_code(x), _ptr(x), _ptr(w_gate), _ptr(w_up),
                                       ctypes.byref(st), T, H, F, n, paths.K, _ptr(u), None, 0,
                                       _stream(stream)], tuning))
    return u


def pcm_project_combine_scored(u, w_down, paths: ScoredPathTable, y=None, accumulate: bool = False,
                               ws: torch.Tensor = None, stream=None,
                               tuning: Optional[Tuning] = None) -> torch.Tensor:
    _dev(u, w_down, y)
    n, H, F = w_down.shape
    T, K = paths.T, paths.K
    dt = _dtype_code(w_down)
    with _on(stream):
        y = y if y is not None else torch.empty((T, H), dtype=torch.float32, device=u.device)
        if ws is None:
            ws = _workspace(workspace_bytes(OP_PROJECT_COMBINE, T, H, F, n, K, dt), u.device)
    st = paths.struct()
    _check(_call("pcm_project_combine_scored", [dt, _ptr(u), _ptr(w_down), ctypes.byref(st), T, H, F,
                                                n, K, _ptr(y), int(bool(accumulate)), _ptr(ws),
                                                ws.numel() if ws is not None else 0,
                                                _stream(stream)], tuning))
    return y


def capture_graph(fn) -> "torch.cuda.CUDAGraph":
    """A HIP graph of fn() (a layer plan's forward on fixed tensors, whose contents are read at
    every replay): graph.replay() then enqueues the whole layer as one launch on the current
    stream, without the host-side cost of each call. fn runs once eagerly on a side stream first
    (so every lazy initialisation happens outside the capture). A plan's forward allocates
    nothing and clears nothing (no memset nodes), so the graph holds kernel nodes only."""
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    with torch.cuda.graph(g):
        fn()
    return g


class ScoredLayerPlan:
    """Preallocated buffers for the scored-routing layer (forward enqueues kernels only).
    The active-pair layout is built once per layer (build_layout)."""

    def __init__(self, T, H, F, n, K, dtype: torch.dtype, device, shared_F: int = 0):
        self.T, self.H, self.F, self.n, self.K, self.shared_F = T, H, F, n, K, shared_F
        dt = PCM_BF16 if dtype == torch.bfloat16 else PCM_F32
        self.layout = PathLayout.empty(n, device)
        self.paths = ScoredPathTable.empty(T, n, K, device)
        self.ws_route = _workspace(workspace_bytes(OP_ROUTE_SCORED, T, 0, 0, n, K, 0), device)
        self.u = torch.empty((T * K, F), dtype=torch.float32, device=device)
        self.ws_proj = _workspace(workspace_bytes(OP_PROJECT_COMBINE, T, H, F, n, K, dt), device)
        self.ws_shared = (_workspace(workspace_bytes(OP_DENSE_SWIGLU, T, H, shared_F, 1, 1, dt), device)
                          if shared_F else None)
        self.y = torch.empty((T, H), dtype=torch.float32, device=device)

    def build_layout(self, mask, bias, stream=None):
        pcm_path_layout_build(mask, bias, out=self.layout, stream=stream)

    def forward(self, x, g_base, g_tgt, lam, w_gate, w_up, w_down, shared=None, stream=None,
                tuning: Optional[Tuning] = None):
        # the shared expert first, storing y; the combine then adds the routed sum to it
        # (y_t = shared_t + routed_t either way, the same two float32 operands)
        if shared is not None:
            pcm_dense_swiglu(x, *shared, y=self.y, accumulate=False, ws=self.ws_shared, stream=stream,
                             tuning=tuning)
        pcm_route_scored(g_base, g_tgt, lam, self.layout, self.K, out=self.paths, ws=self.ws_route,
                         stream=stream)
        pcm_expand_scored(x, w_gate, w_up, self.paths, u=self.u, stream=stream, tuning=tuning)
        pcm_project_combine_scored(self.u, w_down, self.paths, y=self.y, accumulate=shared is not None,
                                   ws=self.ws_proj, stream=stream, tuning=tuning)
        return self.y

    def capture(self, x, g_base, g_tgt, lam, w_gate, w_up, w_down, shared=None,
                tuning: Optional[Tuning] = None) -> "torch.cuda.CUDAGraph":
        """forward() on these tensors as a HIP graph (capture_graph); replay() writes self.y."""
        return capture_graph(lambda: self.forward(x, g_base, g_tgt, lam, w_gate, w_up, w_down, shared,
                                                  tuning=tuning))


class LayerPlan:
    """Preallocated buffers for repeated forward passes of one layer shape, so that a
    forward pass enqueues kernels only (no allocation)."""

    def __init__(self, T, H, F, n, k, dtype: torch.dtype, device, shared_F: int = 0,
                 beta_mode: int = BETA_SRC_COND):
        self.T, self.H, self.F, self.n, self.k, self.shared_F = T, H, F, n, k, shared_F
        self.beta_mode = beta_mode
        dt = PCM_BF16 if dtype == torch.bfloat16 else PCM_F32
        self.ids = torch.empty((T, k), dtype=torch.int32, device=device)
        self.w = torch.empty((T, k), dtype=torch.float32, device=device)
        self.paths = PathTable.empty(T, n, k, device)
        self.ws_paths = _workspace(workspace_bytes(OP_BUILD_PATHS, T, 0, 0, n, k, 0), device)
        self.ws_index = route_paths_workspace(T, n, k, device)
        self.u = torch.empty((T * k, F), dtype=torch.float32, device=device)
        self.ws_proj = _workspace(workspace_bytes(OP_PROJECT_COMBINE, T, H, F, n, k, dt), device)
        self.ws_shared = (_workspace(workspace_bytes(OP_DENSE_SWIGLU, T, H, shared_F, 1, 1, dt), device)
                          if shared_F else None)
        self.y = torch.empty((T, H), dtype=torch.float32, device=device)

    def index(self, logits, mask, stream=None):
        """Route and build the path table: one fused operation when `mask` is the packed
        int64 layout of pcm_mask_pack, else pcm_route then pcm_build_paths over the u8 mask."""
        if mask.dtype == torch.int64:
            pcm_route_paths(logits, mask, self.k, self.beta_mode, self.ids, self.w, out=self.paths,
                            ws=self.ws_index, stream=stream)
        else:
            pcm_route(logits, self.k, self.ids, self.w, stream=stream)
            pcm_build_paths(self.ids, self.w, mask, self.beta_mode, out=self.paths, ws=self.ws_paths,
                            stream=stream)

    def forward(self, x, logits, mask, w_gate, w_up, w_down, shared=None, stream=None,
                tuning: Optional[Tuning] = None):
        # the shared expert first, storing y (its projection's epilogue then has no y to read);
        # the combine adds the routed sum: y_t = shared_t + routed_t, the same two float32
        # operands as accumulating the shared expert last
        if shared is not None:
            pcm_dense_swiglu(x, *shared, y=self.y, accumulate=False, ws=self.ws_shared, stream=stream,
                             tuning=tuning)
        self.index(logits, mask, stream)
        pcm_expand(x, w_gate, w_up, self.paths, u=self.u, stream=stream, tuning=tuning)
        pcm_project_combine(self.u, w_down, self.paths, y=self.y, accumulate=shared is not None,
                            ws=self.ws_proj, stream=stream, tuning=tuning)
        return self.y

    def capture(self, x, logits, mask, w_gate, w_up, w_down, shared=None,
                tuning: Optional[Tuning] = None) -> "torch.cuda.CUDAGraph":
        """forward() on these tensors as a HIP graph (capture_graph); replay() writes self.y.
        With the packed mask (pcm_mask_pack) of T <= 64 tokens the indexing's completion counter
        returns to zero at the end of every replay, as after every eager call."""
        return capture_graph(lambda: self.forward(x, logits, mask, w_gate, w_up, w_down, shared,
                                                  tuning=tuning))


def layer_forward(x, logits, mask, w_gate, w_up, w_down, k: int, beta_mode: int = BETA_SRC_COND,
                  shared=None, stream=None, tuning: Optional[Tuning] = None) -> torch.Tensor:
    """One layer: route, build paths, expand, project and combine (+ shared expert)."""
    T, H = x.shape
    n, F, _ = w_gate.shape
    with _on(stream):
        plan = LayerPlan(T, H, F, n, k, x.dtype, x.device, shared[0].shape[0] if shared else 0,
                         beta_mode)
    return plan.forward(x, logits, mask, w_gate, w_up, w_down, shared, stream, tuning)
