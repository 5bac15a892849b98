"""The C ABI library loads, exports every symbol the header declares, and rejects
invalid arguments on the host before touching a device (no GPU needed)."""
import ctypes
import os
import re

import pytest

import paper_2609_01024_amd as pcm
from paper_2609_01024_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pcomoe.h")

OK, ARG, UNSUP, WS, HIP = 0, 1, 2, 3, 4


def declared_functions():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return sorted(set(re.findall(r"\b(pcm_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return pcm.lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert set(names) == set(binding.EXPORTS), names
    for name in names:
        assert hasattr(L, name), name


def test_abi_version_and_status_strings(L):
    assert L.pcm_abi_version() == 123
    for s in (OK, ARG, UNSUP, WS, HIP):
        assert L.pcm_status_string(s).decode().startswith("PCM_")
    assert L.pcm_status_string(77) == b"unknown pcm_status"


FAKE = ctypes.c_void_p(0x10000)  # never dereferenced: validation fails first


def test_route_validation(L):
    assert L.pcm_route(FAKE, 4, 8, 9, FAKE, FAKE, None) == ARG       # k > n
    assert L.pcm_route(FAKE, 4, 8, 0, FAKE, FAKE, None) == ARG       # k < 1
    assert L.pcm_route(FAKE, -1, 8, 2, FAKE, FAKE, None) == ARG      # T < 0
    assert L.pcm_route(FAKE, 4, 300, 2, FAKE, FAKE, None) == UNSUP   # n > 256
    assert L.pcm_route(FAKE, 4, 16, 9, FAKE, FAKE, None) == UNSUP    # k > 8
    assert L.pcm_route(None, 4, 8, 2, FAKE, FAKE, None) == ARG       # null
    assert L.pcm_route(ctypes.c_void_p(0x10004), 4, 8, 2, FAKE, FAKE, None) == ARG  # misaligned
    assert L.pcm_route(None, 0, 8, 2, None, None, None) == OK        # T = 0 no-op
    assert L.pcm_route(FAKE, 1 << 29, 8, 8, FAKE, FAKE, None) == UNSUP  # T*k >= 2^31


def _paths(null_field=None):
    vals = {f: 0x10000 for f, _ in binding.PcmPaths._fields_}
    if null_field:
        vals[null_field] = 0
    return binding.PcmPaths(**vals)


def test_build_paths_validation(L):
    p = _paths()
    assert L.pcm_build_paths(FAKE, FAKE, FAKE, 4, 8, 2, 3, ctypes.byref(p), None, 0, None) == ARG
    for f, _ in binding.PcmPaths._fields_:
        q = _paths(f)
        assert L.pcm_build_paths(FAKE, FAKE, FAKE, 4, 8, 2, 0, ctypes.byref(q), None, 0, None) == ARG
    need = L.pcm_workspace_bytes(binding.OP_BUILD_PATHS, 5000, 0, 0, 64, 8, 0)
    assert need > 0
    assert L.pcm_build_paths(FAKE, FAKE, FAKE, 5000, 64, 8, 0, ctypes.byref(p), FAKE, need - 1,
                             None) == WS
    assert L.pcm_build_paths(FAKE, FAKE, FAKE, 0, 64, 8, 0, None, None, 0, None) == OK


def test_expand_and_project_validation(L):
    p = _paths()
    bp = ctypes.byref(p)
    assert L.pcm_expand(1, FAKE, FAKE, FAKE, bp, 4, 100, 128, 8, 2, FAKE, None, 0, None) == UNSUP
    assert L.pcm_expand(1, FAKE, FAKE, FAKE, bp, 4, 128, 96, 8, 2, FAKE, None, 0, None) == UNSUP
    assert L.pcm_expand(7, FAKE, FAKE, FAKE, bp, 4, 128, 128, 8, 2, FAKE, None, 0, None) == ARG
    assert L.pcm_expand(1, FAKE, None, FAKE, bp, 4, 128, 128, 8, 2, FAKE, None, 0, None) == ARG
    assert L.pcm_expand(1, FAKE, FAKE, FAKE, None, 4, 128, 128, 8, 2, FAKE, None, 0, None) == ARG
    need = L.pcm_workspace_bytes(binding.OP_PROJECT_COMBINE, 4, 128, 128, 8, 2, 1)
    al = lambda v: (v + 255) // 256 * 256
    R = 4 * 2
    assert need == al(R * 128 * 2) + al(R * 4) + al(R * 128 * 4)      # z f16, scales, o
    assert L.pcm_workspace_bytes(binding.OP_PROJECT_COMBINE, 4, 128, 128, 8, 2, 0) == \
        al(R * 128 * 4) + al(R * 128 * 4)                                  # f32 layer: z f32, o
    assert L.pcm_project_combine(1, FAKE, FAKE, bp, 4, 128, 128, 8, 2, FAKE, 0, FAKE, need - 1,
                                 None) == WS
    assert L.pcm_project_combine(1, FAKE, FAKE, bp, 4, 128, 128, 8, 2, FAKE, 0, None, need,
                                 None) == WS
    assert L.pcm_project_combine(1, FAKE, FAKE, bp, 4, 128, 128, 8, 9, FAKE, 0, FAKE, need,
                                 None) == ARG
    needd = L.pcm_workspace_bytes(binding.OP_DENSE_SWIGLU, 16, 128, 256, 1, 1, 1)
    assert needd == 16 * 256 * 4 + 16 * 256 * 2 + 256                     # u f32, z f16, scales
    assert L.pcm_dense_swiglu(1, FAKE, FAKE, FAKE, FAKE, 16, 128, 256, FAKE, 0, FAKE, needd - 1,
                              None) == WS
    assert L.pcm_dense_swiglu(1, FAKE, FAKE, FAKE, FAKE, 16, 128, 200, FAKE, 0, FAKE, needd,
                              None) == UNSUP
    assert L.pcm_dense_swiglu(1, None, None, None, None, 0, 128, 256, None, 0, None, 0, None) == OK


def test_build_paths_rejects_misaligned_pointers(L):
    p = _paths()
    need = L.pcm_workspace_bytes(binding.OP_BUILD_PATHS, 5000, 0, 0, 64, 8, 0)
    mis = ctypes.c_void_p(0x10004)
    for i in range(3):   # topk_ids, topk_w, mask
        args = [FAKE, FAKE, FAKE]
        args[i] = mis
        assert L.pcm_build_paths(*args, 5000, 64, 8, 0, ctypes.byref(p), FAKE, need, None) == ARG
    for f, _ in binding.PcmPaths._fields_:
        vals = {g: 0x10000 for g, _ in binding.PcmPaths._fields_}
        vals[f] = 0x10008
        q = binding.PcmPaths(**vals)
        assert L.pcm_build_paths(FAKE, FAKE, FAKE, 5000, 64, 8, 0, ctypes.byref(q), FAKE, need,
                                 None) == ARG, f
    assert L.pcm_build_paths(FAKE, FAKE, FAKE, 5000, 64, 8, 0, ctypes.byref(p), mis, need,
                             None) == ARG                                    # workspace


def test_widen_f16_and_f16down_dtype(L):
    mis = ctypes.c_void_p(0x10008)
    assert L.pcm_widen_f16(FAKE, -1, FAKE, None) == ARG
    assert L.pcm_widen_f16(None, 0, None, None) == OK                 # count 0: no-op
    assert L.pcm_widen_f16(None, 8, FAKE, None) == ARG
    assert L.pcm_widen_f16(FAKE, 8, None, None) == ARG
    assert L.pcm_widen_f16(mis, 8, FAKE, None) == ARG
    assert L.pcm_widen_f16(FAKE, 8, mis, None) == ARG
    # a bf16 layer with float16 projection weights needs the same workspaces as a bf16 layer
    for op in (binding.OP_PROJECT_COMBINE, binding.OP_DENSE_SWIGLU, binding.OP_LAYER_PER_PATH,
               binding.OP_ROUTE_LOGITS):
        assert (L.pcm_workspace_bytes(op, 1000, 1024, 2048, 16, 4, binding.PCM_BF16_F16DOWN) ==
                L.pcm_workspace_bytes(op, 1000, 1024, 2048, 16, 4, binding.PCM_BF16)), op
    p = _paths()
    need = L.pcm_workspace_bytes(binding.OP_PROJECT_COMBINE, 100, 256, 256, 8, 2, 1)
    for dt, want in ((3, ARG), (-1, ARG)):
        assert L.pcm_project_combine(dt, FAKE, FAKE, ctypes.byref(p), 100, 256, 256, 8, 2, FAKE, 0,
                                     FAKE, need, None) == want, dt


def test_mask_pack_and_route_paths_validation(L):
    mis = ctypes.c_void_p(0x10008)
    assert L.pcm_mask_pack(FAKE, 0, FAKE, None) == ARG                 # n < 1
    assert L.pcm_mask_pack(FAKE, 300, FAKE, None) == UNSUP             # n > 256
    assert L.pcm_mask_pack(None, 8, FAKE, None) == ARG
    assert L.pcm_mask_pack(FAKE, 8, mis, None) == ARG                  # misaligned packed
    p = _paths()
    bp = ctypes.byref(p)
    # 256 bytes of completion counter, then (T > 64) the counts [ceil(T / 32)][n] i32
    assert L.pcm_workspace_bytes(binding.OP_ROUTE_PATHS, 64, 0, 0, 256, 8, 0) == 256
    assert L.pcm_workspace_bytes(binding.OP_ROUTE_PATHS, 65, 0, 0, 60, 4, 0) == 256 + 768
    need = L.pcm_workspace_bytes(binding.OP_ROUTE_PATHS, 8192, 0, 0, 64, 8, 0)
    assert need == 256 + 256 * 64 * 4
    args = lambda T=8192, n=64, k=8, beta=0, q=bp, ws=FAKE, wsb=need: (
        FAKE, FAKE, T, n, k, beta, FAKE, FAKE, q, ws, wsb, None)
    assert L.pcm_route_paths(*args(k=9)) == UNSUP                      # k > 8
    assert L.pcm_route_paths(*args(n=300)) == UNSUP                    # n > 256
    assert L.pcm_route_paths(*args(n=4)) == ARG                        # k > n
    assert L.pcm_route_paths(*args(beta=3)) == ARG
    assert L.pcm_route_paths(*args(wsb=need - 1)) == WS
    assert L.pcm_route_paths(*args(ws=None)) == WS
    assert L.pcm_route_paths(*args(T=64, ws=None, wsb=0)) == WS      # the counter is needed
    assert L.pcm_route_paths(*args(ws=mis)) == ARG
    assert L.pcm_route_paths(*args(T=0, q=None, ws=None, wsb=0)) == OK  # T = 0 no-op
    for f, _ in binding.PcmPaths._fields_:
        q = _paths(f)
        assert L.pcm_route_paths(*args(q=ctypes.byref(q))) == ARG, f
        vals = {g: 0x10000 for g, _ in binding.PcmPaths._fields_}
        vals[f] = 0x10008
        q = binding.PcmPaths(**vals)
        assert L.pcm_route_paths(*args(q=ctypes.byref(q))) == ARG, f
    for i in (0, 1, 6, 7):  # logits, packed mask, topk_ids, topk_w
        a = list(args())
        a[i] = None
        assert L.pcm_route_paths(*a) == ARG, i
        a[i] = mis
        assert L.pcm_route_paths(*a) == ARG, i


def test_tuning_validation(L):
    p = _paths()
    bp = ctypes.byref(p)
    args = (1, FAKE, FAKE, FAKE, bp, 4, 128, 128, 8, 2, FAKE, None, 0, None)
    for field, bad in (("tile", ord("X")), ("order_expand", 3), ("order_down", -2),
                       ("em_window", -1), ("group_n", -1), ("stream_depth", 5)):
        t = binding.Tuning().struct()
        setattr(t, field, bad)
        assert L.pcm_expand_tuned(*args, ctypes.byref(t)) == ARG, field
        assert L.pcm_project_workspace_layout(1, 4, 128, 128, 8, 2, ctypes.byref(t),
                                              *(ctypes.byref(ctypes.c_size_t()) for _ in range(3)),
                                              ctypes.byref(ctypes.c_int())) == ARG, field
    # a valid tuning passes validation (T = 0 is a no-op), NULL tuning is the plain call
    for tile in ("S", "M", "L", "W"):
        t = binding.Tuning(tile=tile, order_expand=2, em_window=5, stream_depth=0).struct()
        assert L.pcm_expand_tuned(1, None, None, None, None, 0, 128, 128, 8, 2, None, None, 0, None,
                                  ctypes.byref(t)) == OK, tile
    # the K split follows the tile family: the large tiles on four or eight waves split, the
    # medium tiles do not
    for tile, ks in (("L", 2), ("W", 2), ("M", 1)):
        assert binding.project_workspace_layout(300, 256, 4096, 4, 2, binding.PCM_BF16,
                                                binding.Tuning(tile=tile))["ksplit"] == ks, tile
    assert L.pcm_expand_tuned(1, FAKE, FAKE, FAKE, bp, 4, 100, 128, 8, 2, FAKE, None, 0, None,
                              None) == UNSUP


def test_noalloc_validation(L):
    """The allocation-free projection: the same argument checks as pcm_project_combine, and
    sizes whose workspace exceeds its 16 MiB scratch rejected before any device call."""
    p = _paths()
    bp = ctypes.byref(p)
    assert L.pcm_project_combine_noalloc(1, FAKE, FAKE, bp, 2048, 512, 256, 8, 8, FAKE, 0,
                                         None) == UNSUP       # needs 40 MiB
    assert L.pcm_project_combine_noalloc(1, FAKE, FAKE, bp, 4096, 4096, 14336, 8, 2, FAKE, 0,
                                         None) == UNSUP
    assert L.pcm_project_combine_noalloc(1, None, FAKE, bp, 32, 2048, 1024, 64, 8, FAKE, 0,
                                         None) == ARG
    assert L.pcm_project_combine_noalloc(1, FAKE, FAKE, None, 32, 2048, 1024, 64, 8, FAKE, 0,
                                         None) == ARG
    assert L.pcm_project_combine_noalloc(1, ctypes.c_void_p(0x10004), FAKE, bp, 32, 2048, 1024,
                                         64, 8, FAKE, 0, None) == ARG
    assert L.pcm_project_combine_noalloc(1, FAKE, FAKE, bp, 32, 2000, 1024, 64, 8, FAKE, 0,
                                         None) == UNSUP       # H not a multiple of 64
    assert L.pcm_project_combine_noalloc(1, None, None, None, 0, 2048, 1024, 64, 8, None, 0,
                                         None) == OK          # T = 0


def test_project_workspace_layout(L):
    al = lambda v: (v + 255) // 256 * 256
    T, H, F, n, k = 4, 128, 128, 8, 2
    R = T * k
    lay = binding.project_workspace_layout(T, H, F, n, k, binding.PCM_BF16)
    assert lay == {"z": 0, "zscale": al(R * F * 2), "o": al(R * F * 2) + al(R * 4), "ksplit": 1}
    need = L.pcm_workspace_bytes(binding.OP_PROJECT_COMBINE, T, H, F, n, k, 1)
    assert need == lay["o"] + al(lay["ksplit"] * R * H * 4)
    lay = binding.project_workspace_layout(T, H, F, n, k, binding.PCM_F32)
    assert lay == {"z": 0, "zscale": 0, "o": al(R * F * 4), "ksplit": 1}
    # a long F with few output tiles: two K slices of o, unless a forced tile kernel runs
    big = binding.project_workspace_layout(300, 256, 4096, 4, 2, binding.PCM_BF16)
    assert big["ksplit"] == 2
    assert binding.project_workspace_layout(300, 256, 4096, 4, 2, binding.PCM_BF16,
                                            binding.Tuning(tile="M"))["ksplit"] == 1


def test_workspace_bytes_invalid(L):
    assert L.pcm_workspace_bytes(binding.OP_PROJECT_COMBINE, -1, 128, 128, 8, 2, 1) == 0
    assert L.pcm_workspace_bytes(binding.OP_BUILD_PATHS, 256, 0, 0, 8, 2, 0) == 0  # one block
    assert L.pcm_workspace_bytes(binding.OP_BUILD_PATHS, 257, 0, 0, 8, 2, 0) == 256  # 2 blocks x 8


def test_scored_validation(L):
    lay = binding.PcmPathLayout(0x10000, 0x10000, 0x10000)
    assert L.pcm_path_layout_build(FAKE, FAKE, 300, ctypes.byref(lay), None) == UNSUP   # n > 256
    assert L.pcm_path_layout_build(FAKE, FAKE, 0, ctypes.byref(lay), None) == ARG       # n < 1
    assert L.pcm_path_layout_build(None, FAKE, 8, ctypes.byref(lay), None) == ARG       # null
    bad = binding.PcmPathLayout(0x10000, 0, 0x10000)
    assert L.pcm_path_layout_build(FAKE, FAKE, 8, ctypes.byref(bad), None) == ARG
    sp = binding.PcmScoredPaths(*([0x10000] * len(binding._SCORED_FIELDS)))
    spp = ctypes.byref(sp)
    assert L.pcm_route_scored(FAKE, FAKE, 0.5, ctypes.byref(lay), 4, 8, 9, spp, None, 0, None) == ARG    # K > n
    assert L.pcm_route_scored(FAKE, FAKE, 0.5, ctypes.byref(lay), 4, 16, 9, spp, None, 0, None) == UNSUP  # K > 8
    assert L.pcm_route_scored(FAKE, FAKE, float("nan"), ctypes.byref(lay), 4, 8, 2, spp, None, 0, None) == ARG
    assert L.pcm_route_scored(FAKE, FAKE, float("inf"), ctypes.byref(lay), 4, 8, 2, spp, None, 0, None) == ARG
    assert L.pcm_route_scored(None, None, 0.5, None, 0, 8, 2, None, None, 0, None) == OK   # T = 0
    for f in range(len(binding._SCORED_FIELDS)):                  # every field is required
        vals = [0x10000] * len(binding._SCORED_FIELDS)
        vals[f] = 0
        q = binding.PcmScoredPaths(*vals)
        assert L.pcm_route_scored(FAKE, FAKE, 0.5, ctypes.byref(lay), 4, 8, 2, ctypes.byref(q), None,
                                  0, None) == ARG, binding._SCORED_FIELDS[f]
    need = L.pcm_workspace_bytes(binding.OP_ROUTE_SCORED, 5000, 0, 0, 64, 8, 0)
    assert need == 2 * L.pcm_workspace_bytes(binding.OP_BUILD_PATHS, 5000, 0, 0, 64, 8, 0) > 0
    assert L.pcm_route_scored(FAKE, FAKE, 0.5, ctypes.byref(lay), 5000, 64, 8, spp, FAKE, need - 1,
                              None) == WS
    assert L.pcm_expand_scored(1, FAKE, FAKE, FAKE, spp, 4, 100, 128, 8, 2, FAKE, None, 0, None) == UNSUP
    assert L.pcm_expand_scored(1, FAKE, FAKE, FAKE, None, 4, 128, 128, 8, 2, FAKE, None, 0, None) == ARG
    needp = L.pcm_workspace_bytes(binding.OP_PROJECT_COMBINE, 4, 128, 128, 8, 2, 1)
    assert L.pcm_project_combine_scored(1, FAKE, FAKE, spp, 4, 128, 128, 8, 2, FAKE, 0, FAKE,
                                        needp - 1, None) == WS
    assert L.pcm_project_combine_scored(1, FAKE, FAKE, spp, 4, 128, 128, 8, 9, FAKE, 0, FAKE,
                                        needp, None) == ARG


def test_per_path_validation(L):
    bp = binding.PcmPaths(0x10000, 0x10000, 0x10000, 0x10000, 0x10000, 0x10000)
    need = L.pcm_workspace_bytes(binding.OP_LAYER_PER_PATH, 4, 128, 128, 8, 2, 1)
    assert need > 4 * 2 * 2 * (128 * 4 + 128 * 2 + 128 * 4)   # U, z and o for T*k*k paths
    args = (1, FAKE, FAKE, FAKE, FAKE, ctypes.byref(bp), 4, 128, 128, 8, 2, 1, FAKE, 0)
    assert L.pcm_layer_per_path(*args, FAKE, need - 1, None) == WS
    assert L.pcm_layer_per_path(*args, None, need, None) == WS
    assert L.pcm_layer_per_path(1, FAKE, FAKE, FAKE, FAKE, None, 4, 128, 128, 8, 2, 1, FAKE, 0,
                                FAKE, need, None) == ARG
    assert L.pcm_layer_per_path(1, FAKE, FAKE, FAKE, FAKE, ctypes.byref(bp), 1 << 26, 128, 128, 64,
                                8, 1, FAKE, 0, FAKE, need, None) == UNSUP       # T*k*k >= 2^31
    assert L.pcm_layer_per_path(1, None, None, None, None, None, 0, 128, 128, 8, 2, 0, None, 0,
                                None, 0, None) == OK


def test_route_logits_validation(L):
    need = L.pcm_workspace_bytes(binding.OP_ROUTE_LOGITS, 4, 128, 0, 8, 2, 1)
    assert need > 0 and L.pcm_workspace_bytes(binding.OP_ROUTE_LOGITS, 4, 128, 0, 8, 2, 0) == 0
    args = (FAKE, FAKE, 4, 128, 8, 2, None, FAKE, FAKE, FAKE, need, None)
    assert L.pcm_route_logits(7, *args) == ARG                                   # dtype
    assert L.pcm_route_logits(1, FAKE, FAKE, 4, 100, 8, 2, None, FAKE, FAKE, FAKE, need, None) == UNSUP
    assert L.pcm_route_logits(1, FAKE, FAKE, 4, 128, 8, 9, None, FAKE, FAKE, FAKE, need, None) == ARG
    assert L.pcm_route_logits(1, None, FAKE, 4, 128, 8, 2, None, FAKE, FAKE, FAKE, need, None) == ARG
    assert L.pcm_route_logits(1, FAKE, FAKE, 4, 128, 8, 2, ctypes.c_void_p(0x10004), FAKE, FAKE,
                              FAKE, need, None) == ARG                           # misaligned logits
    assert L.pcm_route_logits(1, FAKE, FAKE, 4, 128, 8, 2, None, FAKE, FAKE, FAKE, need - 1,
                              None) == WS
    assert L.pcm_route_logits(1, None, None, 0, 128, 8, 2, None, None, None, None, 0, None) == OK
