"""pcm_project_combine_noalloc (the allocation-free variant that keeps z and o in the
library's per-GPU scratch array) against pcm_project_combine with a caller workspace: the
same kernels on the same inputs, so the outputs must be the same bits. Two calls in a row,
the second on a smaller input, show that what the first call left in the scratch does not
leak into the second."""
import sys

import numpy as np
import pytest
import torch

import paper_2609_01024_amd as pcm
from workloads import CONFIGS, make_inputs, scaled

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def expanded(cfg, seed):
    """Route, path table and U of a layer (the inputs of the project-and-combine call)."""
    inp = make_inputs(cfg, seed=seed)
    x = inp.x.to(DEV)
    ids, w = pcm.pcm_route(torch.from_numpy(inp.logits).to(DEV), cfg.k)
    p = pcm.pcm_build_paths(ids, w, torch.from_numpy(inp.mask).to(DEV))
    u = pcm.pcm_expand(x, inp.w_gate.to(DEV), inp.w_up.to(DEV), p)
    return p, u, inp.w_down.to(DEV)


DECODE_S = scaled(CONFIGS["decode"], H=2048, F=1024, n=64, name="decode_noalloc")
CASES = {
    # decode-shaped bf16 layer (32 tokens, then 16), and the fp32 tiny layer (64, then 24)
    "bf16": (DECODE_S, scaled(DECODE_S, T=16, name="decode_noalloc16")),
    "f32": (CONFIGS["tiny"], scaled(CONFIGS["tiny"], T=24, name="tiny24")),
}


@pytest.mark.parametrize("kind", sorted(CASES))
def test_noalloc_matches_workspace_call(kind):
    for i, cfg in enumerate(CASES[kind]):
        say(f"no-alloc {kind}: call {i} T={cfg.T}")
        p, u, wd = expanded(cfg, seed=40 + i)
        ref = pcm.pcm_project_combine(u, wd, p)
        y = pcm.pcm_project_combine_noalloc(u, wd, p, y=torch.full_like(ref, float("nan")))
        base = torch.randn_like(ref)
        ref_acc = pcm.pcm_project_combine(u, wd, p, y=base.clone(), accumulate=True)
        y_acc = pcm.pcm_project_combine_noalloc(u, wd, p, y=base.clone(), accumulate=True)
        torch.cuda.synchronize()
        assert torch.isfinite(ref).all()
        assert torch.equal(y, ref), f"{cfg.name}: differs from the workspace call"
        assert torch.equal(y_acc, ref_acc), f"{cfg.name}: accumulate differs"


def test_noalloc_rejects_sizes_beyond_its_scratch():
    cfg = scaled(CONFIGS["olmoe"], T=2048, H=512, F=256, n=8, k=8, name="too_big")
    p, u, wd = expanded(cfg, seed=45)
    need = pcm.workspace_bytes(pcm.binding.OP_PROJECT_COMBINE, cfg.T, cfg.H, cfg.F, cfg.n, cfg.k,
                               pcm.PCM_BF16)
    assert need > 16 << 20
    y = torch.zeros((cfg.T, cfg.H), device=DEV)
    with pytest.raises(RuntimeError, match="UNSUPPORTED"):
        pcm.pcm_project_combine_noalloc(u, wd, p, y=y)
    torch.cuda.synchronize()
    assert not y.any(), "a rejected call must not write its output"
