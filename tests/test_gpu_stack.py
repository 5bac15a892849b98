"""A stack of MoE layers with residual connections (multi-layer decode steps) against the
CPU oracle, layer by layer (needs an MI355X).

Each layer's output is checked against the oracle layer evaluated on the same bf16 hidden
states and on the router logits the kernel computed (the top-k decision is taken on those
float32 values); the residual update must equal round_bf16(h + y) bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_01024_amd as pcm
from paper_2609_01024_amd.stack import MoEStack, StackLayer, random_stack
from workloads import CONFIGS, make_inputs, make_router_weights, scaled

from test_gpu_parity import assert_y_close

pytestmark = pytest.mark.gpu
DEV = "cuda"


def host_stack(cfg, L, native=2):
    layers, host = [], []
    for l in range(L):
        c = cfg if l >= native else scaled(cfg, density=0.0, name=f"{cfg.name}_native")
        inp = make_inputs(c, seed=100 + l)
        wr = make_router_weights(c, seed=100 + l)
        layers.append(StackLayer(wr.to(DEV), inp.w_gate.to(DEV), inp.w_up.to(DEV),
                                 inp.w_down.to(DEV), torch.from_numpy(inp.mask).to(DEV)))
        host.append(inp)
    return layers, host


@pytest.mark.parametrize("name,L", [("decode_s", 3), ("olmoe_s", 3), ("tiny", 4)])
def test_stack_layer_by_layer(name, L):
    from test_gpu_parity import SMALL
    cfg = SMALL[name]
    cfg = scaled(cfg, T=min(cfg.T, 96), name=cfg.name + "_stack")
    layers, host = host_stack(cfg, L)
    st = MoEStack(layers, cfg.T, cfg.k)
    h = host[0].x.to(DEV).clone()
    for l in range(L):
        h_in = h.cpu().clone()
        y = st.layer_step(l, h, keep_logits=True)
        torch.cuda.synchronize()
        lg = st.logits.cpu().numpy()
        inp = host[l]
        ref = oracle.layer(h_in, lg, inp.w_gate, inp.w_up, inp.w_down, inp.mask, cfg.k)
        assert_y_close(y.cpu().numpy(), ref, cfg.dtype, f"{name} layer {l}")
        expect = (h_in.float() + y.cpu()).to(h_in.dtype)
        assert torch.equal(h.cpu(), expect), f"residual {name} layer {l}"


def test_random_stack_runs_and_is_deterministic():
    cfg = CONFIGS["decode"]
    st = random_stack(2, 32, 512, 256, 64, 8, 0.2, seed=3, device=DEV)
    x = (torch.randn((32, 512), generator=torch.Generator().manual_seed(0)) * 1.0).to(torch.bfloat16)
    a = st.forward(x.to(DEV).clone())
    b = st.forward(x.to(DEV).clone())
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.isfinite(a.float()).all()
    assert cfg.k == 8


@pytest.mark.parametrize("L", [1, 3])
def test_stack_graph_replays_bit_identical(L):
    """The stack's decode step as one HIP graph (MoEStack.capture): each replay, from the same
    hidden states and with eager work and synchronisations between replays, must give the bits of
    the eager step; the graph holds kernel nodes only (no memsets)."""
    st = random_stack(L, 32, 512, 256, 64, 8, 0.2, seed=5, device=DEV)
    x0 = (torch.randn((32, 512), generator=torch.Generator().manual_seed(1)) * 1.0).to(torch.bfloat16).to(DEV)
    h = x0.clone()
    eager = st.forward(h).clone()
    torch.cuda.synchronize()
    assert torch.isfinite(eager.float()).all() and not torch.equal(eager, x0)
    graph = st.capture(h)
    for i in range(3):
        h.copy_(x0)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(h, eager), f"replay {i}"
        float((torch.randn((1 << 16,), device=DEV) * 3).sum().item())   # other work, a sync
