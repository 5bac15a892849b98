"""The layer captured as a HIP graph (LayerPlan.capture, ScoredLayerPlan.capture) against the eager
calls, through the C ABI (needs an MI355X).

A graph is replayed several times with eager work and synchronisations between the replays, and
every replay must give the bits of the eager forward on the same inputs. y is filled with NaN
before each replay, so an element the replay does not write shows. Then the inputs change in place
and a replay must give the bits of an eager forward, on a second plan, over the new inputs (the
graph reads the tensors' current contents). No pcm call allocates or clears memory, so the
graphs hold kernel nodes only; the T <= 64 indexing's completion counter returns to zero at the
end of each replay (decode_s, packed mask), so consecutive replays agree.
"""
import sys

import pytest
import torch

import paper_2609_01024_amd as pcm
from workloads import make_inputs

from test_gpu_parity import SMALL, dev
from test_gpu_scored import scored_inputs

pytestmark = pytest.mark.gpu
DEV = "cuda"


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def eager_work():
    """Other work on the current stream between replays, and a synchronisation."""
    a = torch.randn((1 << 20,), device=DEV)
    return float((a * 2).sum().item())


def new_inputs(d, seed):
    """The same shapes with other values, copied into d's tensors in place."""
    g = torch.Generator(device=DEV).manual_seed(seed)
    d["x"].copy_((torch.randn(d["x"].shape, generator=g, device=DEV)).to(d["x"].dtype))
    d["logits"].copy_(torch.randn(d["logits"].shape, generator=g, device=DEV))


@pytest.mark.parametrize("packed", [True, False])
@pytest.mark.parametrize("name", ["tiny", "olmoe_s", "fine_s", "decode_s", "splitk_s", "wide_s"])
def test_layer_graph_replays_bit_identical(name, packed):
    cfg = SMALL[name]
    say(f"graph replay {name} packed={packed}")
    d = dev(make_inputs(cfg, seed=51))
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    mask = pcm.pcm_mask_pack(d["mask"]) if packed else d["mask"]
    shared = d.get("shared")

    def args():
        return (d["x"], d["logits"], mask, d["w_gate"], d["w_up"], d["w_down"], shared)

    plan = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, dtype, DEV, cfg.shared_F)
    eager = plan.forward(*args()).clone()
    torch.cuda.synchronize()
    assert torch.isfinite(eager).all()
    graph = plan.capture(*args())
    for i in range(4):
        plan.y.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(plan.y.view(torch.int32), eager.view(torch.int32)), f"replay {i}"
        eager_work()
    new_inputs(d, 52)
    ref = pcm.LayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, dtype, DEV, cfg.shared_F)
    expected = ref.forward(*args()).clone()
    torch.cuda.synchronize()
    assert not torch.equal(expected, eager)
    plan.y.fill_(float("nan"))
    graph.replay()
    torch.cuda.synchronize()
    assert torch.equal(plan.y.view(torch.int32), expected.view(torch.int32)), "new inputs"


@pytest.mark.parametrize("name", ["olmoe_s", "decode_s"])
def test_scored_layer_graph_replays_bit_identical(name):
    cfg = SMALL[name]
    say(f"scored graph replay {name}")
    inp, s = scored_inputs(cfg, 53)
    d = dev(inp)
    g_tgt = torch.from_numpy(s.g_tgt).to(DEV)
    plan = pcm.ScoredLayerPlan(cfg.T, cfg.H, cfg.F, cfg.n, cfg.k, torch.bfloat16, DEV, cfg.shared_F)
    plan.build_layout(d["mask"], torch.from_numpy(s.bias).to(DEV))

    def args():
        return (d["x"], d["logits"], g_tgt, s.lam, d["w_gate"], d["w_up"], d["w_down"], d.get("shared"))

    eager = plan.forward(*args()).clone()
    torch.cuda.synchronize()
    assert torch.isfinite(eager).all()
    graph = plan.capture(*args())
    for i in range(3):
        plan.y.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(plan.y.view(torch.int32), eager.view(torch.int32)), f"replay {i}"
        eager_work()
