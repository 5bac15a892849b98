"""Layer configurations.

The five named workloads are synthetic stand-ins for the MoE layers the paper
evaluates during decoding (Mixtral-8x7B, Qwen1.5-MoE-A2.7B, DeepSeek-V2-Lite;
Section 5.1 "Models"), plus a tiny fp32 case and a decode-shaped case. No model
weights or datasets are used: every tensor is drawn from a seeded generator
with the shape and distribution listed here.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class LayerConfig:
    name: str
    T: int            # tokens
    H: int            # hidden size
    n: int            # routed experts
    F: int            # SwiGLU intermediate size of one routed expert
    k: int            # experts selected per token
    dtype: str        # "f32" or "bf16": dtype of x, the weights and the intermediates
    density: float    # off-diagonal compatibility-mask density (diagonal always kept)
    logits: str       # "router" | "normal" | "normal_bias" | "zipf"
    x_std: float      # standard deviation of the hidden states x
    w_std: float = 0.02
    shared_F: int = 0         # intermediate size of the always-on shared expert (0: none)
    bias_std: float = 0.0     # per-expert logit bias std ("normal_bias")
    zipf_s: float = 0.0       # Zipf exponent ("zipf")

    @property
    def R(self) -> int:
        """Expansion rows: one per (token, selected expert)."""
        return self.T * self.k


CONFIGS = {
    # 64 tokens, hidden 256, 8 experts, ffn 512, top-2, fp32; logits from a
    # router matrix W_r ~ N(0, 0.02^2) applied to x ~ N(0, 0.02^2).
    "tiny": LayerConfig("tiny", 64, 256, 8, 512, 2, "f32", 0.5, "router", x_std=0.02),
    # Mixtral-8x7B-shaped layer: logits N(0,1) plus a per-expert bias N(0, 0.5^2).
    "mixtral": LayerConfig("mixtral", 4096, 4096, 8, 14336, 2, "bf16", 0.5, "normal_bias",
                           x_std=1.0, bias_std=0.5),
    # OLMoE-shaped layer: Zipf-skewed logits (s = 1.1) across 64 experts.
    "olmoe": LayerConfig("olmoe", 8192, 2048, 64, 1024, 8, "bf16", 0.25, "zipf",
                         x_std=1.0, zipf_s=1.1),
    # Fine-grained layer with 60 routed experts and one always-on shared expert.
    "finegrained_shared": LayerConfig("finegrained_shared", 16384, 2048, 60, 1408, 4, "bf16",
                                      0.3, "normal", x_std=1.0, shared_F=5632),
    # Decode-shaped layer: 32 tokens, 256 experts; bound by streaming expert weights.
    "decode": LayerConfig("decode", 32, 7168, 256, 2048, 8, "bf16", 0.2, "normal", x_std=1.0),
}

# The workload the layer throughput is quoted on.
HEADLINE = "mixtral"


def scaled(cfg: LayerConfig, **changes) -> LayerConfig:
    """A copy of `cfg` with some sizes changed (same distributions and structure)."""
    name = changes.pop("name", None) or cfg.name + "_" + "_".join(f"{k}{v}" for k, v in changes.items())
    return replace(cfg, name=name, **changes)


def stress_config(kind: str, base: LayerConfig) -> LayerConfig:
    """Stress variants: 'ties' quantises logits so exact ties are common,
    'one_expert' sends every token to expert 0 first (rows of expert 0 = T)."""
    if kind not in ("ties", "one_expert"):
        raise ValueError(kind)
    return replace(base, name=f"{base.name}_{kind}", logits=f"{base.logits}+{kind}")
