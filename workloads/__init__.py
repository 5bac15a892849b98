"""Seeded synthetic inputs for the path-compositional MoE layer.

This module is shared by the CPU oracle's tests and by the HIP path's tests and
benchmark. It holds the layer configurations and the random-number recipes
only; it contains none of the layer's arithmetic (no routing, no path
construction, no SwiGLU), so neither side of a parity check can borrow the
other's math through it.
"""
from .configs import LayerConfig, CONFIGS, HEADLINE, scaled, stress_config  # noqa: F401
from .gen import LayerInputs, ScoredInputs, make_inputs, make_router_weights, make_scored_inputs, quantise_logits  # noqa: F401
