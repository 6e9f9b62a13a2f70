"""Seeded synthetic inputs for the speculative-verify path.

This package is the only code shared by the CPU oracle and the HIP path.  It
generates model weights, prompts, draft tokens, draft distributions, uniforms
and context lengths from a seed, and holds none of the verifier's arithmetic
(no forward pass, no acceptance rule, no sampler).

The paper (SPADE, arXiv 2608.13076) evaluates with real LLaMA weights on
Spec-Bench and CNN/DailyMail; neither the weights nor the datasets are used.
These shapes and distributions stand in for them.
"""

from .configs import ModelShape, Workload, WORKLOADS, workload, mini_workloads  # noqa: F401
from .weights import (  # noqa: F401
    WEIGHT_KINDS,
    LAYER_KINDS,
    GLOBAL_KINDS,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    tensor_shape,
    make_tensor,
    iter_weights,
    iter_weights_perturbed,
    perturb_tensor,
    ModelWeights,
)
from .inputs import make_inputs, VerifyInputs  # noqa: F401
