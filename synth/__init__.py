"""Seeded synthetic inputs for the TADM reverse-diffusion step.

This module is the only code shared between the CPU oracle and the GPU path.  It
holds workload shapes and random-number plumbing and none of the method's
arithmetic: model shapes, the fixed tensor order of the weights, seeded weight
tensors, prompts, canvases and logits.

Weights follow the random-init recipe N(0, 0.02^2) for every matrix, norm gains 1
and biases 0 (the paired-attention gate bias b_g is -3, the fusion init stated in
the paper's post-training setup).  Unlike the paper's training init, the fusion
output projections (W2 of the gated MLP, W_up of paired attention) are random, not
zero, so that the fusion path is exercised.  ``perturb=True`` additionally draws
norm gains and biases around their defaults so that a dropped gain or bias shows
up in parity tests.
"""
from .configs import CONFIGS, MASK_OFFSET, get_config, mask_id  # noqa: F401
from .weights import weight_specs, make_weights, make_tensor, tensor_seed  # noqa: F401
from .inputs import (make_prompt, make_timing_canvas, make_logits,  # noqa: F401
                     make_teacher_canvas)
