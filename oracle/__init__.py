"""CPU oracle for TADM's reverse-diffusion step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct NumPy implementation of what the GPU path
computes, written from the paper:

* ``network``  -- shared embedding S, transformer layers, anchor network A, the two
  fusion modules Phi (gated residual MLP, App. C.2; paired attention, App. C.1),
  denoiser D and vocabulary head, in float64 (Sec. 3.1, eq. DenoiserOp);
* ``sampler``  -- the masked-diffusion reverse step with confidence-ranked
  unmasking: Philox4x32-10 keyed Gumbel-max sampling and a fixed-point confidence,
  whose decisions are taken in float32, the precision the GPU kernel uses
  (App. B.1.1, MDLM zero-masking and carry-over);
* ``loop``     -- anchor-cache inference (Algorithm 1) with the linear unmask
  schedule and block diffusion with a context KV, the remasking samplers (ReMDM-Cap
  and ReMDM-Loop) and the uniform-state generation of Algorithm 2;
* ``usdm``     -- the entropy-bound sampler of Algorithm 2: temperature schedule,
  Gumbel-max draw, fixed-point entropy, entropy-bound acceptance, uniform re-noising
  and the self-conditioning signal;
* ``train``    -- the pretraining objective (Theorem T-ANELBO with gamma = 0, sigma = 0):
  training times with stale anchors, the corrupted pair (z_t, z_t') and the
  1/t-weighted masked cross-entropy.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline``
leg may import this package.  It shares no code with the GPU path; the only common
dependency is the seeded input module ``synth``.
"""
from . import network, sampler, loop, usdm, train  # noqa: F401
