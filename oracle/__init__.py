"""CPU oracle for speculative sampling (Chen et al., 2023, "Accelerating Large
Language Model Decoding with Speculative Sampling").

This package is TEST INFRASTRUCTURE. It is a plain, slow, obviously-correct
numpy implementation of what the GPU path computes. It exists so that the GPU
path can be checked against something written straight from the paper. Only
``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it; the product path never does.

It shares no code with the HIP library: no kernels, headers, helpers, tables
or constants. The only thing both sides consume is data made by the seeded
input generators in ``paper_2302_01318_amd.synth``.

Modules:
  philox    Philox4x64-10 counter-based uniforms (Salmon et al., SC'11).
  sampling  softmax with temperature, fixed-point weights, categorical draw.
  accept    modified rejection sampling (Algorithm 2; Modified Rejection
            Sampling section; Theorem 1).
  model     decoder-only transformer forward, full recompute and KV-cached
            (Conditional Scoring section).
  generate  the SpS loop (Algorithm 2) and ArS (Algorithm 1).
  fp8       weight-only FP8 (OCP E4M3, one fp32 scale per output row)
            quantisation of the projection matrices.

Every function is pinned by tests under ``tests/`` that check it against
what the paper and mathematics fix. The one function without such a pin is
listed in its module header as "parity unpinned".
"""
from . import philox, sampling, accept, model, generate, fp8  # noqa: F401
