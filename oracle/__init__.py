"""Oracle for the speculative-decoding hot path: TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct CPU implementation of what the GPU path
computes, written from the paper (arXiv 2510.11331, Section II-A "Inference
Mechanism with SD") and from the textbook definitions it relies on.  Floating
point is float64 throughout, except where the model definition itself fixes a
narrower type (bf16 storage points of a bf16 model, float32 distributions fed
to the sampling rule).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
and must never be used as a fallback for it.

Modules
  model     LLaMA-style decoder (RMSNorm, rotary embedding, GQA attention,
            SwiGLU) with a per-layer KV cache; decode and prefill.
  sampling  softmax, the integer inverse-CDF sampling rule, the speculative
            acceptance / residual-resampling rule.
  sd        the draft -> verify -> accept -> rollback loop and plain
            autoregressive decoding.
  exact     exact laws of the implemented sampling rules (for pins).
  sched     the serving scheduler's cost and latency model, the batching
            dynamic program and the speculation-length search, and the
            closed-form uplink allocation.

Parity pins: every function here is pinned by ``tests/test_oracle_*.py``
against closed forms, library routines (torch CPU), brute force or the
distribution-preservation property of speculative sampling.
"""
from . import model, sampling, sd, exact, sched  # noqa: F401
