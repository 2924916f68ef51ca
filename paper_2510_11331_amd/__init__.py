"""MI355X-native speculative-decoding hot path (arXiv 2510.11331).

libsd (HIP kernels for gfx950 behind the C ABI of include/sd.h) does all the
work; this package holds its ctypes binding and a host driver that provides
device memory and streams through PyTorch.
"""
from ._lib import SDError, lib  # noqa: F401
from .engine import (SDEngine, Batch, GPUModel, StepGraph, generate, generate_graph,  # noqa: F401
                     emitted_tokens, accept_resample, resume_prompts)
