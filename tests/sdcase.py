"""Shared helpers of the GPU parity tests: build a libsd engine and the
oracle models on the same seeded weights, run both, and compare."""
from __future__ import annotations

import sys
from typing import List, Optional

import numpy as np

import synth
from oracle import model as om, sampling as osp, sd as osd


def say(*a):
    """Progress line naming the case, flushed before each GPU step."""
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def weights(shape, seed):
    return synth.model_weights(shape, seed)


def make_engine(tshape, dshape, tw, dw, *, max_slots, max_batch, gamma_max, max_ctx,
                prefill_rows=256, temperature=1.0, greedy=False):
    from paper_2510_11331_amd import SDEngine
    return SDEngine(tshape, dshape, tw.__getitem__, dw.__getitem__, max_slots=max_slots,
                    max_batch=max_batch, gamma_max=gamma_max, max_ctx=max_ctx,
                    prefill_rows=prefill_rows, temperature=temperature, greedy=greedy)


def top2_gap(z: np.ndarray) -> float:
    s = np.sort(np.asarray(z, dtype=np.float64))
    return float(s[-1] - s[-2])


def run_gpu_steps(eng, slots, prompts, gamma, n_steps, seed, task_ids, max_new=None,
                  keep_logits=False):
    """Prefill, then n_steps SD steps of one batch on the current stream.
    Returns (per-task emitted tokens, n_acc [n_steps, B], batch, logits
    [n_steps, B, gamma+1, V] or None)."""
    import torch
    from paper_2510_11331_amd import emitted_tokens
    from paper_2510_11331_amd.engine import uniforms_device
    B = len(slots)
    max_new = max_new or [n_steps * (gamma + 1)] * B
    eng.prefill(slots, prompts, max_new)
    b = eng.batch(slots, gamma)
    u = uniforms_device(synth.uniform_table(seed, task_ids, n_steps, gamma))
    z = torch.empty(B, gamma + 1, eng.vocab, dtype=torch.float32, device="cuda") if keep_logits else None
    accs, outs, logs = [], [], []
    for n in range(n_steps):
        eng.step(b, u[n], None, logits=z)
        accs.append(b.n_acc.clone())
        outs.append(b.out_tok.clone())
        if keep_logits:
            logs.append(z.clone())
    torch.cuda.synchronize()
    acc = torch.stack(accs).cpu().numpy()
    out = torch.stack(outs).cpu().numpy()
    lg = torch.stack(logs).cpu().numpy() if keep_logits else None
    return emitted_tokens(acc, out), acc, b, lg


def oracle_sd(target, draft, prompt, gamma, n_tokens, seed, task_id, tau, greedy, batch_rows=False,
              records=None):
    steps = n_tokens + 2
    ut = synth.uniform_table(seed, [task_id], steps, gamma)[:, 0]
    return osd.sd_generate(target, draft, prompt, gamma, n_tokens, ut, tau=tau, greedy=greedy,
                           batch_rows=batch_rows, records=records)


def compare_greedy(gpu_tokens: List[int], ref_tokens: List[int], ref_logits: np.ndarray, tie=1e-3):
    """Greedy comparison with near-tie accounting: identical tokens, except
    that the first divergence is tolerated (and ends the comparison) when the
    oracle's top-2 logit gap at that position is below `tie`.  Returns
    (n_compared, near_tie_or_None); raises on a real mismatch."""
    n = min(len(gpu_tokens), len(ref_tokens))
    for i in range(n):
        if gpu_tokens[i] != ref_tokens[i]:
            gap = top2_gap(ref_logits[i])
            if gap < tie:
                return i, gap
            raise AssertionError(f"greedy token {i}: gpu {gpu_tokens[i]} oracle {ref_tokens[i]} "
                                 f"(oracle top-2 gap {gap:.3g})")
    return n, None
