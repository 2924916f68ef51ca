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
                  keep_logits=False, first_step=0):
    """Prefill, then n_steps SD steps of one batch on the current stream,
    with the uniforms of steps first_step .. first_step + n_steps - 1.
    Returns (per-task emitted tokens, n_acc [n_steps, B], batch, logits
    [n_steps, B, gamma+1, V] or None)."""
    import torch
    from paper_2510_11331_amd import emitted_tokens
    from paper_2510_11331_amd.engine import uniforms_device
    B = len(slots)
    max_new = max_new or [n_steps * (gamma + 1)] * B
    eng.prefill(slots, prompts, max_new)
    b = eng.batch(slots, gamma)
    u = uniforms_device(synth.uniform_table(seed, task_ids, first_step + n_steps, gamma)[first_step:])
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


def greedy_stream_report(target, prompts, emitted, acc, logits, n_new, bound, tie=1e-3):
    """Greedy stream of a GPU run against the oracle target, teacher-forced
    on the GPU's own emitted prefix (so the comparison resynchronises after
    any divergence).  emitted: per task the GPU's tokens; acc [steps, B] and
    logits [steps, B, gamma+1, V] of the run: rows 0..a of a step are the
    logits that chose its emitted tokens.  Asserts, at every position of the
    first n_new tokens of every task: the GPU token is the arg-max of the
    GPU row (lowest index on ties); the row is within `bound` of the plain
    and of the rounded oracle's (per-row max abs error over max abs); where
    the token is not the plain oracle's arg-max, the oracle's top-2 gap is
    a near tie (< tie) or is covered by the two tokens' logit errors.
    Returns the counts and the gaps of the divergences."""
    B = len(prompts)
    rows = [[] for _ in range(B)]                 # GPU logits of each emitted position
    for n in range(acc.shape[0]):
        for k in range(B):
            for j in range(int(acc[n, k]) + 1):
                if len(rows[k]) < n_new:
                    rows[k].append(logits[n, k, j])
    toks = [list(emitted[k][:n_new]) for k in range(B)]
    assert all(len(r) == n_new and len(t) == n_new for r, t in zip(rows, toks))
    seqs = [list(prompts[k]) + toks[k][:-1] for k in range(B)]
    ref = {"plain": target.unrounded().sequence_logits(seqs, n_new), "rounded": target.sequence_logits(seqs, n_new)}
    worst = {f: 0.0 for f in ref}
    near, div, div_gaps = 0, 0, []
    for k in range(B):
        for i in range(n_new):
            z = np.asarray(rows[k][i], dtype=np.float64)
            assert toks[k][i] == osp.argmax_lowest(z), (k, i)
            for f, zz in ref.items():
                worst[f] = max(worst[f], float(np.abs(z - zz[k][i]).max() / np.abs(zz[k][i]).max()))
            zr = ref["plain"][k][i]
            o = osp.argmax_lowest(zr)
            if o == toks[k][i]:
                continue
            gap = top2_gap(zr)
            if gap < tie:
                near += 1
                continue
            dz = np.abs(z - zr)
            assert gap <= dz[o] + dz[toks[k][i]] + 1e-9, (k, i, gap, dz[o], dz[toks[k][i]])
            div += 1
            div_gaps.append(round(gap, 4))
    for f, e in worst.items():
        assert e < bound, (f, e)
    return {"positions": B * n_new, "near_ties": near, "divergences": div, "divergence_gaps": sorted(div_gaps),
            "worst_rel_logit_err": worst}
