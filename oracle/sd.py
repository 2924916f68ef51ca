"""Oracle speculative-decoding loop and plain autoregressive decoding
(test infrastructure only).

One decoding step for one task (Section II-A): the draft model generates
gamma tokens autoregressively with its KV cache (drafting phase), the target
("verify") model scores the current input plus the gamma drafts in one pass
(verification phase), the acceptance rule of ``sampling.accept_resample``
emits the accepted prefix plus one bonus token, and the rejected drafts are
removed from both KV caches.  The bonus token is the input of the next step.

Readings where the paper is silent:
  * The prompt minus its last token is prefilled into both caches; every step
    starts from one un-cached input token x0 at position P (for the first
    step, the last prompt token).  The verify pass scores x0, t_1..t_gamma at
    positions P..P+gamma.
  * The draft consumed x0, t_1..t_{gamma-1}; after the step its cache keeps
    min(a+1, gamma) of them.  When all gamma drafts are accepted, t_gamma was
    never fed to the draft, so the next step's draft input is [t_gamma, y].
  * Uniform slots per (task, step): 0..gamma-1 draft samples, gamma..2gamma-1
    acceptance tests, 2gamma the residual / reward sample.
  * Emitted tokens beyond a task's budget are discarded (whole steps are run).
  * Forced acceptance (a workload rule, not part of the method: it sets the
    acceptance rate alpha of eq. ol from outside on random-weight models):
    under greedy verification, draft t_{i+1} is replaced, after the draft
    produced it and before the draft consumes it, by the token a reference
    continuation holds at its position P + 1 + i when the slot's draft
    uniform u_i (unused by greedy drafting) is below alpha 2^32.
"""
from __future__ import annotations

import math

from typing import Dict, List, Optional, Sequence

import numpy as np

from .model import Model, KVCache
from .sampling import accept_resample, draft_sample, softmax_f32, argmax_lowest, sample_weights


def force_threshold(alpha: float) -> int:
    """alpha as a bound on a uint32 uniform (forced iff u < bound):
    alpha 2^32 rounded to the nearest integer, halves away from zero."""
    assert 0.0 <= alpha <= 1.0
    return int(math.floor(alpha * 4294967296.0 + 0.5))


class SDTask:
    """Per-task state of the SD loop (both caches, the pending draft input)."""

    def __init__(self, target: Model, draft: Model, prompt: Sequence[int],
                 batch_rows: bool = False):
        prompt = [int(t) for t in prompt]
        assert len(prompt) >= 1
        self.target, self.draft = target, draft
        self.tc = target.prefill(prompt[:-1], batch_rows)
        self.dc = draft.prefill(prompt[:-1], batch_rows)
        self.x0 = prompt[-1]
        self.pending: List[int] = []        # draft inputs before x0 (t_gamma after full acceptance)
        self.emitted: List[int] = []
        self.n_steps = 0
        self.accepted: List[int] = []

    @property
    def P(self) -> int:
        return len(self.tc)

    def step(self, gamma: int, u: np.ndarray, tau: float = 1.0, greedy: bool = False,
             batch_rows: bool = False, record: Optional[dict] = None, force: Optional[tuple] = None):
        """One draft -> verify -> accept -> rollback step with the uniform
        vector u [2*gamma+1] (uint32).  force = (continuation by absolute
        position, force_threshold(alpha)) applies forced acceptance (greedy
        only).  Returns (a, emitted tokens)."""
        P = self.P
        # drafting: pending inputs then x0, then t_1..t_{gamma-1}
        feed = self.pending + [self.x0]
        assert len(self.dc) == P - len(self.pending)
        for i, t in enumerate(feed):
            z = self.draft.decode_row(self.dc, t, len(self.dc))
        drafts, qs = [], []
        assert force is None or greedy
        for i in range(gamma):
            t, q = draft_sample(z, tau, int(u[i]), greedy)
            if force is not None:
                cont, bound = force
                pos = P + 1 + i
                if int(u[i]) < bound and pos < len(cont):
                    t = int(cont[pos])
            drafts.append(t)
            qs.append(q)
            if i < gamma - 1:
                z = self.draft.decode_row(self.dc, t, P + 1 + i)
        # verification: x0, t_1..t_gamma at positions P..P+gamma
        rows = [self.x0] + drafts
        if batch_rows:
            logits = self.target.forward_rows(self.tc, rows)
        else:
            logits = np.stack([self.target.decode_row(self.tc, t, P + i) for i, t in enumerate(rows)])
        ps = logits.astype(np.float32) if greedy else softmax_f32(logits, tau)
        a, out = accept_resample(drafts, np.stack(qs), ps, u[gamma:2 * gamma], int(u[2 * gamma]), greedy)
        if record is not None:
            record.update(drafts=drafts, q=np.stack(qs), p=ps, logits=logits, a=a, out=out, P=P)
        # rollback of both caches
        self.tc.truncate(P + a + 1)
        self.dc.truncate(min(P + a + 1, P + gamma))
        self.pending = [drafts[gamma - 1]] if a == gamma else []
        self.x0 = out[-1]
        self.emitted += out
        self.accepted.append(a)
        self.n_steps += 1
        return a, out


def sd_generate(target: Model, draft: Model, prompt: Sequence[int], gamma: int,
                n_new: int, utable: np.ndarray, tau: float = 1.0, greedy: bool = False,
                batch_rows: bool = False, records: Optional[list] = None,
                force: Optional[tuple] = None) -> Dict:
    """Speculative decoding of one task until at least n_new tokens are
    emitted.  utable [n_steps, 2*gamma+1] holds this task's uniforms; force
    as in SDTask.step."""
    task = SDTask(target, draft, prompt, batch_rows)
    while len(task.emitted) < n_new:
        rec = {} if records is not None else None
        task.step(gamma, utable[task.n_steps], tau, greedy, batch_rows, rec, force)
        if records is not None:
            records.append(rec)
    return {"tokens": task.emitted[:n_new], "accepted": task.accepted,
            "steps": task.n_steps, "task": task}


def ar_generate(target: Model, prompt: Sequence[int], n_new: int, tau: float = 1.0,
                greedy: bool = True, r: Optional[Sequence[int]] = None,
                return_logits: bool = False):
    """Plain autoregressive decoding (the reference result SD must
    reproduce): greedy arg-max, or sampling with uniforms r[i]."""
    prompt = [int(t) for t in prompt]
    cache = target.prefill(prompt[:-1])
    tok = prompt[-1]
    out, logs = [], []
    for i in range(n_new):
        z = target.decode_row(cache, tok, len(cache))
        logs.append(z)
        tok = argmax_lowest(z) if greedy else sample_weights(softmax_f32(z, tau), int(r[i]))
        out.append(int(tok))
    return (out, np.stack(logs)) if return_logits else out
