"""Checkpoint and resume on the GPU path.  After sd_kv_commit a task's state
is its prompt, the tokens emitted so far, its step count and its uniform
stream; a fresh context that prefills prompt + emitted (resume_prompts) and
continues with the uniforms of the later steps must emit what the oracle's
uninterrupted SD task emits (tiny fp32 pair: sampling at two temperatures,
and greedy)."""
import numpy as np
import pytest

import synth
from oracle import model as om, sd as osd
from sdcase import say, make_engine, run_gpu_steps

pytestmark = pytest.mark.gpu

TINY = synth.WORKLOADS["tiny"]


def _pair(kind):
    t = TINY.target
    tw = synth.model_weights(t, 1)
    if kind == "independent":
        return t, TINY.draft, tw, synth.model_weights(TINY.draft, 2)
    return t, t, tw, synth.perturbed_weights(tw, t.dtype, 77, 0.5)


@pytest.mark.parametrize("kind,tau,greedy", [("independent", 1.0, False), ("perturbed", 0.1, False),
                                             ("perturbed", 1.0, True)])
def test_resumed_run_continues_the_oracle_stream(kind, tau, greedy):
    from paper_2510_11331_amd import resume_prompts
    say("resume", kind, tau, "greedy" if greedy else "sampling")
    t, d, tw, dw = _pair(kind)
    gamma, B, n1, n2 = 4, 2, 5, 7
    prompts = synth.prompts(B, TINY.prompt_len, t.vocab)
    ctx = TINY.prompt_len + (n1 + n2 + 1) * (gamma + 1) + 8
    budget = [(n1 + n2) * (gamma + 1)] * B

    eng = make_engine(t, d, tw, dw, max_slots=4, max_batch=B, gamma_max=gamma, max_ctx=ctx,
                      temperature=tau, greedy=greedy)
    e1, acc1, _, _ = run_gpu_steps(eng, [0, 1], prompts, gamma, n1, 42, [0, 1], max_new=budget)
    assert eng.check_flags() == 0
    eng.close()

    # a new context (other slots), rebuilt from the checkpoint
    eng = make_engine(t, d, tw, dw, max_slots=4, max_batch=B, gamma_max=gamma, max_ctx=ctx,
                      temperature=tau, greedy=greedy)
    left = [budget[k] - len(e1[k]) for k in range(B)]
    e2, acc2, _, _ = run_gpu_steps(eng, [3, 2], resume_prompts(prompts, e1), gamma, n2, 42, [0, 1],
                                   max_new=left, first_step=n1)
    assert eng.check_flags() == 0
    eng.close()

    tgt, dft = om.Model(t, tw), om.Model(d, dw)
    acc = np.concatenate([acc1, acc2])
    for k in range(B):
        ut = synth.uniform_table(42, [k], n1 + n2, gamma)[:, 0]
        task = osd.SDTask(tgt, dft, prompts[k])
        ref = []
        for n in range(n1 + n2):
            a, out = task.step(gamma, ut[n], tau, greedy)
            ref += out
            assert acc[n, k] == a, (k, n, acc[n, k], a)
        assert e1[k] + e2[k] == ref
