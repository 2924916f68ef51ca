"""Pins of the oracle SD loop against what the method fixes: greedy SD equals
plain greedy decoding of the target, rollback leaves the caches equal to a
fresh prefill of the emitted prefix, a draft equal to the target is always
accepted, and the emitted tokens follow the target's law (exact enumeration
on a 16-token vocabulary, and a chi-square test over many runs)."""
import numpy as np
import pytest
from scipy import stats

import synth
from oracle import model as om, sampling as sp, sd, exact as ex


def pair(dtype="fp32", V=64, eps=None, seed=21):
    t = synth.ModelShape(2, 32, 4, 2, 64, V, dtype)
    d = synth.ModelShape(1, 16, 2, 1, 32, V, dtype)
    wt = synth.model_weights(t, seed)
    if eps is None:
        return om.Model(t, wt), om.Model(d, synth.model_weights(d, seed + 1))
    return om.Model(t, wt), om.Model(t, synth.perturbed_weights(wt, dtype, seed + 7, eps))


@pytest.mark.parametrize("dtype,eps", [("fp32", None), ("fp32", 0.0), ("fp32", 0.3), ("bf16", 0.3)])
def test_greedy_sd_equals_ar_greedy(dtype, eps):
    target, draft = pair(dtype, eps=eps)
    for task, gamma in [(0, 1), (1, 3), (2, 5)]:
        prompt = synth.prompts(1, 9, target.s.vocab, first_task=task)[0]
        u = synth.uniform_table(42, [task], 40, gamma)[:, 0]
        res = sd.sd_generate(target, draft, prompt, gamma, 24, u, greedy=True)
        ar = sd.ar_generate(target, prompt, 24, greedy=True)
        assert res["tokens"] == ar
        if eps == 0.0:
            assert all(a == gamma for a in res["accepted"])      # identical draft
        acc = np.array(res["accepted"])
        assert np.all((acc >= 0) & (acc <= gamma))


def test_rollback_leaves_fresh_prefill():
    target, draft = pair("bf16", eps=0.5)
    gamma = 3
    prompt = synth.prompts(1, 7, target.s.vocab, first_task=5)[0]
    u = synth.uniform_table(43, [5], 40, gamma)[:, 0]
    res = sd.sd_generate(target, draft, prompt, gamma, 30, u, tau=0.05)   # sharp: mixed acceptance
    task = res["task"]
    seq = list(prompt) + task.emitted
    assert set(res["accepted"]) >= {0, gamma}            # both rollback cases occurred
    tc = target.prefill(seq[:-1])                        # everything but the next input x0
    assert len(task.tc) == len(tc)
    for l in range(target.s.n_layers):
        assert np.array_equal(task.tc.K[l], tc.K[l]) and np.array_equal(task.tc.V[l], tc.V[l])
    dlen = len(seq) - 1 - len(task.pending)
    dc = draft.prefill(seq[:dlen])
    assert len(task.dc) == dlen
    for l in range(draft.s.n_layers):
        assert np.array_equal(task.dc.K[l], dc.K[l])
    assert task.x0 == seq[-1]


@pytest.mark.parametrize("tau,greedy", [(1.0, False), (0.05, False), (1.0, True)])
def test_resume_from_prompt_plus_emitted_continues_the_run(tau, greedy):
    """Checkpoint / resume: a task rebuilt from prompt + emitted tokens and
    stepped with the uniforms of the later steps emits what the uninterrupted
    task emits (the committed caches equal a fresh prefill, pinned above)."""
    target, draft = pair("bf16", eps=0.5)
    gamma, n1, n2 = 3, 6, 8
    prompt = synth.prompts(1, 7, target.s.vocab, first_task=9)[0]
    u = synth.uniform_table(44, [9], n1 + n2, gamma)[:, 0]
    whole = sd.SDTask(target, draft, prompt)
    ref = [whole.step(gamma, u[n], tau, greedy) for n in range(n1 + n2)]
    first = sd.SDTask(target, draft, prompt)
    part1 = [first.step(gamma, u[n], tau, greedy) for n in range(n1)]
    resumed = sd.SDTask(target, draft, list(prompt) + first.emitted)
    part2 = [resumed.step(gamma, u[n], tau, greedy) for n in range(n1, n1 + n2)]
    assert part1 + part2 == ref
    assert len({a for a, _ in ref}) >= 2 or greedy


def test_draft_equal_to_target_always_accepts_when_sampling():
    target, _ = pair("fp32")
    gamma = 4
    prompt = synth.prompts(1, 6, target.s.vocab, first_task=3)[0]
    u = synth.uniform_table(44, [3], 20, gamma)[:, 0]
    res = sd.sd_generate(target, target, prompt, gamma, 25, u, tau=1.0)
    assert all(a == gamma for a in res["accepted"])


def test_two_token_law_is_target_law():
    """Exact joint law of the first two emitted tokens for gamma = 2 on a
    16-token vocabulary equals the target's two-step autoregressive law.
    Given t1 accepted, the second token is the first-token law of position 1;
    after a rejection it is the first-token law of the next step, whose
    context (prompt + y1) and distributions are the same."""
    V = 16
    target, draft = pair("fp32", V=V, seed=31)
    prompt = [3, 9, 1, 14]
    tc, dc = target.prefill(prompt[:-1]), draft.prefill(prompt[:-1])
    tau = 0.1                                   # sharp distributions: rejections are common
    p0 = sp.softmax_f32(target.decode_row(tc, prompt[-1], 3), tau)
    q0 = sp.softmax_f32(draft.decode_row(dc, prompt[-1], 3), tau)
    p1, q1 = {}, {}
    for y in range(V):
        tcy, dcy = tc.copy(), dc.copy()
        p1[y] = sp.softmax_f32(target.decode_row(tcy, y, 4), tau)
        q1[y] = sp.softmax_f32(draft.decode_row(dcy, y, 4), tau)
    assert np.abs(p0 - q0).sum() > 0.3
    first = ex.first_token_law(q0, p0)
    joint = np.array([[first[y] * ex.first_token_law(q1[y], p1[y])[y2] for y2 in range(V)]
                      for y in range(V)])
    n = lambda v: v.astype(np.float64) / v.astype(np.float64).sum()
    want = np.array([[n(p0)[y] * n(p1[y])[y2] for y2 in range(V)] for y in range(V)])
    assert np.abs(joint - want).sum() < 2 * ex.quantisation_bound(V) + 1e-6


@pytest.mark.slow
def test_chi_square_first_token():
    """Run the SD decision rules many times from one context with distinct
    uniforms and compare the first emitted token with p (15 degrees of
    freedom).  Distributions along every draft path are computed once; the
    draws go through the oracle's draft_sample and accept_resample."""
    V, gamma, N, tau = 16, 2, 30000, 0.1
    target, draft = pair("fp32", V=V, seed=41)
    prompt = [2, 7, 11, 5, 0]
    tc, dc = target.prefill(prompt[:-1]), draft.prefill(prompt[:-1])
    P = len(tc)
    zt0 = target.decode_row(tc, prompt[-1], P)
    zd0 = draft.decode_row(dc, prompt[-1], P)
    zt1, zd1, zt2 = {}, {}, {}
    for a in range(V):
        tca, dca = tc.copy(), dc.copy()
        zt1[a] = target.decode_row(tca, a, P + 1)
        zd1[a] = draft.decode_row(dca, a, P + 1)
        for b in range(V):
            zt2[a, b] = target.decode_row(tca.copy(), b, P + 2)
    ut = synth.uniform_table(4242, range(N), 1, gamma)[0]
    first = np.zeros(V, np.int64)
    rejected_first = 0
    p0 = sp.softmax_f32(zt0, tau)
    for n in range(N):
        u = ut[n]
        t1, q0 = sp.draft_sample(zd0, tau, int(u[0]), False)
        t2, q1 = sp.draft_sample(zd1[t1], tau, int(u[1]), False)
        p = np.stack([p0, sp.softmax_f32(zt1[t1], tau), sp.softmax_f32(zt2[t1, t2], tau)])
        a, out = sp.accept_resample([t1, t2], np.stack([q0, q1]), p, u[gamma:2 * gamma], int(u[2 * gamma]))
        first[out[0]] += 1
        rejected_first += a == 0
    assert rejected_first > N // 10                      # the residual path carries real weight
    expect = N * p0.astype(np.float64) / p0.astype(np.float64).sum()
    chi2, pval = stats.chisquare(first, expect)
    assert pval > 0.01, (chi2, pval)
