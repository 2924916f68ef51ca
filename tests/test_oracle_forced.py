"""Pins of the forced-acceptance workload rule in the oracle SD loop (greedy
verification with drafts replaced, with probability alpha, by the target's
own greedy continuation): whatever the drafts, the emitted tokens are the
target's greedy continuation; a step accepts exactly the leading run of
drafts that equal it; alpha = 1 accepts every draft; and the tokens emitted
per step follow the expected-length formula of eq. ol."""
import math

import numpy as np
import pytest

import synth
from oracle import model as om, sd


def pair(V=64, seed=21):
    t = synth.ModelShape(2, 32, 4, 2, 64, V, "fp32")
    d = synth.ModelShape(1, 16, 2, 1, 32, V, "fp32")
    return om.Model(t, synth.model_weights(t, seed)), om.Model(d, synth.model_weights(d, seed + 1))


def continuation(target, prompt, n):
    return list(prompt) + sd.ar_generate(target, prompt, n, greedy=True)


def test_threshold_is_alpha_times_2_32_rounded():
    assert sd.force_threshold(0.0) == 0
    assert sd.force_threshold(1.0) == 2 ** 32
    assert sd.force_threshold(0.5) == 2 ** 31
    assert sd.force_threshold(0.8) == 3435973837          # 0.8 * 2^32 = 3435973836.8
    assert sd.force_threshold(1.5 / 2 ** 32) == 2         # a half rounds away from zero


@pytest.mark.parametrize("alpha", [0.0, 0.3, 0.8, 1.0])
def test_forced_greedy_sd_emits_the_greedy_continuation(alpha):
    target, draft = pair()
    gamma, n = 3, 30
    for task in range(3):
        prompt = synth.prompts(1, 8, target.s.vocab, first_task=task)[0]
        cont = continuation(target, prompt, n + gamma + 2)
        u = synth.uniform_table(42, [task], 40, gamma)[:, 0]
        recs = []
        res = sd.sd_generate(target, draft, prompt, gamma, n, u, greedy=True, records=recs,
                             force=(cont, sd.force_threshold(alpha)))
        assert res["tokens"] == cont[len(prompt):len(prompt) + n]
        for r in recs:
            # greedy verification accepts exactly the leading drafts that are
            # the continuation; forced slots always are
            P, drafts = r["P"], r["drafts"]
            lead = 0
            while lead < gamma and drafts[lead] == cont[P + 1 + lead]:
                lead += 1
            assert r["a"] == lead
        if alpha == 1.0:
            assert all(a == gamma for a in res["accepted"])
            assert res["steps"] == math.ceil(n / (gamma + 1))


def test_forced_mean_emitted_follows_eq_ol():
    # a 256-token vocabulary keeps chance matches of the draft rare; the
    # acceptance rate per slot is alpha' = alpha + (1 - alpha) m, m the
    # measured rate at which an unforced draft equals the continuation
    target, draft = pair(V=256, seed=5)
    gamma, alpha, n = 4, 0.6, 400
    bound = sd.force_threshold(alpha)
    emitted, unforced, matched = [], 0, 0
    for task in range(4):
        prompt = synth.prompts(1, 6, target.s.vocab, first_task=task)[0]
        cont = continuation(target, prompt, n + gamma + 2)
        u = synth.uniform_table(7, [task], 400, gamma)[:, 0]
        recs = []
        sd.sd_generate(target, draft, prompt, gamma, n, u, greedy=True, records=recs, force=(cont, bound))
        for k, r in enumerate(recs):
            emitted.append(r["a"] + 1)
            for i in range(r["a"] + 1 if r["a"] < gamma else gamma):
                if int(u[k][i]) >= bound:
                    unforced += 1
                    matched += r["drafts"][i] == cont[r["P"] + 1 + i]
    m = matched / max(unforced, 1)
    a1 = alpha + (1 - alpha) * m
    expect = (1 - a1 ** (gamma + 1)) / (1 - a1)
    e = np.asarray(emitted, dtype=np.float64)
    se = e.std(ddof=1) / math.sqrt(len(e))
    assert abs(e.mean() - expect) < 3 * se, (e.mean(), expect, se, m)
    assert m < 0.05
