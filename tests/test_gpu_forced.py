"""Forced acceptance on the HIP path (sd_force_draft with greedy
verification), the workload rule of the 13B configuration.

Greedy verification emits the target's greedy continuation whatever the
drafts, and every kernel computes a row independently of the other rows of
its pass, so a forced run must emit exactly the GPU's own unforced greedy
sequence.  Checked on the tiny pair and at 13B width in the launch
configuration of the 13B bench line (B = 64, gamma = 4, prompt 512), with:
  * a step accepts at least the leading run of forced drafts (they are the
    continuation), and chance matches of unforced drafts stay rare;
  * tokens per step follow eq. ol, (1 - alpha^(gamma+1)) / (1 - alpha);
  * alpha = 1 accepts every draft; forcing is refused when sampling."""
import math

import numpy as np
import pytest

import synth
from sdcase import say, make_engine, run_gpu_steps

pytestmark = pytest.mark.gpu


def _forced_run(tshape, dshape, B, gamma, prompt_len, n_forced, alpha):
    import torch
    from paper_2510_11331_amd import emitted_tokens
    from paper_2510_11331_amd.engine import uniforms_device
    from oracle import sd as osd
    tw, dw = synth.model_weights(tshape, 1), synth.model_weights(dshape, 2)
    prompts = synth.prompts(B, prompt_len, tshape.vocab)
    need = n_forced * (gamma + 1) + gamma + 2          # unforced greedy emits >= 1 token a step
    eng = make_engine(tshape, dshape, tw, dw, max_slots=B, max_batch=B, gamma_max=gamma,
                      max_ctx=prompt_len + (need + 1) * (gamma + 1) + 16, prefill_rows=2048, greedy=True)
    slots = list(range(B))
    ref, _, _, _ = run_gpu_steps(eng, slots, prompts, gamma, need, 7, slots,
                                 max_new=[(need + 1) * (gamma + 1)] * B)
    assert min(len(e) for e in ref) >= need
    cont = np.array([list(prompts[k]) + ref[k][:need] for k in range(B)], dtype=np.int32)
    for s in slots:
        eng.release(s)
    say("forced run alpha", alpha, "steps", n_forced)
    eng.prefill(slots, prompts, [(need + 1) * (gamma + 1)] * B)
    b = eng.batch(slots, gamma)
    b.set_force(cont, alpha)
    ut = synth.uniform_table(42, slots, n_forced, gamma)
    u = uniforms_device(ut)
    accs, outs = [], []
    for n in range(n_forced):
        eng.step(b, u[n])
        accs.append(b.n_acc.clone())
        outs.append(b.out_tok.clone())
    torch.cuda.synchronize()
    acc = torch.stack(accs).cpu().numpy()
    out = torch.stack(outs).cpu().numpy()
    assert eng.check_flags() == 0
    eng.close()
    emitted = emitted_tokens(acc, out)
    bound = osd.force_threshold(alpha)
    # exactness: the forced run emits the unforced greedy sequence
    for k in range(B):
        assert emitted[k] == list(cont[k, prompt_len:prompt_len + len(emitted[k])]), k
    # every step accepts at least its leading run of forced drafts
    forced = ut[:, :, :gamma].astype(np.uint64) < bound          # [steps, B, gamma]
    lead = np.cumprod(forced, axis=2).sum(axis=2)
    assert (acc >= lead).all()
    extra = (acc > lead).mean()                                  # chance matches of unforced drafts
    return acc, extra


@pytest.mark.parametrize("alpha", [0.5, 0.8])
def test_tiny_forced_run_equals_the_oracle(alpha):
    """The forced rule on the tiny pair, decision by decision: both sides get
    the oracle's greedy continuation of the target as the reference, the
    same uniforms and alpha; the GPU's accepted lengths and emitted tokens
    are the oracle's SD run with the same forcing (sd_generate(force=...))."""
    import torch
    from paper_2510_11331_amd import emitted_tokens
    from paper_2510_11331_amd.engine import uniforms_device
    from oracle import model as om, sd as osd
    say("tiny forced against the oracle", alpha)
    w = synth.WORKLOADS["tiny"]
    t, d, gamma, B, n_steps = w.target, w.draft, 4, 4, 12
    tw, dw = synth.model_weights(t, 1), synth.model_weights(d, 2)
    prompts = synth.prompts(B, w.prompt_len, t.vocab)
    tgt, dft = om.Model(t, tw), om.Model(d, dw)
    n_cont = n_steps * (gamma + 1) + 2
    cont = np.array([list(prompts[k]) + osd.ar_generate(tgt, prompts[k], n_cont, greedy=True) for k in range(B)],
                    dtype=np.int32)
    eng = make_engine(t, d, tw, dw, max_slots=B, max_batch=B, gamma_max=gamma,
                      max_ctx=w.prompt_len + (n_steps + 1) * (gamma + 1) + 16, greedy=True)
    slots = list(range(B))
    eng.prefill(slots, prompts, [(n_steps + 1) * (gamma + 1)] * B)
    b = eng.batch(slots, gamma)
    b.set_force(cont, alpha)
    ut = synth.uniform_table(42, slots, n_steps, gamma)
    u = uniforms_device(ut)
    accs, outs = [], []
    for n in range(n_steps):
        eng.step(b, u[n])
        accs.append(b.n_acc.clone())
        outs.append(b.out_tok.clone())
    torch.cuda.synchronize()
    acc = torch.stack(accs).cpu().numpy()
    out = torch.stack(outs).cpu().numpy()
    assert eng.check_flags() == 0
    eng.close()
    bound = osd.force_threshold(alpha)
    for k in range(B):
        task = osd.SDTask(tgt, dft, prompts[k])
        for n in range(n_steps):
            a, em = task.step(gamma, ut[n, k], greedy=True, force=(cont[k], bound))
            assert acc[n, k] == a and list(out[n, k, :a + 1]) == em, (k, n, acc[n, k], a)


@pytest.mark.parametrize("alpha", [0.5, 0.8, 1.0])
def test_tiny_forced_emits_greedy_sequence_and_follows_eq_ol(alpha):
    say("tiny forced", alpha)
    w = synth.WORKLOADS["tiny"]
    gamma = 4
    acc, extra = _forced_run(w.target, w.draft, B=8, gamma=gamma, prompt_len=w.prompt_len, n_forced=40,
                             alpha=alpha)
    if alpha == 1.0:
        assert (acc == gamma).all()
        return
    e = (acc + 1).astype(np.float64).ravel()
    expect = (1 - alpha ** (gamma + 1)) / (1 - alpha)
    se = e.std(ddof=1) / math.sqrt(e.size)
    print("alpha", alpha, "emitted/step", e.mean(), "eq. ol", expect, "se", se, "chance", extra)
    assert extra < 0.05
    assert abs(e.mean() - expect) < 4 * se + 0.05


def test_13b_width_forced_bench_launch_config():
    """13B width (1-layer cuts), B = 64, gamma = 4, prompt 512, alpha = 0.8."""
    w = synth.WORKLOADS["13b"]
    t = w.target.replace(n_layers=1)
    d = w.draft.replace(n_layers=1)
    say("13b-width forced", w.alpha_forced)
    acc, extra = _forced_run(t, d, B=w.batch, gamma=w.gamma, prompt_len=w.prompt_len, n_forced=20,
                             alpha=w.alpha_forced)
    a = w.alpha_forced
    e = (acc + 1).astype(np.float64).ravel()
    expect = (1 - a ** (w.gamma + 1)) / (1 - a)
    se = e.std(ddof=1) / math.sqrt(e.size)
    print("emitted/step", e.mean(), "eq. ol", expect, "se", se, "chance", extra)
    assert extra < 0.05
    assert abs(e.mean() - expect) < 4 * se + 0.05


def test_forcing_is_refused_when_sampling():
    from paper_2510_11331_amd import _lib
    from paper_2510_11331_amd.engine import uniforms_device
    w = synth.WORKLOADS["tiny"]
    tw, dw = synth.model_weights(w.target, 1), synth.model_weights(w.draft, 2)
    eng = make_engine(w.target, w.draft, tw, dw, max_slots=2, max_batch=2, gamma_max=4, max_ctx=128)
    prompts = synth.prompts(2, 16, w.target.vocab)
    eng.prefill([0, 1], prompts, [32, 32])
    b = eng.batch([0, 1], 4)
    b.set_force(np.zeros((2, 64), dtype=np.int32), 0.5)
    u = uniforms_device(synth.uniform_table(42, [0, 1], 1, 4))
    with pytest.raises(_lib.SDError) as e:
        eng.draft_step(b, 0, u[0])
    assert e.value.code == _lib.SD_ESTATE
    eng.close()
