"""Parity at full workload sizes, in the launch configuration the benchmark
times.

The GPU runs a real SD step: B = 8 tasks, gamma = 4, verify over
B (gamma+1) = 40 rows, so every kernel runs with the tile, wave and split
choices of the benchmarked pass. The oracle then recomputes, for a few
sampled tasks, the target logits of exactly the rows the GPU verified.
These are the GPU's own draft tokens at the same positions. It also
recomputes the draft distributions q that the GPU sampled them from. Both
are compared with the 2e-2 per-row bound on logits.

* The 7B-shape target is cut to its first 2 of 32 layers so that the
  float64 oracle finishes in seconds; the matrix shapes, batch and context
  are those of the full model. The draft is the full 2-layer draft.
* The small GQA configuration (16 layers, d 2048, 32/8 heads, head_dim 64)
  is run whole.
* The single-task, ragged paged and 13B-width configurations are run on
  layer cuts at their real widths, batch sizes and contexts.
* The maximum context (32768 positions per slot) is run on a 1-layer cut
  of the small configuration: 32750 cached positions, so the keys are split
  12 ways over workgroups and merged.
"""
import numpy as np
import pytest

import synth
from oracle import model as om, sampling as osp
from sdcase import say, make_engine, run_gpu_steps

pytestmark = pytest.mark.gpu


def _rel_row_err(z, zr):
    """Per-row max abs error over max abs reference (the logit bound)."""
    return float(np.abs(z - zr).max() / np.abs(zr).max())


def _logq_err(q, zr):
    """Error of the draft distribution q (fp32 probabilities) against
    reference logits zr, in logit units: log q is the logit up to a
    per-row constant, which is removed before taking the same relative
    measure as for logits."""
    lq = np.log(np.maximum(q.astype(np.float64), 1e-45))
    lr = zr - zr.max()
    lr = lr - np.log(np.exp(lr).sum())
    e = lq - lr
    e -= np.median(e)
    return float(np.abs(e).max() / np.abs(zr).max())


def _check(tshape, dshape, tseed, dseed, B, gamma, prompt_len, sample_tasks, max_ctx=None):
    """prompt_len: one length, or a list of B lengths (ragged paged batch)."""
    say("full-size parity", tshape, "B", B, "gamma", gamma, "prompt", prompt_len)
    tw, dw = synth.model_weights(tshape, tseed), synth.model_weights(dshape, dseed)
    prompts = synth.prompts(B, prompt_len, tshape.vocab)
    longest = max(len(pr) for pr in prompts)
    eng = make_engine(tshape, dshape, tw, dw, max_slots=B, max_batch=B, gamma_max=gamma,
                      max_ctx=max_ctx or longest + 2 * (gamma + 1) + 16, prefill_rows=2048)
    slots = list(range(B))
    emitted, acc, b, logits = run_gpu_steps(eng, slots, prompts, gamma, 1, 42, slots, keep_logits=True)
    draft_tok = b.draft_tok.cpu().numpy()
    q = b.q.cpu().numpy()
    assert eng.check_flags() == 0
    eng.close()
    tgt, dft = om.Model(tshape, tw), om.Model(dshape, dw)
    worst_p, worst_q = 0.0, 0.0
    for k in sample_tasks:
        rows = [int(prompts[k][-1])] + [int(t) for t in draft_tok[k]]
        ct = tgt.prefill(prompts[k][:-1], batch_rows=True)
        zt = tgt.forward_rows(ct, rows)                       # [gamma+1, V]
        cd = dft.prefill(prompts[k][:-1], batch_rows=True)
        zd = dft.forward_rows(cd, rows[:gamma])               # the draft saw x0, t1..t_{gamma-1}
        for j in range(gamma + 1):
            worst_p = max(worst_p, _rel_row_err(logits[0, k, j].astype(np.float64), zt[j]))
        for j in range(gamma):
            worst_q = max(worst_q, _logq_err(q[k, j], zd[j]))
        say("task", k, "worst target logit err", worst_p, "worst draft err", worst_q)
    assert worst_p < 2e-2, worst_p
    assert worst_q < 2e-2, worst_q
    # every draft token is the integer inverse-CDF draw from the GPU's own q
    # with that slot's uniform (bit-exact at the full vocabulary)
    ut = synth.uniform_table(42, slots, 1, gamma)[0]
    for k in range(B):
        for j in range(gamma):
            assert int(draft_tok[k, j]) == osp.sample_weights(q[k, j], int(ut[k, j])), (k, j)
    # invariants of the step at this size
    assert ((acc >= 0) & (acc <= gamma)).all()
    for k in range(B):
        assert len(emitted[k]) == int(acc[0, k]) + 1


def test_7b_shape_two_layer_cut_bench_launch_config():
    """The benchmarked workload: B = 8, gamma = 4, prompt 1024."""
    t = synth.MODELS["7b_target"].replace(n_layers=2)
    d = synth.MODELS["7b_draft"]
    _check(t, d, 1, 2, B=8, gamma=4, prompt_len=1024, sample_tasks=[0, 5, 7])


def test_small_gqa_config_whole_model():
    """The small configuration whole: 16 layers, GQA 32/8, B = 8, prompt 512."""
    t = synth.MODELS["small_target"]
    d = synth.MODELS["small_draft"]
    _check(t, d, 1, 2, B=8, gamma=4, prompt_len=512, sample_tasks=[0, 3])


@pytest.mark.parametrize("gamma", [1, 8])
def test_7b_shape_single_task_latency_config(gamma):
    """B = 1 at 7B width (the latency-versus-gamma configuration): 32
    attention items, so the keys are split over workgroups."""
    t = synth.MODELS["7b_target"].replace(n_layers=2)
    d = synth.MODELS["7b_draft"]
    _check(t, d, 1, 2, B=1, gamma=gamma, prompt_len=1024, sample_tasks=[0])


def test_7b_shape_ragged_paged_batch():
    """B = 32 with prompt lengths uniform in [128, 2048] on the paged cache."""
    t = synth.MODELS["7b_target"].replace(n_layers=1)
    d = synth.MODELS["7b_draft"]
    lens = [int(x) for x in synth.ragged_lengths(32, 128, 2048)]
    short, long_ = int(np.argmin(lens)), int(np.argmax(lens))
    _check(t, d, 1, 2, B=32, gamma=4, prompt_len=lens, sample_tasks=[short, long_])


def test_13b_shape_wide_batch():
    """13B width, B = 64, gamma = 4, prompt 512: 320 verify rows, so the
    projections run in 64-row blocks."""
    t = synth.MODELS["13b_target"].replace(n_layers=1)
    d = synth.MODELS["13b_draft"].replace(n_layers=1)
    _check(t, d, 1, 2, B=64, gamma=4, prompt_len=512, sample_tasks=[0, 63])


def test_13b_width_ragged_row_tiles():
    """13B width, B = 52, gamma = 4: 260 verify rows, so the residual
    projections run on 128-row tiles whose last one holds 4 rows, and the
    wide projections on 160-row tiles whose last one holds 100."""
    t = synth.MODELS["13b_target"].replace(n_layers=1)
    d = synth.MODELS["13b_draft"].replace(n_layers=1)
    _check(t, d, 1, 2, B=52, gamma=4, prompt_len=200, sample_tasks=[0, 51])


def test_13b_width_largest_row_tiled_residual():
    """13B width, B = 80, gamma = 7: 640 verify rows, the largest pass whose
    residual projections run on row tiles."""
    t = synth.MODELS["13b_target"].replace(n_layers=1)
    d = synth.MODELS["13b_draft"].replace(n_layers=1)
    _check(t, d, 1, 2, B=80, gamma=7, prompt_len=96, sample_tasks=[0, 79])


def test_small_width_maximum_context():
    """One task at the largest context a slot takes (max_ctx 32768): a
    32750-token prompt, gamma = 4, 1-layer cuts of the small GQA pair."""
    t = synth.MODELS["small_target"].replace(n_layers=1)
    d = synth.MODELS["small_draft"].replace(n_layers=1)
    _check(t, d, 1, 2, B=1, gamma=4, prompt_len=32750, sample_tasks=[0], max_ctx=32768)
