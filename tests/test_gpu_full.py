"""Parity at full workload sizes, in the launch configuration the benchmark
times.

The GPU runs a real SD step: B = 8 tasks, gamma = 4, verify over
B (gamma+1) = 40 rows, so every kernel runs with the tile, wave and split
choices of the benchmarked pass. The oracle then recomputes, for a few
sampled tasks, the target logits of exactly the rows the GPU verified.
These are the GPU's own draft tokens at the same positions. It also
recomputes the draft distributions q that the GPU sampled them from. Both
are compared with the 2e-2 per-row bound on logits against two oracle
forms of the model:
  * the plain model (bf16 weights, every activation and the KV cache in
    float64): the overall error of the path against full precision;
  * the model with the path's own storage points, a tighter check of the
    arithmetic (what remains is summation order and the rare element that a
    different summation order rounds the other way).
The target distribution p that the GPU hands to the acceptance step is
checked element by element over the full vocabulary: against softmax of the
GPU's own logits (the softmax kernel alone) and against softmax of the
oracle's logits, where |log p - log p_ref| <= 2 max|z - z_ref| / tau holds
for every element.

* The 7B-shape target is run whole (32 layers, B = 1, prompt 1024) and, in
  the benchmarked B = 8 configuration, on its first 2 of 32 layers so that
  the float64 oracle finishes in seconds; the matrix shapes, batch and
  context are those of the full model. The draft is the full 2-layer draft.
* The small GQA configuration (16 layers, d 2048, 32/8 heads, head_dim 64)
  is run whole, also as a greedy stream of 128 tokens per task.
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

BOUND = 2e-2


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


def _check_p(p, z_gpu, z_refs, tau):
    """Target distribution rows p [R, V] (GPU) against softmax of the GPU's
    logits (float32 rounding of the kernel only) and, for reference logits,
    the bound log-softmax differences obey."""
    ref = osp.softmax_f32(z_gpu.astype(np.float64), tau)
    assert np.all(np.abs(p - ref) <= 2e-5 * ref + 1e-30), float(np.abs(p - ref).max())
    for zr in z_refs:
        pr = osp.softmax_f32(zr, tau).astype(np.float64)
        dz = np.abs(z_gpu.astype(np.float64) - zr).max(axis=-1, keepdims=True)
        ok = pr > 1e-30
        lhs = np.abs(np.log(np.maximum(p.astype(np.float64), 1e-45)) - np.log(np.maximum(pr, 1e-45)))
        assert np.all(lhs[ok] <= (2 * dz / tau + 1e-5).repeat(p.shape[-1], axis=-1)[ok])


def _gpu_step(tshape, dshape, tw, dw, B, gamma, prompts, max_ctx=None, tau=1.0):
    longest = max(len(pr) for pr in prompts)
    eng = make_engine(tshape, dshape, tw, dw, max_slots=B, max_batch=B, gamma_max=gamma,
                      max_ctx=max_ctx or longest + 2 * (gamma + 1) + 16, prefill_rows=2048, temperature=tau)
    slots = list(range(B))
    emitted, acc, b, logits = run_gpu_steps(eng, slots, prompts, gamma, 1, 42, slots, keep_logits=True)
    out = dict(emitted=emitted, acc=acc, logits=logits[0], draft_tok=b.draft_tok.cpu().numpy(),
               q=b.q.cpu().numpy(), p=b.p.cpu().numpy(), flags=eng.check_flags())
    eng.close()
    return out


def _oracle_rows(tshape, dshape, tw, dw, prompts, g, tasks, plain, lazy=False):
    """Target logits of the verified rows and draft logits of the drafted
    rows of the sampled tasks, by the rounded (plain=False) or the plain
    model.  The draft saw x0, t_1 .. t_{gamma-1}."""
    gamma = g["draft_tok"].shape[1]
    tgt = om.Model(tshape, tw, lazy=lazy)
    dft = om.Model(dshape, dw)
    if plain:
        tgt, dft = tgt.unrounded(), dft.unrounded()
    seqs = [list(prompts[k]) + [int(t) for t in g["draft_tok"][k]] for k in tasks]
    zt = tgt.sequence_logits(seqs, gamma + 1)
    zd = dft.sequence_logits([sq[:-1] for sq in seqs], gamma)
    return zt, zd


def _errors(g, tasks, zt, zd):
    gamma = g["draft_tok"].shape[1]
    ep = max(_rel_row_err(g["logits"][k, j].astype(np.float64), zt[i][j])
             for i, k in enumerate(tasks) for j in range(gamma + 1))
    eq = max(_logq_err(g["q"][k, j], zd[i][j]) for i, k in enumerate(tasks) for j in range(gamma))
    return ep, eq


def _check(tshape, dshape, tseed, dseed, B, gamma, prompt_len, sample_tasks, max_ctx=None):
    """prompt_len: one length, or a list of B lengths (ragged paged batch)."""
    say("full-size parity", tshape, "B", B, "gamma", gamma, "prompt", prompt_len)
    tw, dw = synth.model_weights(tshape, tseed), synth.model_weights(dshape, dseed)
    prompts = synth.prompts(B, prompt_len, tshape.vocab)
    g = _gpu_step(tshape, dshape, tw, dw, B, gamma, prompts, max_ctx)
    assert g["flags"] == 0
    errs = {}
    zts = []
    for plain in (False, True):
        zt, zd = _oracle_rows(tshape, dshape, tw, dw, prompts, g, sample_tasks, plain)
        errs["plain" if plain else "rounded"] = _errors(g, sample_tasks, zt, zd)
        zts.append(zt)
    say("worst target logit / draft errors: against the rounded model", errs["rounded"],
        "against the plain model", errs["plain"])
    for name, (ep, eq) in errs.items():
        assert ep < BOUND, (name, ep)
        assert eq < BOUND, (name, eq)
    # the target distribution over the full vocabulary: every task against
    # the softmax of its GPU logits, sampled tasks against the oracle's
    for k in range(B):
        _check_p(g["p"][k], g["logits"][k], [zt[sample_tasks.index(k)] for zt in zts] if k in sample_tasks else [],
                 1.0)
    _check_step(g, B, gamma)


def _check_step(g, B, gamma):
    # every draft token is the integer inverse-CDF draw from the GPU's own q
    # with that slot's uniform (bit-exact at the full vocabulary)
    ut = synth.uniform_table(42, list(range(B)), 1, gamma)[0]
    for k in range(B):
        for j in range(gamma):
            assert int(g["draft_tok"][k, j]) == osp.sample_weights(g["q"][k, j], int(ut[k, j])), (k, j)
    # invariants of the step at this size
    acc = g["acc"]
    assert ((acc >= 0) & (acc <= gamma)).all()
    for k in range(B):
        assert len(g["emitted"][k]) == int(acc[0, k]) + 1


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


@pytest.mark.parametrize("width,B,gamma,splits", [("13b", 32, 4, 6), ("13b", 64, 6, 3), ("7b", 64, 4, 5)])
def test_residual_projection_k_splits(width, B, gamma, splits):
    """Verify passes whose residual projections split K 6, 3 and 5 ways (160,
    448 and 320 rows): the RMSNorm after them adds that many partial sums."""
    t = synth.MODELS[f"{width}_target"].replace(n_layers=1)
    d = synth.MODELS[f"{width}_draft"].replace(n_layers=1)
    say("residual K split", splits)
    _check(t, d, 1, 2, B=B, gamma=gamma, prompt_len=128, sample_tasks=[0, B - 1])


def test_small_width_maximum_context():
    """One task at the largest context a slot takes (max_ctx 32768): a
    32750-token prompt, gamma = 4, 1-layer cuts of the small GQA pair."""
    t = synth.MODELS["small_target"].replace(n_layers=1)
    d = synth.MODELS["small_draft"].replace(n_layers=1)
    _check(t, d, 1, 2, B=1, gamma=4, prompt_len=32750, sample_tasks=[0], max_ctx=32768)


# ---------------------------------------------------------------- whole 7B-shape target

_FULL7B = {}


def _full_7b_gpu():
    """One SD step of the whole 32-layer 7B-shape target with its draft,
    B = 1, gamma = 4, prompt 1024 (the latency configuration); the GPU
    result is shared by the two oracle comparisons below."""
    if not _FULL7B:
        t, d = synth.MODELS["7b_target"], synth.MODELS["7b_draft"]
        say("whole 7B-shape target: weights")
        tw, dw = synth.model_weights(t, 1), synth.model_weights(d, 2)
        prompts = synth.prompts(1, 1024, t.vocab)
        say("whole 7B-shape target: GPU step")
        g = _gpu_step(t, d, tw, dw, 1, 4, prompts)
        assert g["flags"] == 0
        _check_step(g, 1, 4)
        _FULL7B.update(t=t, d=d, tw=tw, dw=dw, prompts=prompts, g=g)
    return _FULL7B


@pytest.mark.parametrize("form", ["plain", "rounded"])
def test_7b_shape_whole_model_single_task(form):
    """All 32 layers of the 7B-shape target, B = 1, gamma = 4, prompt 1024,
    against the float64 oracle run one layer at a time (each layer's
    weights decoded when it runs): logits of the 5 verified rows, the
    draft's q, and p over the full vocabulary."""
    c = _full_7b_gpu()
    say("whole 7B-shape target: oracle,", form)
    zt, zd = _oracle_rows(c["t"], c["d"], c["tw"], c["dw"], c["prompts"], c["g"], [0], form == "plain", lazy=True)
    ep, eq = _errors(c["g"], [0], zt, zd)
    say("whole 7B-shape target against the", form, "model: target logits", ep, "draft", eq)
    _check_p(c["g"]["p"][0], c["g"]["logits"][0], zt, 1.0)
    assert ep < BOUND, ep
    assert eq < BOUND, eq


# ---------------------------------------------------------------- greedy stream at whole depth

def test_small_whole_model_greedy_stream_near_ties():
    """Greedy speculative decoding of the small configuration whole (16
    layers, GQA), B = 8, gamma = 4, prompt 512, 128 new tokens per task.
    Greedy SD emits at every position the target's arg-max given the
    emitted prefix.  The oracle is run on the GPU's own emitted prefix
    (teacher forcing), which resynchronises it after any divergence, and
    at every emitted position:
      * the GPU's token is the arg-max of the GPU's logits (exact);
      * the GPU's logits are within the bound of the oracle's;
      * where the GPU's token is not the oracle's arg-max, the oracle's
        top-2 gap is counted as a near tie (< 1e-3) or as a divergence; a
        divergence is only possible where the two tokens' logit errors
        together exceed the oracle's gap, which is checked."""
    from sdcase import greedy_stream_report
    wl = synth.WORKLOADS["small"]
    t, d = wl.target, wl.draft
    B, gamma, n_new = wl.batch, wl.gamma, wl.new_tokens
    say("small whole greedy stream")
    tw, dw = synth.model_weights(t, 1), synth.model_weights(d, 2)
    prompts = synth.prompts(B, wl.prompt_len, t.vocab)
    eng = make_engine(t, d, tw, dw, max_slots=B, max_batch=B, gamma_max=gamma,
                      max_ctx=wl.prompt_len + (n_new + 2) * (gamma + 1) + 16, prefill_rows=2048, greedy=True)
    slots = list(range(B))
    # greedy emits at least one token a step: n_new steps give every task n_new
    emitted, acc, b, logits = run_gpu_steps(eng, slots, prompts, gamma, n_new, 42, slots,
                                            max_new=[(n_new + 2) * (gamma + 1)] * B, keep_logits=True)
    assert eng.check_flags() == 0
    eng.close()
    say("small whole greedy stream: oracle")
    rep = greedy_stream_report(om.Model(t, tw), prompts, emitted, acc, logits, n_new, BOUND)
    say("greedy stream:", rep)
    assert rep["positions"] == B * n_new
