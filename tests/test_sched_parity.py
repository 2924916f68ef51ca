"""Parity of the native serving scheduler (libsd, include/sd_sched.h) with
the oracle, on seeded random task sets: identical plans, speculation lengths
and latencies; and its argument checks.  Host code only: no GPU needed."""
import os
import random

import pytest

from oracle import sched as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2510_11331_amd", "libsd.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libsd.so not built (run __graft_entry__.build())")

PAPER = {"draft": (2, 768, 3072), "target": (32, 4096, 11008),
         "c_draft": (4.11e-13, 0.56e-3), "c_verify": (2.08e-14, 1.28e-2)}
SPLIT = dict(PAPER, c_draft=(2e-12, 2e-4), c_verify=(4e-14, 1e-3))


def canon(batches):
    """Batches in pipeline order, each as its sorted task indices."""
    return [sorted(b) for b in batches]


def cases():
    rng = random.Random(17)
    for trial in range(10):
        cfg = dict(rng.choice([PAPER, SPLIT]), prefill_separate=trial % 3 == 2)
        K = rng.randint(1, 14)
        lengths = [rng.choice([rng.randint(1, 64), rng.randint(1, 2048)]) for _ in range(K)]
        alpha = rng.choice([0.0, 0.5, 0.8, 1.0])
        o_max = rng.choice([16, 64, 200])
        yield cfg, lengths, alpha, o_max


@pytest.mark.parametrize("case", list(cases()))
def test_plan_matches_oracle(case):
    from paper_2510_11331_amd import sched as N
    cfg, lengths, alpha, o_max = case
    full = dict(cfg, alpha=alpha, o_max=o_max)
    for l in (1, 3, 6):
        nb, nt = N.batching(full, lengths, l)
        ob, ot = S.dp_batching(cfg, lengths, l, alpha, o_max)
        assert canon(nb) == canon(ob)
        assert nt == pytest.approx(ot, rel=1e-13, abs=0)
        assert N.latency(full, lengths, ob, l) == pytest.approx(S.pipeline_latency(cfg, ob, lengths, l, alpha, o_max),
                                                                rel=1e-13)
    np_, op = N.plan(full, lengths, 7), S.plan(cfg, lengths, 7, alpha, o_max)
    assert np_["l"] == op["l"] and canon(np_["batches"]) == canon(op["batches"])
    assert np_["t_inf_by_l"] == pytest.approx(op["t_inf_by_l"], rel=1e-13)


def test_memory_budget_matches_oracle_and_infeasible_is_enomem():
    from paper_2510_11331_amd import sched as N, _lib
    lengths = [100, 120, 90, 300, 310, 80]
    params = 2 * (8.0 * 768 ** 2 + 4.0 * 768 * 3072)
    budget = params + 2.5 * 4.0 * 2 * 768 * (310 + 64)
    full = dict(PAPER, alpha=0.8, o_max=64, mem_budget=budget)
    nb, nt = N.batching(full, lengths, 3)
    ob, ot = S.dp_batching(PAPER, lengths, 3, 0.8, 64, mem_budget=budget)
    assert canon(nb) == canon(ob) and nt == pytest.approx(ot, rel=1e-13)
    assert len(nb) > 1
    assert all(S.draft_memory(PAPER, len(b), max(lengths[k] for k in b), 64) <= budget for b in nb)
    with pytest.raises(_lib.SDError) as e:
        N.batching(dict(full, mem_budget=params), lengths, 3)
    assert e.value.code == _lib.SD_ENOMEM


def test_uplink_matches_oracle():
    from paper_2510_11331_amd import sched as N
    rng = random.Random(4)
    lengths = [rng.randint(1, 512) for _ in range(12)]
    snr = [10 ** rng.uniform(-1, 3) for _ in range(12)]
    w, t = N.uplink(lengths, snr, 16 * (768 + 4096), 20e6)
    ow, ot = S.uplink_allocation(lengths, snr, 16 * (768 + 4096), 20e6)
    assert w == pytest.approx(ow, rel=1e-14)
    assert t == pytest.approx(ot, rel=1e-14)


def test_invalid_arguments_are_rejected():
    import ctypes as C
    import numpy as np
    from paper_2510_11331_amd import sched as N, _lib
    good = dict(PAPER, alpha=0.8, o_max=64)
    bad_cfgs = [dict(good, alpha=1.5), dict(good, alpha=-0.1), dict(good, o_max=0), dict(good, draft=(0, 768, 3072)),
                dict(good, c_verify=(-1.0, 0.0))]
    for bad in bad_cfgs:
        with pytest.raises(_lib.SDError) as e:
            N.batching(bad, [10, 20], 2)
        assert e.value.code == _lib.SD_EINVAL
    for lengths, l in (([10, 0], 2), ([], 2), ([10], 0)):
        with pytest.raises(_lib.SDError):
            N.batching(good, lengths, l)
    with pytest.raises(_lib.SDError):
        N.latency(good, [10, 20], [[0], []], 2)          # empty batch
    with pytest.raises(_lib.SDError):
        N.uplink([10, 20], [1.0, 0.0], 1.0, 1.0)          # snr must be > 0
    L = _lib.lib()
    lens = np.array([10, 20], dtype=np.int32)
    out = np.zeros(2, dtype=np.int32)
    nb, t = C.c_int(0), C.c_double(0)
    # null pointers
    assert L.sd_sched_batching(None, 2, lens.ctypes.data_as(C.POINTER(C.c_int32)), 2,
                               out.ctypes.data_as(C.POINTER(C.c_int32)), C.byref(nb), C.byref(t)) == _lib.SD_EINVAL
