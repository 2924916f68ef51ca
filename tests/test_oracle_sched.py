"""Pins of the scheduler oracle (cost model, pipeline latency, Algorithm 1,
speculation-length search, uplink allocation) against what the mathematics
fixes: the geometric series and an exact enumeration for the expected
emitted tokens, an explicit count of the block's matrix products for the
FLOPs formulas, hand-derived pipeline latencies for one and two batches,
brute force over every contiguous batching, cases where the optimum is known
(additive cost, fixed cost only), and the equal-finish property of the
uplink allocation."""
import math
import random

import pytest

from oracle import sched as S

# paper Table I shapes (J, h1, h2): LLaMA-68M draft, LLaMA-7B target
CFG = {"draft": (2, 768, 3072), "target": (32, 4096, 11008),
       "c_draft": (4.11e-13, 0.56e-3), "c_verify": (2.08e-14, 1.28e-2)}


def test_expected_emitted_is_geometric_series_and_enumeration():
    for alpha in (0.0, 0.3, 0.8, 0.95):
        for l in (1, 2, 4, 7, 10):
            series = sum(alpha ** i for i in range(l + 1))
            # drafts accepted independently with probability alpha: a = k
            # accepted (k < l) with probability alpha^k (1 - alpha), all l with
            # alpha^l; a + 1 tokens are emitted
            enum = sum((k + 1) * alpha ** k * (1 - alpha) for k in range(l)) + (l + 1) * alpha ** l
            assert S.expected_emitted(alpha, l) == pytest.approx(series, rel=1e-12)
            assert S.expected_emitted(alpha, l) == pytest.approx(enum, rel=1e-12)
    assert S.expected_emitted(1.0, 5) == 6.0
    assert S.expected_emitted(0.999999, 5) == pytest.approx(6.0, rel=1e-5)
    assert S.n_steps(100, 0.0, 3) == 100
    assert S.n_steps(100, 1.0, 3) == 25
    assert S.n_steps(101, 1.0, 3) == 26


def block_flops(h1, h2, n_q, n_k):
    """Matrix-product FLOPs of one decoder block of the paper (eqs. f11, f21,
    f31) for n_q query tokens attending to n_k keys, counted shape by shape:
    2 a b c for an [a, b] x [b, c] product."""
    mm = lambda a, b, c: 2 * a * b * c
    f = 3 * mm(n_q, h1, h1)          # Q, K, V projections
    f += mm(n_q, h1, n_k)            # Q K^T
    f += mm(n_q, n_k, h1)            # softmax(.) V
    f += mm(n_q, h1, h1)             # W_O
    f += mm(n_q, h1, h2)             # W_1
    f += mm(n_q, h2, h1)             # W_2
    return f


def test_flops_match_explicit_product_count():
    J, h1, h2 = 3, 64, 176
    for I_m in (1, 7, 50):
        # draft prefill: I_m tokens over I_m keys
        assert S.flops_draft(J, h1, h2, I_m, 1, 1, 2.0) == J * block_flops(h1, h2, I_m, I_m)
        # a draft decode forward: one token over the cached keys plus itself
        for n, i, L in ((1, 2, 1.0), (3, 1, 2.5), (4, 3, 1.75)):
            kv = I_m + ((n - 1) * L - 1) + i - 1
            assert S.flops_draft(J, h1, h2, I_m, i, n, L) == pytest.approx(J * block_flops(h1, h2, 1, kv + 1))
        for l in (1, 4):
            # verify at step 1: prefill of I_m + l tokens
            assert S.flops_verify(J, h1, h2, I_m, l, 1, 2.0) == J * block_flops(h1, h2, I_m + l, I_m + l)
            # later steps: 1 + l tokens over kv + l + 1 keys
            for n, L in ((2, 1.5), (5, 3.0)):
                kv = I_m + (n - 1) * L - 1
                assert S.flops_verify(J, h1, h2, I_m, l, n, L) == pytest.approx(
                    J * block_flops(h1, h2, 1 + l, kv + l + 1))


def test_pipeline_one_and_two_batches_by_hand():
    lengths = [30, 60, 90]
    l, alpha, o_max = 3, 0.7, 40
    L, N = S.expected_emitted(alpha, l), S.n_steps(o_max, alpha, l)
    one = sum(sum(S.step_times(CFG, 3, 90, l, n, L)) for n in range(1, N + 1))
    assert S.pipeline_latency(CFG, [[0, 1, 2]], lengths, l, alpha, o_max) == pytest.approx(one, rel=1e-14)
    two = 0.0
    for n in range(1, N + 1):
        d1, v1 = S.step_times(CFG, 1, 30, l, n, L)
        d2, v2 = S.step_times(CFG, 2, 90, l, n, L)
        # batch 2 verifies after its own drafting and after batch 1's verify
        two += max(d1 + d2, d1 + v1) + v2
    assert S.pipeline_latency(CFG, [[0], [1, 2]], lengths, l, alpha, o_max) == pytest.approx(two, rel=1e-14)


def rand_tasks(rng, K, imax=512):
    return [rng.randint(1, imax) for _ in range(K)]


# costs where splitting pays: small fixed costs, padding expensive
SPLIT = dict(CFG, c_draft=(2e-12, 2e-4), c_verify=(4e-14, 1e-3))


@pytest.mark.parametrize("cfg", [CFG, SPLIT], ids=["paper_table2", "split_favoured"])
def test_dp_value_is_its_plan_and_bounded_by_brute_force(cfg):
    rng = random.Random(5)
    multi = 0
    for trial in range(14):
        K = rng.randint(1, 7)
        # bimodal input lengths, so that some plans split the tasks
        lengths = [rng.choice([rng.randint(1, 40), rng.randint(300, 512)]) for _ in range(K)]
        l, alpha = rng.randint(1, 6), rng.choice([0.5, 0.8])
        batches, t = S.dp_batching(cfg, lengths, l, alpha, 64)
        multi += len(batches) > 1
        # a partition of every task into runs of the sorted order
        flat = [k for b in batches for k in b]
        assert sorted(flat) == list(range(K))
        order = sorted(range(K), key=lambda k: (lengths[k], k))
        assert flat == order
        # the table value is the latency of the plan it reads back (reading S-1)
        assert t == pytest.approx(S.pipeline_latency(cfg, batches, lengths, l, alpha, 64), rel=1e-12)
        bf_batches, bf = S.brute_force_batching(cfg, lengths, l, alpha, 64)
        assert t >= bf * (1 - 1e-12)
        if K <= 2:
            assert t == pytest.approx(bf, rel=1e-12)
    if cfg is SPLIT:
        assert multi >= 3          # the multi-batch recursion is exercised


def test_dp_optimal_where_the_cost_is_additive_or_fixed():
    rng = random.Random(9)
    lengths = rng.sample(range(1, 400), 7)       # distinct lengths
    # free drafting and no fixed cost: latency is additive over batches and
    # grows with padding, so every task alone is optimal and the DP finds it
    additive = dict(CFG, c_draft=(0.0, 0.0), c_verify=(1e-14, 0.0))
    batches, t = S.dp_batching(additive, lengths, 3, 0.8, 32)
    bf_b, bf = S.brute_force_batching(additive, lengths, 3, 0.8, 32)
    assert t == pytest.approx(bf, rel=1e-12)
    assert len(batches) == len(set(lengths))
    # fixed cost only: every extra batch adds its fixed cost; one batch is optimal
    fixed = dict(CFG, c_draft=(0.0, 1e-3), c_verify=(0.0, 5e-3))
    batches, t = S.dp_batching(fixed, lengths, 3, 0.8, 32)
    assert len(batches) == 1
    N = S.n_steps(32, 0.8, 3)
    assert t == pytest.approx(N * (3 * 1e-3 + 5e-3), rel=1e-12)


def test_memory_budget_splits_batches_and_infeasible_raises():
    lengths = [100] * 6
    per_task = 4.0 * 2 * 768 * (100 + 64)
    params = 2 * (8.0 * 768 ** 2 + 4.0 * 768 * 3072)
    budget = params + 2.5 * per_task          # at most two tasks per batch
    batches, _ = S.dp_batching(CFG, lengths, 2, 0.8, 64, mem_budget=budget)
    assert all(len(b) <= 2 for b in batches)
    assert all(S.draft_memory(CFG, len(b), 100, 64) <= budget for b in batches)
    with pytest.raises(ValueError):
        S.dp_batching(CFG, lengths, 2, 0.8, 64, mem_budget=params)


def test_plan_takes_the_best_speculation_length():
    rng = random.Random(3)
    lengths = rand_tasks(rng, 9)
    p = S.plan(CFG, lengths, 8, 0.8, 128)
    assert len(p["t_inf_by_l"]) == 8
    assert p["t_inf"] == min(p["t_inf_by_l"])
    assert p["t_inf_by_l"][p["l"] - 1] == p["t_inf"]
    _, t = S.dp_batching(CFG, lengths, p["l"], 0.8, 128)
    assert t == p["t_inf"]


def test_uplink_allocation_equalises_and_beats_perturbations():
    rng = random.Random(11)
    K = 10
    lengths = rand_tasks(rng, K)
    snr = [10 ** rng.uniform(-1, 3) for _ in range(K)]
    lam, bw = 16 * (768 + 4096), 20e6
    w, t_star = S.uplink_allocation(lengths, snr, lam, bw)
    assert sum(w) == pytest.approx(1.0, rel=1e-12)
    times = S.upload_times(lengths, snr, w, lam, bw)
    assert max(times) == pytest.approx(t_star, rel=1e-12)
    assert min(times) == pytest.approx(t_star, rel=1e-12)
    # uniform shares, or any other allocation summing to 1, finish later
    assert max(S.upload_times(lengths, snr, [1.0 / K] * K, lam, bw)) >= t_star
    for _ in range(20):
        v = [x * rng.uniform(0.8, 1.25) for x in w]
        s = sum(v)
        v = [x / s for x in v]
        assert max(S.upload_times(lengths, snr, v, lam, bw)) >= t_star * (1 - 1e-12)


def test_prefill_separate_changes_only_the_first_step():
    sep = dict(CFG, prefill_separate=True)
    J, h1, h2 = CFG["draft"]
    Jv, h1v, h2v = CFG["target"]
    for I_m, l, L in ((40, 3, 2.2), (300, 1, 1.8)):
        for n in (2, 3, 7):
            assert S.step_times(sep, 4, I_m, l, n, L) == pytest.approx(S.step_times(CFG, 4, I_m, l, n, L), rel=1e-14)
        # step 1: l draft forwards of one token over I_m - 1, I_m, ... cached
        # tokens, and a verify of 1 + l tokens over I_m - 1 cached tokens,
        # counted product by product
        b = 4
        td = sum(CFG["c_draft"][0] * J * block_flops(h1, h2, 1, I_m - 1 + i) * b + CFG["c_draft"][1]
                 for i in range(1, l + 1))
        tv = CFG["c_verify"][0] * Jv * block_flops(h1v, h2v, 1 + l, I_m - 1 + l + 1) * b + CFG["c_verify"][1]
        got = S.step_times(sep, b, I_m, l, 1, L)
        assert got[0] == pytest.approx(td, rel=1e-12) and got[1] == pytest.approx(tv, rel=1e-12)
    rng = random.Random(8)
    lengths = [rng.choice([rng.randint(1, 40), rng.randint(300, 512)]) for _ in range(6)]
    split = dict(SPLIT, prefill_separate=True)
    batches, t = S.dp_batching(split, lengths, 3, 0.8, 64)
    assert t == pytest.approx(S.pipeline_latency(split, batches, lengths, 3, 0.8, 64), rel=1e-12)
    assert t >= S.brute_force_batching(split, lengths, 3, 0.8, 64)[1] * (1 - 1e-12)
