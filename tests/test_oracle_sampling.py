"""Pins of the oracle's sampling rules: exact integer arithmetic, edge cases,
the distribution-preservation property of speculative sampling (counted
exactly), and the expected number of emitted tokens per step (eq. ol)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import sampling as sp
from oracle import exact as ex


def rand_dist(rng, V, sharp=1.0):
    z = rng.standard_normal(V) * sharp
    return sp.softmax_f32(z, 1.0)


def test_threshold_is_exact_floor():
    rng = np.random.default_rng(0)
    for _ in range(2000):
        S = int(rng.integers(1, 2**62))
        r = int(rng.integers(0, 2**32))
        assert sp.threshold(S, r) == int(Fraction(S * r, 2**32))
        assert sp.threshold(S, r) < S
    # the split form a GPU uses, hi/lo 32-bit halves, gives the same value
    for _ in range(2000):
        S = int(rng.integers(1, 2**56))
        r = int(rng.integers(0, 2**32))
        split = (S >> 32) * r + (((S & 0xFFFFFFFF) * r) >> 32)
        assert split == sp.threshold(S, r)


def test_sample_weights_hand_boundaries():
    # W = [2^38, 0, 2^39, 2^38], S = 2^40, T = r * 2^8
    w = np.array([0.25, 0.0, 0.5, 0.25], dtype=np.float32)
    assert sp.fixed_weights(w) == [2**38, 0, 2**39, 2**38]
    assert sp.sample_weights(w, 0) == 0
    assert sp.sample_weights(w, 2**30 - 1) == 0
    assert sp.sample_weights(w, 2**30) == 2           # index 1 has no mass
    assert sp.sample_weights(w, 3 * 2**30 - 1) == 2
    assert sp.sample_weights(w, 3 * 2**30) == 3
    assert sp.sample_weights(w, 2**32 - 1) == 3
    assert sp.sample_weights(np.zeros(5, np.float32), 123) is None
    # tiny weights: below 2^-40 an entry has no integer mass
    assert sp.sample_weights(np.array([2**-41, 2**-40], np.float32), 0) == 1


def test_sample_law_matches_weights():
    rng = np.random.default_rng(1)
    for V in (2, 16, 1000):
        w = rand_dist(rng, V, 2.0)
        law = ex.sample_law(w)
        assert abs(law.sum() - 1) < 1e-15
        assert np.max(np.abs(law - w / w.astype(np.float64).sum())) < V * 2.0 ** -32 + 1e-9
    # unnormalised weights are normalised implicitly
    w = np.array([3.0, 1.0], np.float32)
    assert np.allclose(ex.sample_law(w), [0.75, 0.25], atol=2**-32)


def test_sample_weights_follows_sample_law():
    # the law counted from the prefix boundaries is the one sample_weights draws
    rng = np.random.default_rng(2)
    w = rand_dist(rng, 7, 1.5)
    W = sp.fixed_weights(w)
    S = sum(W)
    acc, prev = 0, 0
    for j, v in enumerate(W):
        acc += v
        hi = -((-acc * 2**32) // S)          # first r that no longer draws j
        if hi > prev:
            assert sp.sample_weights(w, prev) == j
            assert sp.sample_weights(w, hi - 1) == j
        if hi < 2**32:
            assert sp.sample_weights(w, hi) != j
        prev = hi


def test_accept_rule_edges():
    f = np.float32
    for r in (0, 1, 2**31, 2**32 - 1):
        assert not sp.accepts(f(0.0), f(0.3), r)          # p(t) = 0 always rejects
        assert sp.accepts(f(0.3), f(0.3), r)              # p = q always accepts
        assert sp.accepts(f(0.5), f(0.25), r)             # p > q always accepts
        assert sp.accepts(f(1e-30), f(0.0), r)            # q(t) = 0 accepts iff p(t) > 0
        assert not sp.accepts(f(0.0), f(0.0), r)
    # u = (r >> 8) 2^-24; tie u*q == p rejects
    assert not sp.accepts(f(0.25), f(0.5), 2**31)         # u = 0.5: 0.25 < 0.25 false
    assert sp.accepts(f(0.25), f(0.5), 2**31 - 256)


def test_accept_prob_is_ratio():
    rng = np.random.default_rng(3)
    for _ in range(200):
        p, q = np.float32(rng.random()), np.float32(rng.random())
        want = min(1.0, float(p) / float(q))
        assert abs(ex.accept_prob(p, q) - want) <= 2.0 ** -23


@pytest.mark.parametrize("V,sharp", [(16, 1.0), (16, 3.0), (1000, 2.0), (32000, 1.3)])
def test_first_token_law_is_target(V, sharp):
    """Speculative sampling preserves the target distribution (Section II-A,
    after Leviathan et al.): the exact law of the first emitted token equals
    p up to the integer rules' quantisation."""
    rng = np.random.default_rng(V)
    p, q = rand_dist(rng, V, sharp), rand_dist(rng, V, sharp)
    law = ex.first_token_law(q, p)
    p64 = p.astype(np.float64) / p.astype(np.float64).sum()
    assert abs(law.sum() - 1) < 1e-12
    assert np.abs(law - p64).sum() < ex.quantisation_bound(V) + V * 1e-9


def test_first_token_law_special_cases():
    rng = np.random.default_rng(9)
    p = rand_dist(rng, 16)
    law = ex.first_token_law(p.copy(), p)                      # draft == target: always accepts
    assert np.abs(law - ex.sample_law(p)).max() < 1e-15
    q = np.zeros(16, np.float32); q[:8] = sp.softmax_f32(rng.standard_normal(8), 1.0)
    p = np.zeros(16, np.float32); p[8:] = sp.softmax_f32(rng.standard_normal(8), 1.0)
    law = ex.first_token_law(q, p)                             # disjoint: residual is p
    assert np.abs(law - ex.sample_law(p)).max() < 1e-15


def test_accept_resample_invariants_and_cases():
    rng = np.random.default_rng(4)
    V = 50
    for trial in range(300):
        gamma = int(rng.integers(1, 9))
        q = np.stack([rand_dist(rng, V) for _ in range(gamma)])
        p = np.stack([rand_dist(rng, V) for _ in range(gamma + 1)])
        draft = [int(sp.sample_weights(q[i], int(rng.integers(2**32)))) for i in range(gamma)]
        u = rng.integers(0, 2**32, gamma + 1)
        a, out = sp.accept_resample(draft, q, p, u[:gamma], int(u[gamma]))
        assert 0 <= a <= gamma and len(out) == a + 1 and out[:a] == draft[:a]
        for i in range(a):                               # every accepted draft passed the test
            assert sp.accepts(p[i][draft[i]], q[i][draft[i]], int(u[i]))
        if a < gamma:
            assert not sp.accepts(p[a][draft[a]], q[a][draft[a]], int(u[a]))
            assert out[a] == sp.sample_weights(sp.residual(p[a], q[a]), int(u[gamma]))
        else:
            assert out[a] == sp.sample_weights(p[gamma], int(u[gamma]))
    # gamma = 0 reduces to one plain sample from p
    p = rand_dist(rng, V)[None]
    a, out = sp.accept_resample([], np.zeros((0, V), np.float32), p, [], 77777)
    assert a == 0 and out == [sp.sample_weights(p[0], 77777)]
    # greedy: point masses at the arg-max of the logits
    z = rng.standard_normal((4, V)).astype(np.float32)
    zq = rng.standard_normal((3, V)).astype(np.float32)
    draft = [sp.argmax_lowest(z[0]), sp.argmax_lowest(z[1]), (sp.argmax_lowest(z[2]) + 1) % V]
    a, out = sp.accept_resample(draft, zq, z, [0, 0, 0], 0, greedy=True)
    assert a == 2 and out == draft[:2] + [sp.argmax_lowest(z[2])]
    assert sp.argmax_lowest(np.array([1.0, 3.0, 3.0, 2.0])) == 1


def test_residual_fallback_when_no_mass():
    V = 8
    p = np.full(V, 1 / V, np.float32)
    q = p.copy()
    q[3] = np.float32(0.0)             # draft proposes 3? it cannot; craft a rejection instead
    draft = [5]
    q5 = p.copy(); q5[5] = np.float32(1.0)      # q(5) > p(5): rejected for large u
    pp = np.stack([p, p])
    # p - q5 is zero except at 5 where it is negative -> no residual mass -> fall back to p
    a, out = sp.accept_resample(draft, q5[None], pp, [2**32 - 1], 12345)
    assert a == 0 and out == [sp.sample_weights(p, 12345)]


def test_expected_emitted_tokens_eq_ol():
    """eq. ol: with i.i.d. acceptance of probability alpha, the expected
    number of tokens emitted per step is (1 - alpha^(gamma+1)) / (1 - alpha).
    Context-free p and q make every position's acceptance i.i.d. with
    alpha = sum_x Pq(x) A(x) (counted exactly)."""
    rng = np.random.default_rng(5)
    V, gamma, N = 12, 4, 20000
    p, q = rand_dist(rng, V, 1.2), rand_dist(rng, V, 1.2)
    alpha = float(np.sum(ex.sample_law(q) * np.array([ex.accept_prob(p[x], q[x]) for x in range(V)])))
    L = (1 - alpha ** (gamma + 1)) / (1 - alpha)
    P = np.stack([p] * (gamma + 1))
    Q = np.stack([q] * gamma)
    u = rng.integers(0, 2**32, (N, 2 * gamma + 1))
    emitted = np.empty(N)
    for n in range(N):
        draft = [sp.sample_weights(q, int(u[n, i])) for i in range(gamma)]
        a, out = sp.accept_resample(draft, Q, P, u[n, gamma:2 * gamma], int(u[n, 2 * gamma]))
        emitted[n] = len(out)
    se = emitted.std() / np.sqrt(N)
    assert abs(emitted.mean() - L) < 4 * se, (emitted.mean(), L, se)
    assert 0.3 < alpha < 0.95


def test_softmax_f32_hand_example_and_library():
    """softmax(z / tau): a hand-computed case at tau = 0.5 (exp(z / tau) =
    1, 2, 3, 4, so p = 0.1 .. 0.4), the same under a shift of 1000 (the
    maximum is subtracted: exp(2000) would overflow), and torch's softmax of
    z / tau on random rows at several temperatures.  A z * tau for z / tau,
    a dropped max-subtraction or a wrong axis fails one of them."""
    tau = 0.5
    z = 0.5 * np.log(np.array([1.0, 2.0, 3.0, 4.0]))
    want = np.array([0.1, 0.2, 0.3, 0.4], dtype=np.float32)
    got = sp.softmax_f32(z, tau)
    assert got.dtype == np.float32
    assert np.array_equal(got, want)
    assert np.array_equal(sp.softmax_f32(z + 1000.0, tau), want)
    # two rows at once: normalised over the last axis
    got2 = sp.softmax_f32(np.stack([z, z[::-1]]), tau)
    assert np.array_equal(got2, np.stack([want, want[::-1]]))
    import torch
    rng = np.random.default_rng(3)
    for t in (0.1, 0.5, 1.0, 2.0):
        zz = rng.standard_normal((4, 1000)) * 3.0
        ref = torch.softmax(torch.from_numpy(zz) / t, dim=-1).to(torch.float32).numpy()
        # float64 exponentials of two libraries may differ in the last bit,
        # which can move the float32 result by one unit of its last place
        got = sp.softmax_f32(zz, t)
        assert np.all(np.abs(got - ref) <= np.spacing(ref))
        assert np.allclose(got.sum(axis=-1), 1.0, atol=1e-5)
