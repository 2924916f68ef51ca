"""Exact laws of the implemented sampling rules (test infrastructure only).

Every rule in ``sampling`` is a deterministic function of a uint32 uniform,
so its law is a finite sum that can be counted exactly.  These laws pin the
rules against the property the paper relies on (Section II-A, after Leviathan
et al.): speculative sampling emits tokens with the target model's
distribution.
"""
from __future__ import annotations

import numpy as np

from .sampling import fixed_weights, residual

TWO32 = 1 << 32
TWO24 = 1 << 24


def _ceil_div(a: int, b: int) -> int:
    return -((-a) // b)


def sample_law(w: np.ndarray) -> np.ndarray:
    """P(sample_weights(w, r) = j) for r uniform on [0, 2^32), exactly
    (returned as float64).  Index j is drawn iff prefix_{j-1} <= T < prefix_j
    with T = floor(S r / 2^32), i.e. iff
    ceil(prefix_{j-1} 2^32 / S) <= r < ceil(prefix_j 2^32 / S)."""
    W = fixed_weights(w)
    S = sum(W)
    assert S > 0
    out = np.zeros(len(W))
    acc, lo = 0, 0
    for j, v in enumerate(W):
        acc += v
        hi = _ceil_div(acc * TWO32, S)
        out[j] = (hi - lo) / TWO32
        lo = hi
    return out


def accept_prob(p_t: float, q_t: float) -> float:
    """P(accepts(p_t, q_t, r)) for r uniform: the share of k in [0, 2^24)
    with fl32(k 2^-24 * q_t) < p_t.  The rounded product is monotone in k, so
    the accepted k form a prefix found by bisection."""
    p32, q32 = np.float32(p_t), np.float32(q_t)

    def ok(k: int) -> bool:
        return bool(np.float32(np.float32(k * 2.0 ** -24) * q32) < p32)

    if ok(TWO24 - 1):
        return 1.0
    if not ok(0):
        return 0.0
    lo, hi = 0, TWO24 - 1            # ok(lo) true, ok(hi) false
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if ok(mid):
            lo = mid
        else:
            hi = mid
    return hi / TWO24


def first_token_law(q: np.ndarray, p: np.ndarray) -> np.ndarray:
    """Exact law of the first token emitted by one speculative step, given
    the float32 draft distribution q and target distribution p of the first
    position: the first draft is accepted with its acceptance probability,
    otherwise the correction token is drawn from the residual (falling back
    to p when the residual has no integer mass)."""
    Pq = sample_law(q)
    A = np.array([accept_prob(p[x], q[x]) for x in range(len(q))])
    res = residual(p, q)
    R = sample_law(res) if sum(fixed_weights(res)) > 0 else sample_law(p)
    reject = float(np.sum(Pq * (1.0 - A)))
    return Pq * A + reject * R


def quantisation_bound(V: int) -> float:
    """Total-variation slack of the integer rules: each sample loses at most
    V * 2^-40 of mass to flooring and 2^-32 per entry to the threshold, and
    each acceptance probability is quantised to 2^-24 (plus float32 rounding
    of the product)."""
    return 4 * (V * 2.0 ** -40 + V * 2.0 ** -32 + 2.0 ** -24) + 1e-7
