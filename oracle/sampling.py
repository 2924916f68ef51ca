"""Oracle sampling rules (test infrastructure only).

Speculative sampling (Section II-A, verification phase, after Leviathan et
al.): draft token t_l is accepted with probability min(1, p_l(t_l)/q_l(t_l));
at the first rejected position the correction token is drawn from
norm(max(0, p_l - q_l)); if all l drafts are accepted, a reward token is drawn
from the target distribution of the next position.  Exactly one such bonus
token follows the accepted prefix.

The paper leaves the random-number details open.  The rules below are the
readings the GPU path shares; both sides take every decision on the same
float32 distributions and the same uint32 uniforms:

* acceptance: with u = (r >> 8) * 2^-24 (a float32 in [0, 1)), accept iff the
  correctly rounded float32 product u * q(t) is below p(t).  This is
  u < min(1, p/q) without a division; p(t) = 0 always rejects, q(t) = 0
  accepts iff p(t) > 0.
* sampling from a weight vector w (float32, >= 0, any scale):
  W_j = floor(w_j * 2^40) as an integer (exact), S = sum W_j,
  T = floor(S * r / 2^32), pick the smallest j whose prefix sum exceeds T.
  This samples w / sum(w) to within V * 2^-40 of mass and makes the result
  independent of summation order.  If S = 0 the caller falls back.
* residual weights: max(0, p_j - q_j) with the float32 subtraction correctly
  rounded.
* greedy mode: the distributions are point masses at the arg-max (lowest
  index on ties) of the logits; a draft token is accepted iff it equals the
  target arg-max, and the bonus token is the target arg-max.
"""
from __future__ import annotations

from typing import Sequence, Tuple

import numpy as np

TWO40 = float(2 ** 40)


def softmax_f32(z: np.ndarray, tau: float) -> np.ndarray:
    """softmax(z / tau) over the last axis, computed in float64 and delivered
    as the float32 distribution the sampling rules consume."""
    z = np.asarray(z, dtype=np.float64) / tau
    m = np.max(z, axis=-1, keepdims=True)
    e = np.exp(z - m)
    return (e / np.sum(e, axis=-1, keepdims=True)).astype(np.float32)


def argmax_lowest(z: np.ndarray) -> int:
    """Index of the maximum; the lowest index among equal maxima."""
    z = np.asarray(z)
    return int(np.flatnonzero(z == z.max())[0])


def fixed_weights(w: np.ndarray) -> list:
    """W_j = floor(w_j * 2^40) as Python integers (exact: w_j * 2^40 is an
    exact float64 for float32 w_j)."""
    w = np.asarray(w, dtype=np.float32)
    assert np.all(w >= 0)
    return [int(v) for v in np.floor(w.astype(np.float64) * TWO40)]


def threshold(S: int, r: int) -> int:
    """floor(S * r / 2^32) for a uint32 r."""
    return (S * int(r)) >> 32


def sample_weights(w: np.ndarray, r: int):
    """Integer inverse-CDF draw from weights w with uniform r (uint32).
    Returns the index, or None when every W_j is zero."""
    W = fixed_weights(w)
    S = sum(W)
    if S == 0:
        return None
    T = threshold(S, r)
    acc = 0
    for j, v in enumerate(W):
        acc += v
        if acc > T:
            return j
    raise AssertionError("unreachable: T < S")


def accept_u(r: int) -> np.float32:
    """The acceptance uniform u = (r >> 8) * 2^-24 as float32."""
    return np.float32((int(r) >> 8) * 2.0 ** -24)


def accepts(p_t: np.float32, q_t: np.float32, r: int) -> bool:
    """Ratio test: accept iff fl32(u * q(t)) < p(t)."""
    prod = np.float32(accept_u(r)) * np.float32(q_t)     # float32 * float32 -> rounded float32
    return bool(prod < np.float32(p_t))


def residual(p: np.ndarray, q: np.ndarray) -> np.ndarray:
    """max(0, p - q) with the float32 subtraction."""
    d = np.asarray(p, dtype=np.float32) - np.asarray(q, dtype=np.float32)
    return np.where(d > 0, d, np.float32(0)).astype(np.float32)


def accept_resample(draft: Sequence[int], q: np.ndarray, p: np.ndarray,
                    u_acc: Sequence[int], u_res: int, greedy: bool = False
                    ) -> Tuple[int, list]:
    """One verification decision for one task.

    draft [gamma] token ids; q [gamma, V] draft rows (float32 probabilities,
    or draft logits in greedy mode); p [gamma+1, V] target rows (float32
    probabilities, or target logits in greedy mode); u_acc [gamma] and u_res
    uint32 uniforms.  Returns (a, emitted) with a in [0, gamma] the number of
    accepted drafts and emitted = draft[:a] + [bonus] (length a + 1).
    """
    gamma = len(draft)
    a = gamma
    for i in range(gamma):
        t = int(draft[i])
        if greedy:
            ok = t == argmax_lowest(p[i])
        else:
            ok = accepts(p[i][t], q[i][t], u_acc[i])
        if not ok:
            a = i
            break
    if greedy:
        y = argmax_lowest(p[a])
    elif a < gamma:
        y = sample_weights(residual(p[a], q[a]), u_res)
        if y is None:                       # residual mass below 2^-40 per entry
            y = sample_weights(p[a], u_res)
    else:
        y = sample_weights(p[gamma], u_res)
    return a, [int(t) for t in draft[:a]] + [int(y)]


def draft_sample(z: np.ndarray, tau: float, r: int, greedy: bool):
    """Draft token from draft logits z: (token, q row).  q is the float32
    softmax(z / tau) (the logits themselves in greedy mode)."""
    if greedy:
        return argmax_lowest(z), np.asarray(z, dtype=np.float32)
    q = softmax_f32(z, tau)
    return sample_weights(q, r), q
