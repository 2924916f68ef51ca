"""sd_accept_resample against the oracle's rule, decision by decision: both
sides get the same float32 distributions and the same uint32 uniforms, so
the accepted length and every emitted token must agree exactly."""
import numpy as np
import pytest

import synth
from oracle import sampling as osp
from sdcase import say

pytestmark = pytest.mark.gpu


def build_case(V, gamma, B, seed):
    rng = np.random.default_rng(seed)
    q = np.zeros((B, gamma, V), np.float32)
    p = np.zeros((B, gamma + 1, V), np.float32)
    dt = np.zeros((B, gamma), np.int32)
    u = synth.uniforms(seed, range(B), 0, 2 * gamma + 1)
    for b in range(B):
        kind = b % 7
        sharp = [0.3, 1.0, 3.0][b % 3]
        for i in range(gamma + 1):
            p[b, i] = osp.softmax_f32(rng.standard_normal(V) * sharp, 1.0)
        for i in range(gamma):
            if kind == 1:                      # draft == target: always accepted
                q[b, i] = p[b, i]
            elif kind == 2:                    # disjoint supports
                half = V // 2
                q[b, i, :half] = osp.softmax_f32(rng.standard_normal(half), 1.0)
                p[b, i, :half] = 0
                p[b, i, half:] = osp.softmax_f32(rng.standard_normal(V - half), 1.0)
            elif kind == 3:                    # q = 2p: empty residual, fallback to p
                q[b, i] = np.float32(2) * p[b, i]
            elif kind == 5:                    # near q: high acceptance
                q[b, i] = osp.softmax_f32(np.log(p[b, i].astype(np.float64) + 1e-30)
                                          + 0.05 * rng.standard_normal(V), 1.0)
            else:
                q[b, i] = osp.softmax_f32(rng.standard_normal(V) * sharp, 1.0)
            t = osp.sample_weights(q[b, i], int(u[b, i]))
            dt[b, i] = 0 if t is None else t
            if kind == 4:                      # the drafted token has no target mass
                p[b, i, dt[b, i]] = 0
    return dt, q, p, u


def run_gpu(dt, q, p, u, greedy):
    import torch
    from paper_2510_11331_amd import accept_resample
    B, gamma = dt.shape
    V = q.shape[2]
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    n_acc = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    out = torch.full((B, gamma + 1), -7, dtype=torch.int32, device="cuda")
    accept_resample(B, gamma, V, greedy, T(dt), T(q), T(p), T(u.view(np.int32)), n_acc, out)
    torch.cuda.synchronize()
    return n_acc.cpu().numpy(), out.cpu().numpy()


@pytest.mark.parametrize("V,gamma", [(16, 1), (16, 4), (1024, 3), (32000, 4), (32000, 8)])
def test_accept_resample_bit_exact(V, gamma):
    say("accept_resample", V, gamma)
    B = 70
    dt, q, p, u = build_case(V, gamma, B, seed=V + gamma)
    n_acc, out = run_gpu(dt, q, p, u, greedy=False)
    kinds = set()
    for b in range(B):
        a, em = osp.accept_resample(dt[b], q[b], p[b], u[b, gamma:2 * gamma], int(u[b, 2 * gamma]))
        assert n_acc[b] == a, (b, n_acc[b], a)
        assert list(out[b, :a + 1]) == em, (b, out[b], em)
        assert np.all(out[b, a + 1:] == -1)
        kinds.add((a == gamma, a == 0))
    assert len(kinds) >= 2                  # both full acceptance and rejection occurred


@pytest.mark.parametrize("V,gamma", [(16, 3), (32000, 4)])
def test_accept_greedy_bit_exact(V, gamma):
    say("accept_greedy", V, gamma)
    rng = np.random.default_rng(3 + V)
    B = 40
    p = rng.standard_normal((B, gamma + 1, V)).astype(np.float32)       # target logits
    q = rng.standard_normal((B, gamma, V)).astype(np.float32)
    p[::5, :, 3] = p[::5, :, 7] = 50.0                                   # exact ties -> lowest index
    dt = np.zeros((B, gamma), np.int32)
    for b in range(B):
        for i in range(gamma):
            dt[b, i] = osp.argmax_lowest(p[b, i]) if rng.random() < 0.7 else rng.integers(V)
    u = synth.uniforms(9, range(B), 0, 2 * gamma + 1)
    n_acc, out = run_gpu(dt, q, p, u, greedy=True)
    for b in range(B):
        a, em = osp.accept_resample(dt[b], q[b], p[b], u[b, gamma:2 * gamma], 0, greedy=True)
        assert n_acc[b] == a and list(out[b, :a + 1]) == em, b
