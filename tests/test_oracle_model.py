"""Pins of the oracle transformer against closed forms, hand-computed values
and independent library routines (torch CPU, float64)."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle import model as om


def tiny_shape(dtype="fp32", kv=2):
    return synth.ModelShape(n_layers=2, d_model=64, n_heads=4, n_kv_heads=kv,
                            d_ffn=96, vocab=40, dtype=dtype)


# ---------------------------------------------------------------- bf16 rounding

def test_round_bf16_hand_cases():
    one = 1.0
    ulp = 2.0 ** -7                       # bf16 spacing in [1, 2)
    cases = [
        (one, one),
        (one + ulp / 2, one),             # tie -> even (mantissa 0)
        (one + 1.5 * ulp, one + 2 * ulp),  # tie -> even (mantissa 2)
        (one + ulp / 2 + 2.0 ** -40, one + ulp),   # just above the tie
        (one + ulp / 2 - 2.0 ** -40, one),         # just below the tie
        (-(one + 1.5 * ulp), -(one + 2 * ulp)),
        (3.0e-39, None),                  # subnormal range handled like the rest
        (0.0, 0.0),
    ]
    for x, want in cases:
        got = float(om.round_bf16(x))
        if want is not None:
            assert got == want, (x, got, want)
    # idempotent, and exactly representable in bf16: low 16 bits of fp32 zero
    r = om.round_bf16(np.array([0.1, -3.7, 1e-3, 12345.678]))
    assert np.all(om.round_bf16(r) == r)
    assert np.all(r.astype(np.float32).view(np.uint32) & 0xFFFF == 0)


def test_round_bf16_matches_torch_on_fp32_values():
    # torch converts through float32; on float32-representable inputs that is
    # a single rounding, so it must agree bit for bit
    x = np.random.default_rng(0).standard_normal(200000).astype(np.float32)
    hi = np.random.default_rng(1).integers(0, 2**16, 1000).astype(np.uint32)
    hi = hi[((hi >> 7) & 0xFF) != 0xFF]                  # finite values only
    x[:len(hi)] = (hi << 16 | np.uint32(0x8000)).view(np.float32)     # exact ties
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = om.round_bf16(x.astype(np.float64))
    assert np.array_equal(got, want)


def test_weights_decode_roundtrip():
    shape = tiny_shape("bf16")
    w = synth.model_weights(shape, seed=3, names=["l0.wq"])
    f = om.weights_to_f64(w, "bf16")["l0.wq"]
    # a bf16 pattern is the upper half of the float32 with the same value
    t = (w["l0.wq"].astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    assert np.array_equal(f, t)
    # and hand values: 0x3F80 = 1.0, 0xC040 = -3.0, 0x0001 = 2^-133 (smallest subnormal)
    hand = om.weights_to_f64({"x": np.array([0x3F80, 0xC040, 0x0001, 0x7F7F], np.uint16)}, "bf16")["x"]
    assert list(hand[:3]) == [1.0, -3.0, 2.0 ** -133] and hand[3] == float.fromhex("0x1.fep127")

# ---------------------------------------------------------------- building blocks


def test_rmsnorm_closed_form():
    n, c, eps = 16, -0.37, 1e-5
    g = np.linspace(0.5, 1.5, n)
    y = om.rmsnorm(np.full(n, c), g, eps)
    assert np.allclose(y, np.sign(c) * g * abs(c) / math.sqrt(c * c + eps), rtol=1e-14)
    x = np.random.default_rng(2).standard_normal((3, n))
    want = F.rms_norm(torch.from_numpy(x), (n,), torch.from_numpy(g), eps).numpy()
    assert np.allclose(om.rmsnorm(x, g, eps), want, rtol=1e-13, atol=1e-15)


def test_rope_hand_example():
    # hd = 4, theta = 10000: frequencies 1 and 10000^-0.5 = 0.01, pairs (0,2), (1,3)
    x = np.array([[1.0, 2.0, 3.0, 4.0]])
    y = om.rope(x, 1, 10000.0)[0]
    c1, s1, c2, s2 = math.cos(1), math.sin(1), math.cos(0.01), math.sin(0.01)
    want = [1 * c1 - 3 * s1, 2 * c2 - 4 * s2, 1 * s1 + 3 * c1, 2 * s2 + 4 * c2]
    assert np.allclose(y, want, rtol=0, atol=1e-15)
    assert np.array_equal(om.rope(x, 0, 10000.0), x)        # position 0 is the identity


def test_rope_relative_and_norm():
    rng = np.random.default_rng(4)
    q, k = rng.standard_normal((1, 128)), rng.standard_normal((1, 128))
    for m, n, s in [(5, 3, 7), (1000, 1, 900), (17, 17, 2000)]:
        a = om.rope(q, m, 1e4)[0] @ om.rope(k, n, 1e4)[0]
        b = om.rope(q, m + s, 1e4)[0] @ om.rope(k, n + s, 1e4)[0]
        assert abs(a - b) < 1e-9
        assert abs(np.linalg.norm(om.rope(q, m, 1e4)) - np.linalg.norm(q)) < 1e-12


def test_attention_vs_torch_sdpa_gqa():
    rng = np.random.default_rng(5)
    shape = tiny_shape(kv=2)
    m = om.Model.__new__(om.Model)
    m.s = shape
    H, KV, hd, n = 4, 2, 16, 9
    q = rng.standard_normal((H, hd))
    K = rng.standard_normal((n, KV, hd))
    V = rng.standard_normal((n, KV, hd))
    got = om.Model.attention(m, q, K, V)
    tq = torch.from_numpy(q)[:, None, :]                 # [H, 1, hd]
    tk = torch.from_numpy(K).permute(1, 0, 2)            # [KV, n, hd]
    tv = torch.from_numpy(V).permute(1, 0, 2)
    want = F.scaled_dot_product_attention(tq[None], tk[None], tv[None], enable_gqa=True)[0, :, 0]
    assert np.allclose(got, want.numpy(), rtol=1e-12, atol=1e-13)

# ---------------------------------------------------------------- whole model


def torch_reference_logits(shape, w64, tokens, rnd=None):
    """Full causal forward over all tokens with torch library routines:
    F.rms_norm, scaled_dot_product_attention(is_causal, GQA), F.silu.
    rnd: rounding function applied at the model's storage points."""
    rnd = rnd or (lambda t: t)
    T = lambda a: torch.from_numpy(a)
    H, KV, hd, eps = shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.rms_eps
    n = len(tokens)
    x = T(w64["embed"])[torch.tensor(tokens)]
    pos = torch.arange(n, dtype=torch.float64)
    inv = shape.rope_theta ** (-2.0 * torch.arange(hd // 2, dtype=torch.float64) / hd)
    ang = pos[:, None] * inv[None, :]
    cos, sin = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]

    def rot(t):                                     # [n, heads, hd]
        a, b = t[..., :hd // 2], t[..., hd // 2:]
        return torch.cat([a * cos - b * sin, a * sin + b * cos], -1)

    for l in range(shape.n_layers):
        p = f"l{l}."
        h = rnd(F.rms_norm(x, (shape.d_model,), T(w64[p + "attn_norm"]), eps))
        q = rot((h @ T(w64[p + "wq"]).T).view(n, H, hd))
        k = rnd(rot((h @ T(w64[p + "wk"]).T).view(n, KV, hd)))
        v = rnd((h @ T(w64[p + "wv"]).T).view(n, KV, hd))
        o = F.scaled_dot_product_attention(q.permute(1, 0, 2)[None], k.permute(1, 0, 2)[None],
                                           v.permute(1, 0, 2)[None], is_causal=True, enable_gqa=True)
        o = o[0].permute(1, 0, 2).reshape(n, H * hd)
        x = x + rnd(o) @ T(w64[p + "wo"]).T
        h = rnd(F.rms_norm(x, (shape.d_model,), T(w64[p + "ffn_norm"]), eps))
        a = F.silu(h @ T(w64[p + "w_gate"]).T) * (h @ T(w64[p + "w_up"]).T)
        x = x + rnd(a) @ T(w64[p + "w_down"]).T
    h = rnd(F.rms_norm(x, (shape.d_model,), T(w64["final_norm"]), eps))
    return (h @ T(w64["lm_head"]).T).numpy()


@pytest.mark.parametrize("kv", [4, 2, 1])
def test_decode_rows_vs_torch_full_forward_fp32(kv):
    shape = tiny_shape("fp32", kv)
    w = synth.model_weights(shape, seed=11)
    m = om.Model(shape, w)
    toks = list(np.random.default_rng(6).integers(0, shape.vocab, 13))
    c = m.new_cache()
    got = np.stack([m.decode_row(c, t, i) for i, t in enumerate(toks)])
    want = torch_reference_logits(shape, m.w, toks)
    assert np.allclose(got, want, rtol=1e-10, atol=1e-12)


def test_decode_rows_vs_torch_full_forward_bf16():
    shape = tiny_shape("bf16", 2)
    w = synth.model_weights(shape, seed=12)
    m = om.Model(shape, w)
    toks = list(np.random.default_rng(7).integers(0, shape.vocab, 11))
    c = m.new_cache()
    got = np.stack([m.decode_row(c, t, i) for i, t in enumerate(toks)])
    # fp16 operands at every storage point and for the matrices (round_fp16
    # is pinned on its own below; torch's float64 -> float16 conversion goes
    # through float32, two roundings, so it is not used here)
    rnd = lambda t: torch.from_numpy(om.round_fp16(t.numpy()))
    ops = {k: (om.round_fp16(v) if om.is_matrix(k) else v) for k, v in m.w.items()}
    want = torch_reference_logits(shape, ops, toks, rnd)
    # a storage point can flip by one ulp when float64 rounding order
    # differs; the two must otherwise agree
    rel = np.abs(got - want).max() / np.abs(want).max()
    assert rel < 1e-6, rel
    # and the rounding points matter: without them the logits move visibly
    plain = torch_reference_logits(shape, m.w, toks)
    assert np.abs(got - plain).max() / np.abs(plain).max() > 1e-5


def test_round_fp16_hand_cases_and_library():
    one, ulp = 1.0, 2.0 ** -10                # fp16 spacing in [1, 2)
    cases = [(one + ulp / 2, one), (one + 1.5 * ulp, one + 2 * ulp),            # ties to even
             (one + ulp / 2 + 2.0 ** -40, one + ulp),                           # one rounding, not two
             (-(one + 1.5 * ulp), -(one + 2 * ulp)), (65504.0, 65504.0),
             (2.0 ** -24, 2.0 ** -24), (2.0 ** -25, 0.0), (3 * 2.0 ** -25, 2.0 ** -23),   # subnormals
             (3e-5, round(3e-5 / 2.0 ** -24) * 2.0 ** -24)]
    for x, want in cases:
        assert float(om.round_fp16(x)) == want, (x, float(om.round_fp16(x)), want)
    x = np.random.default_rng(2).standard_normal(100000).astype(np.float32) * 3
    want = torch.from_numpy(x).to(torch.float16).to(torch.float64).numpy()   # one rounding from float32
    assert np.array_equal(om.round_fp16(x.astype(np.float64)), want)


def test_bf16_model_operands():
    """The products of a bf16 model read each matrix as fp16: the bf16 value
    itself from 2^-14 up, the fp16 subnormal grid below; embedding rows and
    norm gains are read as they are; the plain form reads nothing rounded."""
    shape = tiny_shape("bf16", 2)
    w = synth.model_weights(shape, seed=18)
    m = om.Model(shape, w)
    for k, v in m.w.items():
        if om.is_matrix(k):
            big = np.abs(v) >= 2.0 ** -14
            assert np.array_equal(m.ops[k][big], v[big]), k
            assert np.all(np.abs(m.ops[k] - v) <= 2.0 ** -25), k
            assert np.array_equal(m.ops[k], om.round_fp16(v))
        else:
            assert m.ops[k] is v, k
    assert {k for k in m.w if om.is_matrix(k)} == {k for k in m.w if k == "lm_head" or k.split(".")[-1] in (
        "wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")}
    assert m.unrounded().ops is m.w
    lazy = om.Model(shape, w, lazy=True)
    for k in m.w:
        assert np.array_equal(lazy.ops[k], m.ops[k]), k


def test_kv_incremental_equals_batched_rows():
    shape = tiny_shape("bf16", 2)
    m = om.Model(shape, synth.model_weights(shape, seed=13))
    toks = list(np.random.default_rng(8).integers(0, shape.vocab, 20))
    c1 = m.prefill(toks[:12])
    z1 = np.stack([m.decode_row(c1, t, 12 + i) for i, t in enumerate(toks[12:])])
    c2 = m.prefill(toks[:12], batch_rows=True)
    z2 = m.forward_rows(c2, toks[12:])
    assert np.allclose(z1, z2, rtol=1e-9, atol=1e-11)
    for l in range(shape.n_layers):
        assert np.allclose(c1.K[l], c2.K[l], rtol=0, atol=1e-2)   # bf16 values, may differ by an ulp
        assert np.mean(c1.K[l] == c2.K[l]) > 0.999


def test_table1_shapes_golden():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "table1_model_shapes.txt")
    rows = {}
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            name, L, h, f = line.split()
            rows[name] = (int(L), int(h), int(f))
    M = synth.MODELS
    assert (M["small_draft"].n_layers, M["small_draft"].d_model, M["small_draft"].d_ffn) == rows["LLaMA-68M"]
    assert (M["7b_target"].n_layers, M["7b_target"].d_model, M["7b_target"].d_ffn) == rows["LLaMA-7B"]
    assert (M["13b_target"].n_layers, M["13b_target"].d_model, M["13b_target"].d_ffn) == rows["LLaMA-13B"]
    assert M["small_target"].d_model == rows["LLaMA-1.1B"][1] and M["small_target"].d_ffn == rows["LLaMA-1.1B"][2]
    # the paper's footprint for LLaMA-7B in FP16 is about 14 GB (Section II)
    assert 13e9 < 2 * M["7b_target"].n_params() < 14.5e9


# ---------------------------------------------------------------- plain model, whole-sequence forward

def test_plain_bf16_model_vs_torch_full_forward():
    """round_activations=False: bf16 weights and nothing else rounded, equal
    to the independent torch formulation without rounding points."""
    shape = tiny_shape("bf16", 2)
    w = synth.model_weights(shape, seed=14)
    m = om.Model(shape, w, round_activations=False)
    toks = list(np.random.default_rng(9).integers(0, shape.vocab, 12))
    c = m.new_cache()
    got = np.stack([m.decode_row(c, t, i) for i, t in enumerate(toks)])
    want = torch_reference_logits(shape, m.w, toks)
    assert np.allclose(got, want, rtol=1e-10, atol=1e-12)
    # the rounded model differs from it by its storage points only
    r = om.Model(shape, w)
    c = r.new_cache()
    zr = np.stack([r.decode_row(c, t, i) for i, t in enumerate(toks)])
    assert np.abs(zr - got).max() / np.abs(got).max() > 1e-4


def test_causal_attention_vs_torch_sdpa_with_offset():
    """n query rows at positions p0 .. p0 + n - 1 over p0 + n keys: torch's
    attention with an explicit mask (key j visible to row i iff j <= p0 + i)."""
    rng = np.random.default_rng(10)
    H, KV, hd, p0, n = 4, 2, 16, 7, 5
    q = rng.standard_normal((n, H, hd))
    K = rng.standard_normal((p0 + n, KV, hd))
    V = rng.standard_normal((p0 + n, KV, hd))
    got = om.causal_attention(q, K, V, p0)
    mask = torch.arange(p0 + n)[None, :] <= (p0 + torch.arange(n))[:, None]
    want = F.scaled_dot_product_attention(torch.from_numpy(q).permute(1, 0, 2)[None],
                                          torch.from_numpy(K).permute(1, 0, 2)[None],
                                          torch.from_numpy(V).permute(1, 0, 2)[None],
                                          attn_mask=mask, enable_gqa=True)[0].permute(1, 0, 2)
    assert np.allclose(got, want.numpy(), rtol=1e-12, atol=1e-13)
    # one row is the single-query attention of the decoder
    m = om.Model.__new__(om.Model)
    m.s = tiny_shape(kv=KV)
    assert np.allclose(got[2], om.Model.attention(m, q[2], K[:p0 + 3], V[:p0 + 3]), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("dtype,rounded", [("fp32", True), ("bf16", True), ("bf16", False)])
def test_sequence_logits_equal_cached_rows(dtype, rounded):
    """The whole-sequence forward (one layer at a time, lazily decoded
    weights) gives the logits of prefill + forward_rows, and, for the plain
    model, those of the torch formulation."""
    shape = tiny_shape(dtype, 2)
    w = synth.model_weights(shape, seed=15)
    toks = list(np.random.default_rng(11).integers(0, shape.vocab, 16))
    m = om.Model(shape, w, round_activations=rounded)
    c = m.prefill(toks[:11], batch_rows=True)
    want = m.forward_rows(c, toks[11:])
    lazy = om.Model(shape, w, round_activations=rounded, lazy=True)
    got = lazy.sequence_logits(toks, 5)
    if dtype == "bf16" and rounded:
        # a bf16 storage point may flip by one ulp under another summation order
        assert np.abs(got - want).max() / np.abs(want).max() < 1e-6
    else:
        assert np.allclose(got, want, rtol=1e-10, atol=1e-12)
    if not rounded:
        assert np.allclose(got, torch_reference_logits(shape, m.w, toks)[11:], rtol=1e-10, atol=1e-12)
    assert np.allclose(lazy.sequence_logits(toks, 1), got[-1:], rtol=1e-12, atol=1e-13)


def test_lazy_weights_decode_like_eager():
    shape = tiny_shape("bf16", 2)
    w = synth.model_weights(shape, seed=16)
    eager = om.weights_to_f64(w, "bf16")
    lazy = om.LazyF64(w, "bf16")
    for k in eager:
        assert np.array_equal(lazy[k], eager[k]), k


def test_sequence_logits_of_several_sequences():
    """Several sequences in one call equal each sequence alone (rows of one
    sequence never see another's keys), and unrounded() is the plain model."""
    shape = tiny_shape("bf16", 2)
    w = synth.model_weights(shape, seed=17)
    rng = np.random.default_rng(12)
    seqs = [list(rng.integers(0, shape.vocab, n)) for n in (9, 4, 13)]
    m = om.Model(shape, w)
    many = m.sequence_logits(seqs, [3, 4, 1])
    for sq, o, z in zip(seqs, [3, 4, 1], many):
        assert z.shape == (o, shape.vocab)
        alone = m.sequence_logits(sq, o)
        assert np.abs(z - alone).max() / np.abs(alone).max() < 1e-6
    plain = om.Model(shape, w, round_activations=False)
    assert np.allclose(m.unrounded().sequence_logits(seqs[0], 2), plain.sequence_logits(seqs[0], 2),
                       rtol=1e-12, atol=1e-13)
