"""Oracle transformer (test infrastructure only).

The paper's decoder block (Section II-A, eqs. f11, f21, f31 for prefill and
d_kv, d_atte, d_out for the cached decoding stage) is query/key/value
projections, softmax(Q K^T / sqrt(d0)) V W_O with a residual, then a
feed-forward network with a residual.  The workloads here use the LLaMA
layout of that block: RMSNorm before each sub-block and before the LM head,
rotary position embedding on queries and keys, SwiGLU feed-forward, and
grouped KV heads.  d0 is the head dimension.

Precision (the model definition, shared with the GPU path):
  * fp32 models: no storage rounding anywhere.
  * bf16 models: the weights are bf16 values.  The products take their
    operands in IEEE fp16: the projection matrices and the LM head enter as
    the nearest fp16 of each bf16 weight (the same value from 2^-14 up;
    smaller magnitudes round to fp16's subnormal grid of 2^-24); every
    matrix-product input (the normed activations, the attention output, the
    SwiGLU output) is rounded to the nearest fp16; keys and values are stored
    in the cache as fp16.  The embedding rows and norm gains are used as bf16
    values.  The residual stream, norms, rotary embedding, softmax and all
    accumulations are exact here (float64).
  * the plain form of a bf16 model (round_activations=False): the bf16
    weights as they are and nothing else rounded; every activation and the
    KV cache stay float64.  This is the unquantised model an implementation
    approximates, and the reference for its overall error.

The KV cache is the paper's per-block K^j, V^j, grown by concatenation
(eq. d_kv) and truncated on rollback.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence

import numpy as np


def round_bf16(x) -> np.ndarray:
    """Nearest bf16 value (ties to even) of float64 data, returned as float64."""
    a = np.array(x, dtype=np.float64, copy=True)
    u = a.view(np.uint64)
    drop = np.uint64(45)                       # 52 - 7 mantissa bits dropped
    lsb = (u >> drop) & np.uint64(1)
    u += np.uint64((1 << 44) - 1) + lsb        # half an ulp minus one, plus the lsb: ties to even
    u &= ~np.uint64((1 << 45) - 1)
    # below 2^-126 bf16 is subnormal, with a fixed spacing of 2^-133
    x64 = np.asarray(x, dtype=np.float64)
    tiny = np.abs(x64) < 2.0 ** -126
    if np.any(tiny):
        a[tiny] = np.round(x64[tiny] * 2.0 ** 133) * 2.0 ** -133   # np.round: ties to even
    return a


def round_fp16(x) -> np.ndarray:
    """Nearest IEEE fp16 value (ties to even, subnormals kept) of float64
    data, returned as float64 (numpy converts float64 to float16 directly,
    with one rounding)."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


# the weights a product reads (the projection matrices and the LM head)
_MATRICES = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def is_matrix(name: str) -> bool:
    return name == "lm_head" or name.split(".")[-1] in _MATRICES


def _decode_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """bf16 bit patterns (uint16) or float32 values -> float64, exactly (a
    plain dtype conversion; torch's is used for bf16, which numpy lacks)."""
    if dtype == "bf16":
        import torch
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).view(torch.bfloat16)
        return t.to(torch.float64).numpy()
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def weights_to_f64(w: Dict[str, np.ndarray], dtype: str) -> Dict[str, np.ndarray]:
    """Decode stored weights (bf16 bit patterns or float32) into float64 (exact)."""
    return {k: _decode_f64(a, dtype) for k, a in w.items()}


class LazyF64:
    """Read-only mapping name -> float64 weight that decodes the stored
    tensor (bf16 bits or float32) on every access and keeps nothing, so a
    model whose float64 weights do not fit in memory can be run one layer at
    a time (Model.sequence_logits reads each tensor once).  operands=True
    gives the matrices as the products read them (round_fp16)."""

    def __init__(self, w: Dict[str, np.ndarray], dtype: str, operands: bool = False):
        self.src, self.dtype, self.operands = w, dtype, operands

    def __getitem__(self, name: str) -> np.ndarray:
        a = _decode_f64(self.src[name], self.dtype)
        return round_fp16(a) if self.operands and is_matrix(name) else a

    def __contains__(self, name: str) -> bool:
        return name in self.src


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def rope(x: np.ndarray, pos, theta: float) -> np.ndarray:
    """Rotary embedding, rotate-half pairing (i, i + hd/2), frequency
    theta^(-2i/hd) for i < hd/2, absolute 0-based position.
    x: [..., n_heads, hd]; pos: scalar or [...] broadcast over heads."""
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(pos, dtype=np.float64)[..., None, None] * inv
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax64(z: np.ndarray) -> np.ndarray:
    m = np.max(z, axis=-1, keepdims=True)
    e = np.exp(z - m)
    return e / np.sum(e, axis=-1, keepdims=True)


class KVCache:
    """Per-layer K and V of one task: K[l] is [n_tokens, n_kv_heads, hd]."""

    def __init__(self, n_layers: int, n_kv: int, hd: int):
        self.K: List[np.ndarray] = [np.zeros((0, n_kv, hd)) for _ in range(n_layers)]
        self.V: List[np.ndarray] = [np.zeros((0, n_kv, hd)) for _ in range(n_layers)]

    def __len__(self) -> int:
        return self.K[0].shape[0]

    def append(self, l: int, k: np.ndarray, v: np.ndarray) -> None:
        self.K[l] = np.concatenate([self.K[l], k.reshape(-1, *self.K[l].shape[1:])])
        self.V[l] = np.concatenate([self.V[l], v.reshape(-1, *self.V[l].shape[1:])])

    def truncate(self, n: int) -> None:
        """Rollback: keep the first n positions."""
        for l in range(len(self.K)):
            self.K[l] = self.K[l][:n]
            self.V[l] = self.V[l][:n]

    def copy(self) -> "KVCache":
        c = KVCache.__new__(KVCache)
        c.K = [k.copy() for k in self.K]
        c.V = [v.copy() for v in self.V]
        return c


def causal_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, p0: int) -> np.ndarray:
    """Attention of n consecutive query rows, row i at position p0 + i,
    each over exactly the keys at positions 0 .. p0 + i (eq. f21 with the
    causal mask of a decoder): q [n, H, hd], K, V [p0 + n, KV, hd]; query
    head h reads kv head h // (H / KV); scale 1 / sqrt(hd).  The mask is
    applied by giving the invisible keys a weight of exactly zero."""
    n, H, hd = q.shape
    group = H // K.shape[1]
    vis = np.arange(K.shape[0])[None, :] <= (p0 + np.arange(n))[:, None]     # [n, keys]
    out = np.empty((n, H, hd))
    for h in range(H):
        s = q[:, h, :] @ K[:, h // group, :].T / math.sqrt(hd)               # [n, keys]
        s = np.where(vis, s, -np.inf)
        e = np.exp(s - s.max(axis=1, keepdims=True))
        out[:, h, :] = (e / e.sum(axis=1, keepdims=True)) @ V[:, h // group, :]
    return out


class Model:
    """A decoder-only model: shape (synth.ModelShape-like) + float64 weights.

    round_activations (bf16 models only): True applies the bf16 storage
    points of the model definition above; False gives the plain form (bf16
    weights, float64 everything else).  lazy=True decodes each weight on
    access instead of holding all of them in float64 (for models whose
    float64 weights exceed host memory; use sequence_logits then)."""

    def __init__(self, shape, weights: Dict[str, np.ndarray], round_activations: bool = True,
                 lazy: bool = False):
        self.s = shape
        self.bf16 = shape.dtype == "bf16" and round_activations
        if lazy:
            self.w = LazyF64(weights, shape.dtype)
            self.ops = LazyF64(weights, shape.dtype, operands=self.bf16)
        else:
            self.w = weights_to_f64(weights, shape.dtype)
            self.ops = ({k: round_fp16(v) if is_matrix(k) else v for k, v in self.w.items()} if self.bf16
                        else self.w)

    # storage rounding point of a bf16 model: an fp16 operand
    def r(self, x: np.ndarray) -> np.ndarray:
        return round_fp16(x) if self.bf16 else x

    def new_cache(self) -> KVCache:
        return KVCache(self.s.n_layers, self.s.n_kv_heads, self.s.head_dim)

    def attention(self, q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
        """One query position q [H, hd] over exactly its visible keys
        K, V [n, KV, hd]; query head h reads kv head h // (H / KV)."""
        H, hd = q.shape
        group = H // K.shape[1]
        out = np.empty((H, hd))
        for h in range(H):
            kh, vh = K[:, h // group, :], V[:, h // group, :]
            p = softmax64(kh @ q[h] / math.sqrt(hd))
            out[h] = p @ vh
        return out

    def decode_row(self, cache: KVCache, token: int, pos: int) -> np.ndarray:
        """Process one token at absolute position pos == len(cache); appends
        its K/V to the cache and returns its next-token logits [vocab]."""
        s, w = self.s, self.ops
        assert pos == len(cache), (pos, len(cache))
        H, KV, hd = s.n_heads, s.n_kv_heads, s.head_dim
        x = w["embed"][int(token)].copy()
        for l in range(s.n_layers):
            p = f"l{l}."
            h = self.r(rmsnorm(x, w[p + "attn_norm"], s.rms_eps))
            q = rope((w[p + "wq"] @ h).reshape(H, hd), pos, s.rope_theta)
            k = rope((w[p + "wk"] @ h).reshape(KV, hd), pos, s.rope_theta)
            v = (w[p + "wv"] @ h).reshape(KV, hd)
            cache.append(l, self.r(k), self.r(v))
            o = self.attention(q, cache.K[l], cache.V[l]).reshape(-1)
            x = x + w[p + "wo"] @ self.r(o)
            h = self.r(rmsnorm(x, w[p + "ffn_norm"], s.rms_eps))
            a = silu(w[p + "w_gate"] @ h) * (w[p + "w_up"] @ h)
            x = x + w[p + "w_down"] @ self.r(a)
        h = self.r(rmsnorm(x, w["final_norm"], s.rms_eps))
        return w["lm_head"] @ h

    def forward_rows(self, cache: KVCache, tokens: Sequence[int], logits: bool = True) -> np.ndarray:
        """Consecutive tokens at positions len(cache)..; same arithmetic as
        repeated decode_row (row i attends to keys 0..its own position), with
        the projections done as one matrix product over the rows.  Appends
        their K/V; returns logits [n, vocab] (or None: then the rows' output
        of the last layer is never used, and only its K/V are computed)."""
        s, w = self.s, self.ops
        H, KV, hd = s.n_heads, s.n_kv_heads, s.head_dim
        n = len(tokens)
        p0 = len(cache)
        pos = np.arange(p0, p0 + n)
        x = w["embed"][np.asarray(tokens, dtype=np.int64)].copy()
        for l in range(s.n_layers):
            p = f"l{l}."
            h = self.r(rmsnorm(x, w[p + "attn_norm"], s.rms_eps))
            q = rope((h @ w[p + "wq"].T).reshape(n, H, hd), pos, s.rope_theta)
            k = rope((h @ w[p + "wk"].T).reshape(n, KV, hd), pos, s.rope_theta)
            v = (h @ w[p + "wv"].T).reshape(n, KV, hd)
            cache.append(l, self.r(k), self.r(v))
            if not logits and l == s.n_layers - 1:
                return None
            o = np.stack([self.attention(q[i], cache.K[l][:p0 + i + 1], cache.V[l][:p0 + i + 1])
                          for i in range(n)]).reshape(n, -1)
            x = x + self.r(o) @ w[p + "wo"].T
            h = self.r(rmsnorm(x, w[p + "ffn_norm"], s.rms_eps))
            a = silu(h @ w[p + "w_gate"].T) * (h @ w[p + "w_up"].T)
            x = x + self.r(a) @ w[p + "w_down"].T
        if not logits:
            return None
        h = self.r(rmsnorm(x, w["final_norm"], s.rms_eps))
        return h @ w["lm_head"].T

    def unrounded(self) -> "Model":
        """The plain form of this model (same weights, no activation or KV
        rounding), sharing the decoded weights."""
        m = Model.__new__(Model)
        m.s, m.w, m.ops, m.bf16 = self.s, self.w, self.w, False
        return m

    def sequence_logits(self, seqs, n_out):
        """Logits of the last n_out tokens of each sequence of token ids,
        each sequence starting at position 0 of an empty cache: the rows of
        all sequences go through one layer at a time (each weight is read
        once per call), with the attention of every row over exactly the
        keys of its own sequence up to its own position.  The same arithmetic
        as prefill + forward_rows, without a cache: keys and values are
        rounded where the cache would store them.  seqs: a list of token-id
        sequences (or one sequence); n_out: an int or one per sequence.
        Returns a list of [n_out, vocab] arrays (one array for one sequence)."""
        s, w = self.s, self.ops
        H, KV, hd = s.n_heads, s.n_kv_heads, s.head_dim
        single = len(seqs) > 0 and np.isscalar(seqs[0])
        seqs = [list(seqs)] if single else [list(q) for q in seqs]
        outs = [int(n_out)] * len(seqs) if np.isscalar(n_out) else [int(k) for k in n_out]
        lens = [len(q) for q in seqs]
        assert all(1 <= o <= n for o, n in zip(outs, lens))
        starts = np.cumsum([0] + lens)
        pos = np.concatenate([np.arange(n) for n in lens])
        x = w["embed"][np.concatenate([np.asarray(q, dtype=np.int64) for q in seqs])]
        for l in range(s.n_layers):
            p = f"l{l}."
            last = l == s.n_layers - 1
            h = self.r(rmsnorm(x, w[p + "attn_norm"], s.rms_eps))
            q = rope((h @ w[p + "wq"].T).reshape(-1, H, hd), pos, s.rope_theta)
            k = self.r(rope((h @ w[p + "wk"].T).reshape(-1, KV, hd), pos, s.rope_theta))
            v = self.r((h @ w[p + "wv"].T).reshape(-1, KV, hd))
            o, keep = [], []
            for i, (a, n) in enumerate(zip(starts[:-1], lens)):
                m = outs[i] if last else n            # the last layer needs only the output rows
                o.append(causal_attention(q[a + n - m:a + n], k[a:a + n], v[a:a + n], n - m).reshape(m, -1))
                keep.append(np.arange(a + n - m, a + n))
            if last:
                x = x[np.concatenate(keep)]
            x = x + self.r(np.concatenate(o)) @ w[p + "wo"].T
            h = self.r(rmsnorm(x, w[p + "ffn_norm"], s.rms_eps))
            a_ = silu(h @ w[p + "w_gate"].T) * (h @ w[p + "w_up"].T)
            x = x + self.r(a_) @ w[p + "w_down"].T
        h = self.r(rmsnorm(x, w["final_norm"], s.rms_eps))
        z = h @ w["lm_head"].T
        res = np.split(z, np.cumsum(outs)[:-1])
        return res[0] if single else res

    def prefill(self, tokens: Sequence[int], batch_rows: bool = False) -> KVCache:
        """Fresh cache holding the K/V of ``tokens`` at positions 0..n-1."""
        c = self.new_cache()
        if batch_rows and len(tokens):
            self.forward_rows(c, tokens, logits=False)
        else:
            for i, t in enumerate(tokens):
                self.decode_row(c, t, i)
        return c
