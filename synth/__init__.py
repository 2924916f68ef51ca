"""Seeded synthetic inputs for the speculative-decoding hot path.

This module is the only code shared by the oracle side (tests, bench's CPU
baseline) and the GPU side (binding, bench).  It holds no arithmetic of the
method itself: it only draws numbers and fixes model shapes.

* Model shapes and workloads.  The target/draft shapes follow the paper's
  model table (Table I: LLaMA-68M, LLaMA-7B, LLaMA-13B) in the LLaMA layout
  (RMSNorm, rotary embedding, SwiGLU feed-forward, optional grouped KV heads).
* Weights.  Every matrix (embedding and untied LM head included) is drawn from
  N(0, 0.02^2) in float32 with a per-tensor seeded PCG64 stream; bf16 models
  store the round-to-nearest-even bf16 value of that draw, so oracle and GPU
  see identical weight bits.  Norm gains are 1 + N(0, 0.1^2) so that a missing
  or misplaced gain shows up in parity tests.
* Prompts.  Uniform-random token ids; the paper's tasks are synthetic too
  (input and output lengths uniform, Section IV).
* Uniforms.  The random numbers speculative sampling consumes are drawn here,
  on the host, with SplitMix64 (Steele, Lea and Flood, 2014) used as a
  counter-based generator keyed by (seed, task, step, slot), and handed to
  both sides as uint32 arrays.
"""
from __future__ import annotations

import dataclasses
import os
import zlib
from concurrent.futures import ThreadPoolExecutor
from typing import Callable, Dict, Iterable, List, Optional, Sequence

import numpy as np

__all__ = [
    "ModelShape", "Workload", "MODELS", "WORKLOADS", "weight_names",
    "weight_shapes", "gen_tensor", "gen_tensor_chunks", "model_weights",
    "perturbed_weights", "bf16_bits", "bf16_bits_to_f32", "prompts",
    "ragged_lengths", "splitmix64", "uniforms", "uniform_table",
    "slot_layout",
]

# --------------------------------------------------------------------------
# shapes


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Decoder-only LLaMA-style model shape.

    ``dtype`` is the storage type of weights and KV cache: ``"bf16"`` or
    ``"fp32"``.
    """
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    d_ffn: int
    vocab: int
    dtype: str = "bf16"
    rope_theta: float = 10000.0
    rms_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    def replace(self, **kw) -> "ModelShape":
        return dataclasses.replace(self, **kw)

    def n_params(self) -> int:
        d, f, hd = self.d_model, self.d_ffn, self.head_dim
        per_layer = (d * (self.n_heads + 2 * self.n_kv_heads) * hd
                     + self.n_heads * hd * d + 3 * d * f + 2 * d)
        return self.n_layers * per_layer + 2 * self.vocab * d + d


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    target: ModelShape
    draft: ModelShape
    batch: int
    prompt_len: int          # fixed prompt length (0 = ragged, see prompt_range)
    gamma: int
    new_tokens: int
    temperature: float = 1.0
    greedy: bool = False
    prompt_range: Optional[tuple] = None
    kv_block: int = 16
    # forced acceptance rate (greedy verification, drafts replaced by the
    # target's greedy continuation with this probability); None: off
    alpha_forced: Optional[float] = None


MODELS: Dict[str, ModelShape] = {
    # tiny fp32 pair (CPU-in-seconds case)
    "tiny_target": ModelShape(2, 256, 4, 4, 1024, 1024, "fp32"),
    "tiny_draft": ModelShape(1, 128, 2, 2, 512, 1024, "fp32"),
    # small bf16 pair: GQA target, LLaMA-68M-shaped draft (Table I)
    "small_target": ModelShape(16, 2048, 32, 8, 5632, 32000, "bf16"),
    "small_draft": ModelShape(2, 768, 12, 12, 3072, 32000, "bf16"),
    # LLaMA-7B shape (Table I) and its 2-layer draft
    "7b_target": ModelShape(32, 4096, 32, 32, 11008, 32000, "bf16"),
    "7b_draft": ModelShape(2, 1024, 16, 16, 2816, 32000, "bf16"),
    # LLaMA-13B shape (Table I) and its 4-layer draft
    "13b_target": ModelShape(40, 5120, 40, 40, 13824, 32000, "bf16"),
    "13b_draft": ModelShape(4, 1024, 16, 16, 2816, 32000, "bf16"),
}

WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", MODELS["tiny_target"], MODELS["tiny_draft"],
                     batch=2, prompt_len=32, gamma=4, new_tokens=64),
    "small": Workload("small", MODELS["small_target"], MODELS["small_draft"],
                      batch=8, prompt_len=512, gamma=4, new_tokens=128),
    "7b_b1": Workload("7b_b1", MODELS["7b_target"], MODELS["7b_draft"],
                      batch=1, prompt_len=1024, gamma=4, new_tokens=256),
    "7b_b8": Workload("7b_b8", MODELS["7b_target"], MODELS["7b_draft"],
                      batch=8, prompt_len=1024, gamma=4, new_tokens=128),
    "7b_paged": Workload("7b_paged", MODELS["7b_target"], MODELS["7b_draft"],
                         batch=32, prompt_len=0, gamma=4, new_tokens=128,
                         prompt_range=(128, 2048)),
    "13b": Workload("13b", MODELS["13b_target"], MODELS["13b_draft"],
                    batch=64, prompt_len=512, gamma=4, new_tokens=128, greedy=True, alpha_forced=0.8),
}

# --------------------------------------------------------------------------
# weights


def weight_names(shape: ModelShape) -> List[str]:
    names = ["embed", "lm_head", "final_norm"]
    for l in range(shape.n_layers):
        names += [f"l{l}.{n}" for n in ("attn_norm", "wq", "wk", "wv", "wo",
                                        "ffn_norm", "w_gate", "w_up", "w_down")]
    return names


def weight_shapes(shape: ModelShape) -> Dict[str, tuple]:
    """Weight shapes in the [out_features, in_features] convention (y = x W^T)."""
    d, f, hd, V = shape.d_model, shape.d_ffn, shape.head_dim, shape.vocab
    H, KV = shape.n_heads, shape.n_kv_heads
    out = {"embed": (V, d), "lm_head": (V, d), "final_norm": (d,)}
    for l in range(shape.n_layers):
        out.update({
            f"l{l}.attn_norm": (d,), f"l{l}.wq": (H * hd, d),
            f"l{l}.wk": (KV * hd, d), f"l{l}.wv": (KV * hd, d),
            f"l{l}.wo": (d, H * hd), f"l{l}.ffn_norm": (d,),
            f"l{l}.w_gate": (f, d), f"l{l}.w_up": (f, d),
            f"l{l}.w_down": (d, f),
        })
    return out


def _tensor_rng(seed: int, name: str) -> np.random.Generator:
    return np.random.default_rng([int(seed), zlib.crc32(name.encode())])


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


_CHUNK = 1 << 20


def gen_tensor_chunks(seed: int, name: str, n: int, dtype: str,
                      chunk: int = _CHUNK) -> Iterable[tuple]:
    """Yield (offset, values) chunks of one weight tensor, flattened.

    values are uint16 bf16 bits (dtype "bf16") or float32 (dtype "fp32").
    Chunking does not change the values: the PCG64 stream is consumed in
    order.  Norm gains (names ending in ``norm``) are 1 + 0.1 N(0,1); every
    other tensor is 0.02 N(0,1).
    """
    rng = _tensor_rng(seed, name)
    is_norm = name.endswith("norm")
    buf = np.empty(min(chunk, max(n, 1)), dtype=np.float32)
    off = 0
    while off < n:
        m = min(chunk, n - off)
        v = buf[:m]
        rng.standard_normal(out=v, dtype=np.float32)
        if is_norm:
            v *= np.float32(0.1)
            v += np.float32(1.0)
        else:
            v *= np.float32(0.02)
        yield off, (bf16_bits(v) if dtype == "bf16" else v.copy())
        off += m


def gen_tensor(seed: int, name: str, shape: tuple, dtype: str) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16 if dtype == "bf16" else np.float32)
    for off, v in gen_tensor_chunks(seed, name, n, dtype):
        out[off:off + len(v)] = v
    return out.reshape(shape)


def model_weights(shape: ModelShape, seed: int,
                  names: Optional[Sequence[str]] = None,
                  threads: Optional[int] = None) -> Dict[str, np.ndarray]:
    """All (or the named) weights of a model: uint16 bf16 bits or float32."""
    shapes = weight_shapes(shape)
    names = list(names) if names is not None else weight_names(shape)
    threads = threads or min(16, len(os.sched_getaffinity(0)))
    with ThreadPoolExecutor(max_workers=threads) as ex:
        arrs = list(ex.map(lambda n: gen_tensor(seed, n, shapes[n], shape.dtype), names))
    return dict(zip(names, arrs))


def perturbed_weights(w: Dict[str, np.ndarray], dtype: str, seed: int,
                      eps: float) -> Dict[str, np.ndarray]:
    """A draft that is the target plus eps-scaled N(0, 0.02^2) noise on every
    matrix (gains kept).  eps = 0 gives the target itself."""
    out = {}
    for name, a in w.items():
        if name.endswith("norm") or eps == 0.0:
            out[name] = a.copy()
            continue
        base = bf16_bits_to_f32(a) if dtype == "bf16" else a.astype(np.float32)
        noise = _tensor_rng(seed, "perturb." + name).standard_normal(a.shape, dtype=np.float32)
        v = base + np.float32(0.02 * eps) * noise
        out[name] = bf16_bits(v) if dtype == "bf16" else v.astype(np.float32)
    return out

# --------------------------------------------------------------------------
# prompts


def ragged_lengths(n: int, lo: int, hi: int, seed: int = 7) -> np.ndarray:
    """n prompt lengths, uniform integers in [lo, hi]."""
    return np.random.default_rng(seed).integers(lo, hi + 1, size=n)


def prompts(n: int, lengths, vocab: int, base_seed: int = 1000,
            first_task: int = 0) -> List[np.ndarray]:
    """Uniform-random token ids; task k uses seed base_seed + k."""
    if np.isscalar(lengths):
        lengths = [int(lengths)] * n
    return [np.random.default_rng(base_seed + first_task + k)
            .integers(0, vocab, size=int(lengths[k])).astype(np.int32)
            for k in range(n)]

# --------------------------------------------------------------------------
# uniforms (SplitMix64, counter-based)

_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def splitmix64(seed: int, counters: np.ndarray) -> np.ndarray:
    """Output number ``counters`` (0-based) of the SplitMix64 stream that
    starts from state ``seed``: z = seed + (c + 1) * golden, then the
    published xor-shift-multiply finaliser."""
    c = np.asarray(counters, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = np.uint64(seed & 0xFFFFFFFFFFFFFFFF) + (c + np.uint64(1)) * _GOLDEN
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        z = z ^ (z >> np.uint64(31))
    return z


def slot_layout(gamma: int) -> dict:
    """Slots of the per-(task, step) uniform vector: draft samples, acceptance
    tests, residual/bonus sample."""
    return {"draft": slice(0, gamma), "accept": slice(gamma, 2 * gamma),
            "resample": 2 * gamma, "n": 2 * gamma + 1}


def uniforms(seed: int, tasks: Sequence[int], step: int, n_slots: int) -> np.ndarray:
    """uint32 [len(tasks), n_slots]: the upper 32 bits of SplitMix64 output
    number ((task * 2^20 + step) * 2^12 + slot)."""
    t = np.asarray(tasks, dtype=np.uint64)[:, None]
    s = np.arange(n_slots, dtype=np.uint64)[None, :]
    ctr = ((t << np.uint64(20)) + np.uint64(step)) << np.uint64(12)
    ctr = ctr + s
    return (splitmix64(seed, ctr) >> np.uint64(32)).astype(np.uint32)


def uniform_table(seed: int, tasks: Sequence[int], n_steps: int, gamma: int) -> np.ndarray:
    """uint32 [n_steps, len(tasks), 2*gamma+1]."""
    n = 2 * gamma + 1
    return np.stack([uniforms(seed, tasks, st, n) for st in range(n_steps)])


class StreamingWeights:
    """Callable name -> array that generates a model's weights on a thread
    pool, at most `window` tensors ahead of the consumer, in the order of
    weight_names(shape).  Any order works; out-of-order names are generated
    on demand."""

    def __init__(self, shape: ModelShape, seed: int, workers: Optional[int] = None, window: int = 24):
        self.shape, self.seed = shape, seed
        self.shapes = weight_shapes(shape)
        self.order = weight_names(shape)
        self.window = window
        self.ex = ThreadPoolExecutor(max_workers=workers or min(16, len(os.sched_getaffinity(0))))
        self.fut: Dict[str, object] = {}
        self.next = 0
        self._fill()

    def _fill(self):
        while self.next < len(self.order) and len(self.fut) < self.window:
            n = self.order[self.next]
            self.fut[n] = self.ex.submit(gen_tensor, self.seed, n, self.shapes[n], self.shape.dtype)
            self.next += 1

    def __call__(self, name: str) -> np.ndarray:
        f = self.fut.pop(name, None)
        a = f.result() if f is not None else gen_tensor(self.seed, name, self.shapes[name], self.shape.dtype)
        self._fill()
        return a

    def close(self):
        self.ex.shutdown(wait=False, cancel_futures=True)
