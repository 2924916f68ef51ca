"""ctypes binding of the serving scheduler (include/sd_sched.h): argument
marshalling only; the planning runs in libsd's native code.

A scheduler configuration is a dict:
  draft, target   (n_layers, d_model, d_ffn) of each model
  c_draft         (c1, c2) of the draft forward runtime T = c1 F b + c2 (s)
  c_verify        (c1, c2) of the verify forward runtime
  alpha           acceptance rate
  o_max           output tokens given to every task
  mem_budget      draft memory budget in bytes (optional, <= 0: none)
  prefill_separate  prompts processed before step 1 (optional, default False)
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, List, Sequence, Tuple

import numpy as np

from . import _lib


def _cfg(cfg: Dict) -> _lib.SchedCfg:
    c = _lib.SchedCfg()
    c.draft = _lib.SchedModel(*[int(v) for v in cfg["draft"]])
    c.target = _lib.SchedModel(*[int(v) for v in cfg["target"]])
    c.c1_draft, c.c2_draft = (float(v) for v in cfg["c_draft"])
    c.c1_verify, c.c2_verify = (float(v) for v in cfg["c_verify"])
    c.alpha = float(cfg["alpha"])
    c.o_max = int(cfg["o_max"])
    c.mem_budget = float(cfg.get("mem_budget", 0.0))
    c.prefill_separate = int(bool(cfg.get("prefill_separate", False)))
    return c


def _i32(a: Sequence[int]) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(a: np.ndarray, t):
    return a.ctypes.data_as(C.POINTER(t))


def _batches(batch_of: np.ndarray, n: int) -> List[List[int]]:
    out = [[] for _ in range(n)]
    for k, m in enumerate(batch_of):
        out[int(m)].append(k)
    return out


def latency(cfg: Dict, lengths: Sequence[int], batches: Sequence[Sequence[int]], l: int) -> float:
    """T_inf of a plan (sd_sched_latency); batches in pipeline order."""
    lens = _i32(lengths)
    bo = np.zeros(len(lens), dtype=np.int32)
    for m, b in enumerate(batches):
        bo[list(b)] = m
    t = C.c_double(0)
    _lib.check(_lib.lib().sd_sched_latency(C.byref(_cfg(cfg)), len(lens), _ptr(lens, C.c_int32), len(batches),
                                           _ptr(bo, C.c_int32), int(l), C.byref(t)), "sd_sched_latency")
    return float(t.value)


def batching(cfg: Dict, lengths: Sequence[int], l: int) -> Tuple[List[List[int]], float]:
    """Algorithm 1 for speculation length l (sd_sched_batching)."""
    lens = _i32(lengths)
    bo = np.zeros(len(lens), dtype=np.int32)
    nb, t = C.c_int(0), C.c_double(0)
    _lib.check(_lib.lib().sd_sched_batching(C.byref(_cfg(cfg)), len(lens), _ptr(lens, C.c_int32), int(l),
                                            _ptr(bo, C.c_int32), C.byref(nb), C.byref(t)), "sd_sched_batching")
    return _batches(bo, nb.value), float(t.value)


def plan(cfg: Dict, lengths: Sequence[int], l_max: int) -> Dict:
    """Batching and speculation length (sd_sched_plan)."""
    lens = _i32(lengths)
    bo = np.zeros(len(lens), dtype=np.int32)
    by_l = np.zeros(int(l_max), dtype=np.float64)
    nb, lb, t = C.c_int(0), C.c_int(0), C.c_double(0)
    _lib.check(_lib.lib().sd_sched_plan(C.byref(_cfg(cfg)), len(lens), _ptr(lens, C.c_int32), int(l_max),
                                        _ptr(bo, C.c_int32), C.byref(nb), C.byref(lb), C.byref(t),
                                        _ptr(by_l, C.c_double)), "sd_sched_plan")
    return {"l": lb.value, "batches": _batches(bo, nb.value), "t_inf": float(t.value),
            "t_inf_by_l": [float(v) for v in by_l]}


def uplink(lengths: Sequence[int], snr: Sequence[float], lam: float, bw: float) -> Tuple[List[float], float]:
    """Bandwidth shares and common upload time (sd_sched_uplink)."""
    lens = _i32(lengths)
    s = np.ascontiguousarray(np.asarray(snr, dtype=np.float64))
    w = np.zeros(len(lens), dtype=np.float64)
    t = C.c_double(0)
    _lib.check(_lib.lib().sd_sched_uplink(len(lens), _ptr(lens, C.c_int32), _ptr(s, C.c_double), float(lam),
                                          float(bw), _ptr(w, C.c_double), C.byref(t)), "sd_sched_uplink")
    return [float(v) for v in w], float(t.value)
