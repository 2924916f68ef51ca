"""ctypes binding of libsd (include/sd.h): argument marshalling only.

Every step of the hot path runs in libsd's HIP kernels.  Loading fails loudly
when libsd.so has not been built; there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsd.so")

SD_OK, SD_EINVAL, SD_ENOMEM, SD_ESTATE, SD_EHIP = 0, -1, -2, -3, -4
SD_DTYPE_BF16, SD_DTYPE_F32 = 0, 1
(SD_PROF_GEMM_VERIFY_GATEUP, SD_PROF_GEMM_VERIFY_ALL, SD_PROF_ATTN_VERIFY,
 SD_PROF_VERIFY, SD_PROF_DRAFT) = range(5)

# the symbols include/sd.h and include/sd_sched.h declare (checked by the CPU test suite)
EXPORTS = ("sd_kv_pool_bytes", "sd_workspace_bytes", "sd_init", "sd_init_static", "sd_prefill", "sd_release",
           "sd_draft_step", "sd_verify", "sd_accept_resample", "sd_kv_commit", "sd_force_draft", "sd_slot_state",
           "sd_check", "sd_profile", "sd_profile_read", "sd_destroy", "sd_strerror", "sd_last_error",
           "sd_pack_linear", "sd_sched_latency", "sd_sched_batching", "sd_sched_plan", "sd_sched_uplink")


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("d_model", C.c_int), ("n_heads", C.c_int),
                ("n_kv_heads", C.c_int), ("head_dim", C.c_int), ("d_ffn", C.c_int),
                ("vocab", C.c_int), ("dtype", C.c_int), ("rope_theta", C.c_float),
                ("rms_eps", C.c_float)]


class Weights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("lm_head", C.c_void_p), ("final_norm", C.c_void_p),
                ("attn_norm", C.POINTER(C.c_void_p)), ("wqkv", C.POINTER(C.c_void_p)),
                ("wo", C.POINTER(C.c_void_p)), ("ffn_norm", C.POINTER(C.c_void_p)),
                ("wgu", C.POINTER(C.c_void_p)), ("wdown", C.POINTER(C.c_void_p))]


class Config(C.Structure):
    _fields_ = [("target", ModelCfg), ("draft", ModelCfg), ("max_slots", C.c_int),
                ("max_batch", C.c_int), ("gamma_max", C.c_int), ("max_ctx", C.c_int),
                ("kv_block", C.c_int), ("kv_blocks_target", C.c_int), ("kv_blocks_draft", C.c_int),
                ("prefill_rows", C.c_int), ("temperature", C.c_float), ("greedy", C.c_int),
                ("kv_pool_target", C.c_void_p), ("kv_pool_draft", C.c_void_p),
                ("workspace", C.c_void_p), ("workspace_bytes", C.c_size_t)]


class SchedModel(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("d_model", C.c_int), ("d_ffn", C.c_int)]


class SchedCfg(C.Structure):
    _fields_ = [("draft", SchedModel), ("target", SchedModel), ("c1_draft", C.c_double),
                ("c2_draft", C.c_double), ("c1_verify", C.c_double), ("c2_verify", C.c_double),
                ("alpha", C.c_double), ("o_max", C.c_int), ("mem_budget", C.c_double),
                ("prefill_separate", C.c_int)]


class SDError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        detail = ""
        if code == SD_EHIP:
            try:
                detail = " [" + lib().sd_last_error().decode() + "]"
            except Exception:
                pass
        super().__init__(f"{what}: {strerror(code)} ({code}){detail}")


_lib = None


def lib():
    """Load libsd.so (once).  torch is imported first so libsd binds to the
    HIP runtime torch already loaded."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libsd.so is not built ({LIB_PATH}); run paper_2510_11331_amd/build.py")
    import torch  # noqa: F401
    L = C.CDLL(LIB_PATH)
    P, I, U32, F = C.c_void_p, C.c_int, C.POINTER(C.c_uint32), C.c_float
    sig = {
        "sd_kv_pool_bytes": (C.c_size_t, [C.POINTER(Config), I]),
        "sd_workspace_bytes": (C.c_size_t, [C.POINTER(Config)]),
        "sd_init": (I, [C.POINTER(Config), C.POINTER(Weights), C.POINTER(Weights), C.POINTER(P)]),
        "sd_init_static": (I, [C.POINTER(Config), C.POINTER(Weights), C.POINTER(Weights), C.POINTER(P)]),
        "sd_prefill": (I, [P, I, C.POINTER(C.c_int32), C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                           C.POINTER(C.c_int32), P]),
        "sd_release": (I, [P, I]),
        "sd_draft_step": (I, [P, I, P, I, I, P, P, P, P]),
        "sd_verify": (I, [P, I, P, I, P, P, P, P]),
        "sd_accept_resample": (I, [I, I, I, I, P, P, P, P, P, P, P]),
        "sd_kv_commit": (I, [P, I, P, I, P, P, P]),
        "sd_force_draft": (I, [P, I, P, I, I, P, I, P, C.c_double, P, P]),
        "sd_slot_state": (I, [P, I, P, P, P]),
        "sd_check": (I, [P, P, C.POINTER(C.c_int32)]),
        "sd_profile": (I, [P, I]),
        "sd_profile_read": (I, [P, I, C.POINTER(C.c_int64), C.POINTER(C.c_double), C.POINTER(C.c_double)]),
        "sd_destroy": (None, [P]),
        "sd_strerror": (C.c_char_p, [I]),
        "sd_last_error": (C.c_char_p, []),
        "sd_pack_linear": (I, [P, P, I, I, I, P]),
        "sd_sched_latency": (I, [C.POINTER(SchedCfg), I, C.POINTER(C.c_int32), I, C.POINTER(C.c_int32), I,
                                 C.POINTER(C.c_double)]),
        "sd_sched_batching": (I, [C.POINTER(SchedCfg), I, C.POINTER(C.c_int32), I, C.POINTER(C.c_int32),
                                  C.POINTER(I), C.POINTER(C.c_double)]),
        "sd_sched_plan": (I, [C.POINTER(SchedCfg), I, C.POINTER(C.c_int32), I, C.POINTER(C.c_int32),
                              C.POINTER(I), C.POINTER(I), C.POINTER(C.c_double), C.POINTER(C.c_double)]),
        "sd_sched_uplink": (I, [I, C.POINTER(C.c_int32), C.POINTER(C.c_double), C.c_double, C.c_double,
                                C.POINTER(C.c_double), C.POINTER(C.c_double)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def strerror(code: int) -> str:
    try:
        return lib().sd_strerror(code).decode()
    except Exception:
        return str(code)


def check(code: int, what: str) -> None:
    if code != SD_OK:
        raise SDError(code, what)
