"""C ABI checks that need no GPU: libsd loads, exports every function
include/sd.h declares, sizes follow the documented layouts, and invalid
arguments are rejected on the host before anything is enqueued."""
import ctypes as C
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2510_11331_amd", "libsd.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libsd.so not built (run __graft_entry__.build())")


def header_functions():
    names = set()
    for h in ("sd.h", "sd_sched.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(sd_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_exports_every_declared_function():
    from paper_2510_11331_amd import _lib
    L = _lib.lib()
    names = header_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_lib.EXPORTS)


def make_cfg(tshape=None, dshape=None, **kw):
    from paper_2510_11331_amd import _lib
    from paper_2510_11331_amd.engine import model_cfg
    c = _lib.Config()
    c.target = model_cfg(tshape or synth.MODELS["tiny_target"])
    c.draft = model_cfg(dshape or synth.MODELS["tiny_draft"])
    c.max_slots, c.max_batch, c.gamma_max, c.max_ctx = 4, 2, 4, 128
    c.kv_block, c.kv_blocks_target, c.kv_blocks_draft = 16, 32, 32
    c.prefill_rows, c.temperature, c.greedy = 64, 1.0, 0
    for k, v in kw.items():
        setattr(c, k, v)
    return c


def test_sizes_and_validation():
    from paper_2510_11331_amd import _lib
    L = _lib.lib()
    c = make_cfg()
    t = synth.MODELS["tiny_target"]
    # pool: per layer [kv heads][blocks][K|V][16 tokens x head_dim] in the model dtype (fp32 here)
    assert L.sd_kv_pool_bytes(C.byref(c), 0) == t.n_layers * 32 * 2 * t.n_kv_heads * 16 * t.head_dim * 4
    assert L.sd_workspace_bytes(C.byref(c)) > 0
    bad = [dict(kv_block=8), dict(gamma_max=0), dict(gamma_max=17), dict(max_batch=5),
           dict(temperature=0.0), dict(prefill_rows=0), dict(max_ctx=1), dict(max_ctx=32769)]
    for kw in bad:
        cb = make_cfg(**kw)
        assert L.sd_workspace_bytes(C.byref(cb)) == 0, kw
        h = C.c_void_p()
        w = _lib.Weights()
        assert L.sd_init(C.byref(cb), C.byref(w), C.byref(w), C.byref(h)) == _lib.SD_EINVAL
    # shapes the kernels do not cover are refused: head_dim 96, vocab not a multiple of 16
    for shape in (synth.ModelShape(1, 192, 2, 2, 512, 1024, "fp32"),
                  synth.ModelShape(1, 128, 2, 2, 512, 1000, "fp32"),
                  synth.ModelShape(1, 128, 2, 2, 520, 1024, "bf16")):
        assert L.sd_workspace_bytes(C.byref(make_cfg(dshape=shape))) == 0
    # valid configuration but null weights / buffers: rejected before any HIP call
    h = C.c_void_p()
    w = _lib.Weights()
    assert L.sd_init(C.byref(c), C.byref(w), C.byref(w), C.byref(h)) == _lib.SD_EINVAL
    assert L.sd_init(None, None, None, C.byref(h)) == _lib.SD_EINVAL


def test_context_free_and_null_context_errors():
    from paper_2510_11331_amd import _lib
    L = _lib.lib()
    E = _lib.SD_EINVAL
    assert L.sd_accept_resample(0, 4, 16, 0, None, None, None, None, None, None, None) == E
    assert L.sd_accept_resample(1, 0, 16, 0, 1, 1, 1, 1, 1, 1, None) == E
    # rows are read as 16-byte vectors: a vocabulary that is not a multiple of
    # 4, or q / p rows that do not start on 16 bytes, are refused before any
    # launch (the pointers below are never dereferenced)
    A = 1 << 20
    for V in (1, 2, 3, 1001, 31999, 32002):
        assert L.sd_accept_resample(2, 4, V, 0, A, A, A, A, A, A, None) == E, V
    assert L.sd_accept_resample(2, 4, 1024, 0, A, A + 8, A, A, A, A, None) == E
    assert L.sd_accept_resample(2, 4, 1024, 0, A, A, A + 4, A, A, A, None) == E
    assert L.sd_accept_resample(2, 4, 32772, 0, A, A, A, A, A, A, None) == E
    assert L.sd_draft_step(None, 1, 1, 4, 0, 1, 1, 1, None) == E
    assert L.sd_verify(None, 1, 1, 4, 1, 1, None, None) == E
    assert L.sd_kv_commit(None, 1, 1, 4, 1, 1, None) == E
    assert L.sd_release(None, 0) == E
    assert L.sd_profile(None, 1) == E
    for code in (0, -1, -2, -3, -4):
        assert len(_lib.strerror(code)) >= 2 and _lib.strerror(code) != str(code)
