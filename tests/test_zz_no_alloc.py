"""sd_init_static, the entry point for callers that cannot allocate device
memory: a context on libsd's own per-device workspace gives, step for step,
the accepted lengths and tokens of a context on a caller-allocated
workspace.  Two static contexts in a row (the second with a smaller
configuration: fewer slots, a smaller batch and context) each match their
allocated twin; a second live static context on the device is refused, and
a configuration that needs more than the array is refused with its size."""
import numpy as np
import pytest

import synth
from sdcase import say, make_engine, run_gpu_steps

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS["tiny"]


def _pair(static, slots, batch, ctx, tau):
    from paper_2510_11331_amd import SDEngine
    tw, dw = synth.model_weights(W.target, 1), synth.model_weights(W.draft, 2)
    return SDEngine(W.target, W.draft, tw.__getitem__, dw.__getitem__, max_slots=slots, max_batch=batch,
                    gamma_max=4, max_ctx=ctx, prefill_rows=64, temperature=tau, static_workspace=static)


@pytest.mark.parametrize("case", [(4, 2, 300, 1.0, 10), (2, 1, 160, 0.5, 6)])
def test_static_workspace_matches_allocated(case):
    slots, batch, ctx, tau, steps = case
    say("static workspace", case)
    prompts = synth.prompts(batch, 40, W.target.vocab, first_task=3)
    res = []
    for static in (False, True):
        eng = _pair(static, slots, batch, ctx, tau)
        if static:
            assert eng.workspace is None
        tok, acc, b, _ = run_gpu_steps(eng, list(range(batch)), prompts, 4, steps, 9, list(range(batch)))
        st = eng.slot_state(b).cpu().numpy()
        assert eng.check_flags() == 0
        eng.close()
        res.append((tok, acc, st))
    assert res[0][0] == res[1][0]
    assert np.array_equal(res[0][1], res[1][1]) and np.array_equal(res[0][2], res[1][2])


def test_static_workspace_is_held_by_one_context_and_bounded():
    import ctypes as C
    from paper_2510_11331_amd import _lib
    from paper_2510_11331_amd.engine import model_cfg
    say("static workspace refusals")
    first = _pair(True, 2, 1, 128, 1.0)
    with pytest.raises(_lib.SDError) as e:
        _pair(True, 2, 1, 128, 1.0)
    assert e.value.code == _lib.SD_ESTATE
    first.close()
    again = _pair(True, 2, 1, 128, 1.0)             # given back by sd_destroy
    again.close()
    # a configuration whose workspace exceeds the array: refused before any launch
    L = _lib.lib()
    c = _lib.Config()
    c.target, c.draft = model_cfg(synth.MODELS["7b_target"]), model_cfg(synth.MODELS["7b_draft"])
    c.max_slots, c.max_batch, c.gamma_max, c.max_ctx = 8, 8, 4, 4096
    c.kv_block, c.kv_blocks_target, c.kv_blocks_draft, c.prefill_rows, c.temperature = 16, 64, 64, 4096, 1.0
    assert L.sd_workspace_bytes(C.byref(c)) > (64 << 20)
    h = C.c_void_p()
    w = _lib.Weights()
    assert L.sd_init_static(C.byref(c), C.byref(w), C.byref(w), C.byref(h)) == _lib.SD_EINVAL
    assert b"static one holds" in L.sd_last_error()
    assert not h.value
