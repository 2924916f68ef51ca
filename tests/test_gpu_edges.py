"""Edge cases of the HIP path on the tiny pair: a slot run past its KV
capacity, a bad slot id in a device batch, and a slot reused after release.
Every condition is handled on the device by a bounds check that flags it
(sd_check) and skips the access; none of these runs faults."""
import numpy as np
import pytest

import synth
from sdcase import say, make_engine, run_gpu_steps

pytestmark = pytest.mark.gpu

W = synth.WORKLOADS["tiny"]
ERR_KV_OVERFLOW, ERR_BAD_TOKEN = 1, 2


def _engine(greedy=True, max_slots=4, max_batch=2):
    tw, dw = synth.model_weights(W.target, 1), synth.model_weights(W.draft, 2)
    return make_engine(W.target, W.draft, tw, dw, max_slots=max_slots, max_batch=max_batch, gamma_max=4,
                       max_ctx=W.prompt_len + 200, greedy=greedy)


def test_kv_capacity_overflow_is_flagged_not_faulted():
    say("kv capacity overflow")
    eng = _engine()
    prompts = synth.prompts(2, W.prompt_len, W.target.vocab)
    # capacity: prompt + 8 new tokens + gamma_max, rounded up to 16 positions;
    # 30 steps emit at least 30 tokens, so the slots run past it
    _, acc, b, _ = run_gpu_steps(eng, [0, 1], prompts, 4, 30, 42, [0, 1], max_new=[8, 8])
    assert eng.check_flags() & ERR_KV_OVERFLOW
    assert eng.check_flags() == 0                      # reading clears the flags
    state = eng.slot_state(b).cpu().numpy()
    assert (state[:, 0] > state[:, 3]).all()           # committed length is past the capacity
    eng.close()


def test_bad_slot_id_is_flagged_and_the_other_task_is_unaffected():
    import torch
    say("bad slot id")
    prompts = synth.prompts(2, W.prompt_len, W.target.vocab)
    ref = _engine()
    tok_ref, _, _, _ = run_gpu_steps(ref, [0], prompts[:1], 4, 6, 42, [0])
    assert ref.check_flags() == 0
    ref.close()
    eng = _engine()
    from paper_2510_11331_amd import emitted_tokens
    from paper_2510_11331_amd.engine import uniforms_device
    eng.prefill([0, 1], prompts, [64, 64])
    b = eng.batch([0, 1], 4)
    b.slots[1] = 7                                     # no such slot (max_slots = 4)
    u = uniforms_device(synth.uniform_table(42, [0, 1], 6, 4))
    accs, outs = [], []
    for n in range(6):
        eng.step(b, u[n])
        accs.append(b.n_acc.clone())
        outs.append(b.out_tok.clone())
    torch.cuda.synchronize()
    assert eng.check_flags() & ERR_BAD_TOKEN
    tok = emitted_tokens(torch.stack(accs).cpu().numpy(), torch.stack(outs).cpu().numpy())
    assert tok[0] == tok_ref[0]                        # rows are computed independently
    eng.close()


def test_slot_reused_after_release_matches_a_fresh_engine():
    say("slot reuse")
    prompts = synth.prompts(3, W.prompt_len, W.target.vocab)
    eng = _engine(greedy=False)
    first, _, _, _ = run_gpu_steps(eng, [0], prompts[:1], 4, 8, 42, [0])
    eng.release(0)
    again, _, _, _ = run_gpu_steps(eng, [0], prompts[2:3], 4, 8, 43, [2])
    assert eng.check_flags() == 0
    eng.close()
    fresh_eng = _engine(greedy=False)
    fresh, _, _, _ = run_gpu_steps(fresh_eng, [0], prompts[2:3], 4, 8, 43, [2])
    fresh_eng.close()
    assert again[0] == fresh[0]
    assert first[0] != again[0]
