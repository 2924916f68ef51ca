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


def test_step_call_order_is_checked_on_the_host():
    """Out-of-order step calls are refused with SD_ESTATE before anything is
    enqueued; a restarted step (draft 0 again before the commit) discards
    the uncommitted work and gives the tokens of an uninterrupted step."""
    import torch
    from paper_2510_11331_amd import _lib
    from paper_2510_11331_amd.engine import uniforms_device
    say("call order")
    prompts = synth.prompts(2, W.prompt_len, W.target.vocab)
    ref = _engine(greedy=False)
    tok_ref, acc_ref, _, _ = run_gpu_steps(ref, [0, 1], prompts, 4, 2, 42, [0, 1])
    ref.close()
    eng = _engine(greedy=False)
    eng.prefill([0, 1], prompts, [64, 64])
    b = eng.batch([0, 1], 4)
    u = uniforms_device(synth.uniform_table(42, [0, 1], 2, 4))

    def refused(fn):
        with pytest.raises(_lib.SDError) as e:
            fn()
        assert e.value.code == _lib.SD_ESTATE

    refused(lambda: eng.verify(b))                     # no drafts yet
    refused(lambda: eng.commit(b))                     # nothing verified
    refused(lambda: eng.draft_step(b, 1, u[0]))        # draft 1 before draft 0
    eng.draft_step(b, 0, u[0])
    refused(lambda: eng.draft_step(b, 2, u[0]))        # skips draft 1
    refused(lambda: eng.verify(b))                     # 1 of 4 drafts
    for i in range(1, 4):
        eng.draft_step(b, i, u[0])
    eng.verify(b)
    eng.verify(b)                                      # a repeated verify rewrites the same positions
    refused(lambda: eng.draft_step(b, 3, u[0]))        # drafting after verify needs a new step
    # restart: the uncommitted step is discarded and run again in full
    for i in range(4):
        eng.draft_step(b, i, u[0])
    eng.verify(b)
    eng.accept(b, u[0])
    eng.commit(b)
    refused(lambda: eng.commit(b))                     # a second commit of the same step
    a0, o0 = b.n_acc.clone(), b.out_tok.clone()
    eng.step(b, u[1])
    torch.cuda.synchronize()
    from paper_2510_11331_amd import emitted_tokens
    tok = emitted_tokens(torch.stack([a0, b.n_acc]).cpu().numpy(), torch.stack([o0, b.out_tok]).cpu().numpy())
    assert tok == tok_ref
    assert eng.check_flags() == 0
    eng.close()


def test_released_slot_named_by_a_batch_writes_no_kv():
    """A batch that still names a released slot: the slot's capacity is 0 on
    the device, so its rows skip their KV writes (flagged) and the other
    task, now in blocks the released slot gave back, is unaffected."""
    import torch
    from paper_2510_11331_amd import emitted_tokens
    from paper_2510_11331_amd.engine import uniforms_device
    say("released slot in a batch")
    prompts = synth.prompts(3, W.prompt_len, W.target.vocab)
    ref = _engine()
    tok_ref, _, _, _ = run_gpu_steps(ref, [2], prompts[2:3], 4, 6, 42, [2])
    assert ref.check_flags() == 0
    ref.close()
    eng = _engine()
    eng.prefill([0, 1], prompts[:2], [32, 32])
    eng.release(1)
    eng.prefill([2], prompts[2:3], [32])               # may take the blocks slot 1 gave back
    b = eng.batch([2, 1], 4)
    u = uniforms_device(synth.uniform_table(42, [2, 1], 6, 4))
    accs, outs = [], []
    for n in range(6):
        eng.step(b, u[n])
        accs.append(b.n_acc.clone())
        outs.append(b.out_tok.clone())
    torch.cuda.synchronize()
    assert eng.check_flags() & ERR_KV_OVERFLOW
    tok = emitted_tokens(torch.stack(accs).cpu().numpy(), torch.stack(outs).cpu().numpy())
    assert tok[0] == tok_ref[0]
    eng.close()
