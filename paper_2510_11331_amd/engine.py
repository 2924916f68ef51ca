"""Host-side driver over libsd: device buffers (PyTorch allocations), weight
upload in libsd's layout, and the draft -> verify -> accept -> commit loop,
optionally pipelined over two HIP streams (Section II-B: drafting of one
batch overlaps verification of another).

PyTorch only provides device memory, streams and events here; all arithmetic
of the path runs in libsd's kernels.
"""
from __future__ import annotations

import ctypes as C
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np
import torch

from . import _lib
from ._lib import check, lib


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(s: Optional[torch.cuda.Stream]):
    return C.c_void_p(s.cuda_stream) if s is not None else C.c_void_p(torch.cuda.current_stream().cuda_stream)


def model_cfg(shape) -> _lib.ModelCfg:
    return _lib.ModelCfg(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                         shape.head_dim, shape.d_ffn, shape.vocab,
                         _lib.SD_DTYPE_BF16 if shape.dtype == "bf16" else _lib.SD_DTYPE_F32,
                         float(shape.rope_theta), float(shape.rms_eps))


def interleave_gate_up(gate: np.ndarray, up: np.ndarray) -> np.ndarray:
    """[F, d] gate and up -> [2F, d] with 16-row blocks alternating gate, up."""
    F, d = gate.shape
    return np.stack([gate.reshape(F // 16, 16, d), up.reshape(F // 16, 16, d)], axis=1).reshape(2 * F, d)


def rotary_pair_order(w: np.ndarray, head_dim: int) -> np.ndarray:
    """[heads * hd, d] query or key rows -> the same rows with each head in
    rotary pair order: for b < hd/16, rows 16b..16b+7 are dims 8b..8b+7 and
    rows 16b+8..16b+15 are dims hd/2+8b..hd/2+8b+7."""
    n, d = w.shape
    h = w.reshape(n // head_dim, 2, head_dim // 16, 8, d)       # [head, half, b, 8, d]
    return np.ascontiguousarray(h.transpose(0, 2, 1, 3, 4)).reshape(n, d)


class GPUModel:
    """Weights of one model on the device, in libsd's layout: fused QKV rows
    (query and key heads in rotary pair order), gate/up rows interleaved in
    16-row blocks, and the five projection
    matrices (QKV, O, gate/up, down, LM head) repacked on the device by
    sd_pack_linear into the MFMA-tile layout."""

    def __init__(self, shape, get: Callable[[str], np.ndarray], device="cuda"):
        self.shape = shape
        self.bf16 = shape.dtype == "bf16"
        self.device = device
        self.keep: List[torch.Tensor] = []
        up, pk = self._upload, self._packed
        self.embed = up(get("embed"))
        self.lm_head = pk(get("lm_head"))
        self.final_norm = up(get("final_norm"))
        L = shape.n_layers
        self.attn_norm, self.wqkv, self.wo, self.ffn_norm, self.wgu, self.wdown = ([] for _ in range(6))
        for l in range(L):
            p = f"l{l}."
            self.attn_norm.append(up(get(p + "attn_norm")))
            hd = shape.head_dim
            self.wqkv.append(pk(np.concatenate([rotary_pair_order(get(p + "wq"), hd),
                                                rotary_pair_order(get(p + "wk"), hd), get(p + "wv")], axis=0)))
            self.wo.append(pk(get(p + "wo")))
            self.ffn_norm.append(up(get(p + "ffn_norm")))
            self.wgu.append(pk(interleave_gate_up(get(p + "w_gate"), get(p + "w_up"))))
            self.wdown.append(pk(get(p + "w_down")))
        arr = lambda ts: (C.c_void_p * L)(*[t.data_ptr() for t in ts])
        self._arrays = [arr(self.attn_norm), arr(self.wqkv), arr(self.wo), arr(self.ffn_norm),
                        arr(self.wgu), arr(self.wdown)]
        a = self._arrays
        cast = lambda x: C.cast(x, C.POINTER(C.c_void_p))
        self.cstruct = _lib.Weights(self.embed.data_ptr(), self.lm_head.data_ptr(), self.final_norm.data_ptr(),
                                    cast(a[0]), cast(a[1]), cast(a[2]), cast(a[3]), cast(a[4]), cast(a[5]))

    def _to_device(self, a: np.ndarray) -> torch.Tensor:
        a = np.ascontiguousarray(a)
        if self.bf16:
            return torch.from_numpy(a.view(np.int16)).to(self.device).view(torch.bfloat16)
        return torch.from_numpy(a.astype(np.float32, copy=False)).to(self.device)

    def _upload(self, a: np.ndarray) -> torch.Tensor:
        t = self._to_device(a)
        self.keep.append(t)
        return t

    def _packed(self, a: np.ndarray) -> torch.Tensor:
        """[N, K] row-major on the host -> packed on the device."""
        N, K = a.shape
        src = self._to_device(a)
        dst = torch.empty_like(src)
        stream = torch.cuda.current_stream(src.device).cuda_stream
        _lib.check(_lib.lib().sd_pack_linear(src.data_ptr(), dst.data_ptr(), N, K,
                                             _lib.SD_DTYPE_BF16 if self.bf16 else _lib.SD_DTYPE_F32, stream),
                   "sd_pack_linear")
        torch.cuda.current_stream(src.device).synchronize()
        del src
        self.keep.append(dst)
        return dst


class Batch:
    """Device buffers of one batch of tasks for one speculation length."""

    def __init__(self, slots: Sequence[int], gamma: int, vocab: int, device="cuda"):
        B = len(slots)
        self.B, self.gamma, self.V = B, gamma, vocab
        self.slots_host = [int(s) for s in slots]
        self.slots = torch.tensor(self.slots_host, dtype=torch.int32, device=device)
        self.draft_tok = torch.zeros(B, gamma, dtype=torch.int32, device=device)
        self.q = torch.zeros(B, gamma, vocab, dtype=torch.float32, device=device)
        self.p = torch.zeros(B, gamma + 1, vocab, dtype=torch.float32, device=device)
        self.n_acc = torch.zeros(B, dtype=torch.int32, device=device)
        self.out_tok = torch.zeros(B, gamma + 1, dtype=torch.int32, device=device)
        # forced acceptance (greedy engines only): (cont [B, L] int32 device, alpha)
        self.force: Optional[tuple] = None

    def set_force(self, cont: Optional[np.ndarray], alpha: float = 0.0, device="cuda") -> None:
        """Draft token i of task b becomes cont[b, position] with probability
        alpha (sd_force_draft); cont [B, L] holds each task's reference
        continuation by absolute position.  None switches forcing off."""
        if cont is None:
            self.force = None
            return
        c = torch.from_numpy(np.ascontiguousarray(cont, dtype=np.int32)).to(device)
        assert c.shape[0] == self.B
        self.force = (c, float(alpha))


class SDEngine:
    def __init__(self, tshape, dshape, tget, dget, *, max_slots: int, max_batch: int, gamma_max: int,
                 max_ctx: int, kv_blocks_target: Optional[int] = None, kv_blocks_draft: Optional[int] = None,
                 prefill_rows: int = 1024, temperature: float = 1.0, greedy: bool = False,
                 device: str = "cuda", static_workspace: bool = False):
        """static_workspace: the context uses libsd's own per-device
        workspace (sd_init_static) instead of one allocated here."""
        L = lib()
        self.device = device
        self.tshape, self.dshape = tshape, dshape
        self.gamma_max = gamma_max
        self.vocab = tshape.vocab
        blocks = max_slots * ((max_ctx + 15) // 16)
        cfg = _lib.Config()
        cfg.target = model_cfg(tshape)
        cfg.draft = model_cfg(dshape)
        cfg.max_slots, cfg.max_batch, cfg.gamma_max, cfg.max_ctx = max_slots, max_batch, gamma_max, max_ctx
        cfg.kv_block = 16
        cfg.kv_blocks_target = kv_blocks_target or blocks
        cfg.kv_blocks_draft = kv_blocks_draft or blocks
        cfg.prefill_rows = prefill_rows
        cfg.temperature = float(temperature)
        cfg.greedy = int(bool(greedy))
        pt, pd = L.sd_kv_pool_bytes(C.byref(cfg), 0), L.sd_kv_pool_bytes(C.byref(cfg), 1)
        ws = L.sd_workspace_bytes(C.byref(cfg))
        if not (pt and pd and ws):
            raise _lib.SDError(_lib.SD_EINVAL, "configuration rejected")
        self.pool_t = torch.empty(pt, dtype=torch.uint8, device=device)
        self.pool_d = torch.empty(pd, dtype=torch.uint8, device=device)
        cfg.kv_pool_target = self.pool_t.data_ptr()
        cfg.kv_pool_draft = self.pool_d.data_ptr()
        if static_workspace:
            self.workspace = None
        else:
            self.workspace = torch.empty(ws, dtype=torch.uint8, device=device)
            cfg.workspace = self.workspace.data_ptr()
            cfg.workspace_bytes = ws
        self.cfg = cfg
        self.target = GPUModel(tshape, tget, device)
        self.draft = GPUModel(dshape, dget, device)
        h = C.c_void_p()
        init = L.sd_init_static if static_workspace else L.sd_init
        rc = init(C.byref(cfg), C.byref(self.target.cstruct), C.byref(self.draft.cstruct), C.byref(h))
        if rc != _lib.SD_OK and static_workspace:
            raise _lib.SDError(rc, "sd_init_static: " + L.sd_last_error().decode())
        check(rc, "sd_init")
        self.ctx = h
        self.L = L

    # ------------------------------------------------------------ lifecycle
    def prefill(self, slots: Sequence[int], prompts: Sequence[np.ndarray], max_new: Sequence[int],
                stream=None) -> None:
        B = len(slots)
        toks = np.concatenate([np.asarray(p, dtype=np.int32) for p in prompts])
        lens = np.array([len(p) for p in prompts], dtype=np.int32)
        mn = np.asarray(max_new, dtype=np.int32)
        sl = np.asarray(slots, dtype=np.int32)
        I32 = C.POINTER(C.c_int32)
        check(self.L.sd_prefill(self.ctx, B, sl.ctypes.data_as(I32), toks.ctypes.data_as(I32),
                                lens.ctypes.data_as(I32), mn.ctypes.data_as(I32), _stream(stream)), "sd_prefill")

    def release(self, slot: int) -> None:
        check(self.L.sd_release(self.ctx, int(slot)), "sd_release")

    def close(self) -> None:
        if getattr(self, "ctx", None):
            self.L.sd_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ------------------------------------------------------------ step pieces
    def batch(self, slots: Sequence[int], gamma: int) -> Batch:
        return Batch(slots, gamma, self.vocab, self.device)

    def draft_step(self, b: Batch, i: int, u: torch.Tensor, stream=None) -> None:
        """Draft call i of the step; with b.force set, followed by the forced
        acceptance of draft token i (sd_force_draft)."""
        check(self.L.sd_draft_step(self.ctx, b.B, _ptr(b.slots), b.gamma, i, _ptr(u), _ptr(b.draft_tok),
                                   _ptr(b.q), _stream(stream)), "sd_draft_step")
        if b.force is not None:
            cont, alpha = b.force
            check(self.L.sd_force_draft(self.ctx, b.B, _ptr(b.slots), b.gamma, i, _ptr(cont), int(cont.shape[1]),
                                        _ptr(u), alpha, _ptr(b.draft_tok), _stream(stream)), "sd_force_draft")

    def verify(self, b: Batch, logits: Optional[torch.Tensor] = None, stream=None) -> None:
        check(self.L.sd_verify(self.ctx, b.B, _ptr(b.slots), b.gamma, _ptr(b.draft_tok), _ptr(b.p),
                               _ptr(logits), _stream(stream)), "sd_verify")

    def accept(self, b: Batch, u: torch.Tensor, stream=None) -> None:
        accept_resample(b.B, b.gamma, self.vocab, bool(self.cfg.greedy), b.draft_tok, b.q, b.p, u,
                        b.n_acc, b.out_tok, stream)

    def commit(self, b: Batch, stream=None) -> None:
        check(self.L.sd_kv_commit(self.ctx, b.B, _ptr(b.slots), b.gamma, _ptr(b.n_acc), _ptr(b.out_tok),
                                  _stream(stream)), "sd_kv_commit")

    def step(self, b: Batch, u: torch.Tensor, stream=None, logits: Optional[torch.Tensor] = None) -> None:
        """One SD step of a batch: gamma draft calls, verify, accept, commit."""
        for i in range(b.gamma):
            self.draft_step(b, i, u, stream)
        self.verify(b, logits, stream)
        self.accept(b, u, stream)
        self.commit(b, stream)

    def slot_state(self, b: Batch, stream=None) -> torch.Tensor:
        out = torch.empty(b.B, 4, dtype=torch.int32, device=self.device)
        check(self.L.sd_slot_state(self.ctx, b.B, _ptr(b.slots), _ptr(out), _stream(stream)), "sd_slot_state")
        return out

    def check_flags(self, stream=None) -> int:
        f = C.c_int32(0)
        check(self.L.sd_check(self.ctx, _stream(stream), C.byref(f)), "sd_check")
        return int(f.value)

    def profile(self, enable: bool) -> None:
        check(self.L.sd_profile(self.ctx, int(enable)), "sd_profile")

    def profile_read(self, kind: int):
        n, ms, by = C.c_int64(0), C.c_double(0), C.c_double(0)
        check(self.L.sd_profile_read(self.ctx, kind, C.byref(n), C.byref(ms), C.byref(by)), "sd_profile_read")
        return int(n.value), float(ms.value), float(by.value)


class StepGraph:
    """One SD step of a batch (gamma draft calls, verify, accept, commit)
    captured as a HIP graph.  Every launch reads per-step data from device
    memory (slot state, uniforms), so one capture replays every step: before
    each replay the step's uniforms are copied into the captured buffer.
    Capturing records launches only; it does not advance any state."""

    def __init__(self, engine: "SDEngine", b: Batch):
        self.engine, self.b = engine, b
        self.u = torch.zeros(b.B, 2 * b.gamma + 1, dtype=torch.int32, device=engine.device)
        self.g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.g):
            engine.step(b, self.u)

    def run(self, u_step: torch.Tensor) -> None:
        self.u.copy_(u_step)
        self.g.replay()


def accept_resample(B, gamma, vocab, greedy, draft_tok, q, p, u, n_acc, out_tok, stream=None) -> None:
    """Context-free acceptance / resampling kernel (sd_accept_resample)."""
    check(lib().sd_accept_resample(B, gamma, vocab, int(bool(greedy)), _ptr(draft_tok), _ptr(q), _ptr(p),
                                   _ptr(u), _ptr(n_acc), _ptr(out_tok), _stream(stream)), "sd_accept_resample")


def uniforms_device(table: np.ndarray, device="cuda") -> torch.Tensor:
    """uint32 uniforms -> a device int32 tensor with the same bits."""
    return torch.from_numpy(np.ascontiguousarray(table).view(np.int32)).to(device)


def generate_graph(engine: SDEngine, batch: Batch, utable: np.ndarray, n_steps: int,
                   graph: Optional[StepGraph] = None):
    """n_steps SD steps of one batch by graph replay on the current stream;
    returns (n_acc [n_steps, B], out_tok [n_steps, B, gamma+1]) on the host."""
    dev = engine.device
    u = uniforms_device(utable, dev)
    graph = graph or StepGraph(engine, batch)
    hist_acc = torch.empty(n_steps, batch.B, dtype=torch.int32, device=dev)
    hist_out = torch.empty(n_steps, batch.B, batch.gamma + 1, dtype=torch.int32, device=dev)
    for n in range(n_steps):
        graph.run(u[n])
        hist_acc[n].copy_(batch.n_acc)
        hist_out[n].copy_(batch.out_tok)
    torch.cuda.synchronize(dev)
    return hist_acc.cpu().numpy(), hist_out.cpu().numpy()


def generate(engine: SDEngine, batches: List[Batch], utables: List[np.ndarray], n_steps: int,
             two_streams: bool = True, logits_hook=None):
    """Run n_steps SD steps on every batch.  utables[m] is [n_steps, B_m,
    2 gamma + 1] uint32.  With two streams, drafting of batch m+1 overlaps
    verification of batch m; every dependency is an event, the host never
    waits inside the loop.  Returns per batch the stacked (n_acc, out_tok)
    of every step as host arrays."""
    dev = engine.device
    us = [uniforms_device(t, dev) for t in utables]
    M = len(batches)
    hist_acc = [torch.empty(n_steps, b.B, dtype=torch.int32, device=dev) for b in batches]
    hist_out = [torch.empty(n_steps, b.B, b.gamma + 1, dtype=torch.int32, device=dev) for b in batches]
    if two_streams:
        sD, sV = torch.cuda.Stream(device=dev), torch.cuda.Stream(device=dev)
    else:
        sD = sV = torch.cuda.current_stream(dev)
    cur = torch.cuda.current_stream(dev)
    sD.wait_stream(cur)
    sV.wait_stream(cur)
    evD = [torch.cuda.Event() for _ in range(M)]
    evV = [torch.cuda.Event() for _ in range(M)]
    for n in range(n_steps):
        for m, b in enumerate(batches):
            u = us[m][n]
            if n > 0 and two_streams:
                sD.wait_event(evV[m])
            for i in range(b.gamma):
                engine.draft_step(b, i, u, sD)
            if two_streams:
                evD[m].record(sD)
                sV.wait_event(evD[m])
            engine.verify(b, None, sV)
            if logits_hook is not None:
                logits_hook(m, n, b, sV)
            engine.accept(b, u, sV)
            engine.commit(b, sV)
            with torch.cuda.stream(sV):
                hist_acc[m][n].copy_(b.n_acc)
                hist_out[m][n].copy_(b.out_tok)
            if two_streams:
                evV[m].record(sV)
    cur.wait_stream(sV)
    cur.wait_stream(sD)
    torch.cuda.synchronize(dev)
    return [(a.cpu().numpy(), o.cpu().numpy()) for a, o in zip(hist_acc, hist_out)]


def emitted_tokens(n_acc: np.ndarray, out_tok: np.ndarray) -> List[List[int]]:
    """Per task, the tokens emitted over the recorded steps (accepted drafts
    then the bonus token of each step)."""
    S, B = n_acc.shape
    res = [[] for _ in range(B)]
    for s in range(S):
        for b in range(B):
            a = int(n_acc[s, b])
            res[b].extend(int(t) for t in out_tok[s, b, :a + 1])
    return res


def resume_prompts(prompts: Sequence[np.ndarray], emitted: Sequence[Sequence[int]]) -> List[np.ndarray]:
    """Checkpoint / resume.  After sd_kv_commit a task's whole state is its
    prompt, the tokens emitted so far, its step count and its uniform stream
    (uniforms are indexed by task and step).  Prefilling prompt + emitted
    into a slot re-creates the committed caches; the run then continues with
    the uniforms of the steps that follow."""
    return [np.concatenate([np.asarray(p, dtype=np.int32), np.asarray(e, dtype=np.int32)])
            for p, e in zip(prompts, emitted)]
