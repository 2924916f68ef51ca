#!/usr/bin/env python3
"""Benchmark of the speculative-decoding hot path on one MI355X.

Workload: LLaMA-7B-shaped bf16 target (32 layers, d 4096, 32 heads, FFN
11008, vocab 32000) with a 2-layer d-1024 draft, B = 8 tasks, gamma = 4,
prompts of 1024 uniform-random tokens, temperature 1.0, random-init weights.
A step is one full pass of the hot path for the batch: gamma draft forwards
with sampling, the verify forward over B*(gamma+1) rows, acceptance /
resampling, and the KV commit.

Prints one JSON line: verified tokens/s (emitted tokens of the timed steps /
wall time), verify-step latency (HIP events, p50/p90), the roofline of the
dominant kernel (the target's FFN gate/up GEMM), and the oracle timed on the
host cores on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
METRIC = "verified tokens/sec + verify-step latency, 7B-shape bf16 B=8 gamma=4; HBM GB/s"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="7b_b8", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--batch", type=int, default=0, help="override the workload's batch size")
    ap.add_argument("--gamma", type=int, default=0, help="override the workload's gamma")
    ap.add_argument("--alpha", type=float, default=None,
                    help="override the forced acceptance rate of a forced-acceptance workload (13B)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="short eager run for rocprofv3 --pmc: a 1 GiB copy kernel (counter calibration) "
                         "and two eager steps, no JSON line")
    ap.add_argument("--trace-summary", metavar="KERNEL_TRACE_CSV",
                    help="summarise a rocprofv3 --kernel-trace csv of a default bench run (whole run by kernel, "
                         "and the median timed step by kernel and launch shape) as markdown and exit")
    ap.add_argument("--fit-runtime", metavar="OUT_JSON",
                    help="fit the runtime model T(b, F) = c1 F b + c2 of the verify and draft forwards of the "
                         "7B-shape pair on this GPU (graph-replayed passes over batch sizes, contexts and "
                         "speculation lengths), write the fit to OUT_JSON and exit")
    ap.add_argument("--sweep-gamma", metavar="GAMMAS", default=None,
                    help="comma-separated speculation lengths: step time, verify / draft latency and tokens per "
                         "step of --workload at each (one JSON line per length), then exit")
    ap.add_argument("--oracle-timing", action="store_true",
                    help="the oracle's step time for every configuration on this host, all BLAS threads and one; "
                         "no GPU; then exit")
    ap.add_argument("--schedule", metavar="FIT_JSON",
                    help="with a runtime fit: plan batches and speculation length for synthetic task sets, "
                         "compare with the baseline policies (predicted), and run plans on the GPU (measured)")
    ap.add_argument("--counters-summary", metavar="COUNTER_CSV",
                    help="markdown per-kernel summary of a rocprofv3 --pmc counter_collection.csv, then exit")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="summarise two rocprofv3 --pmc counter_collection.csv files of --pmc-pass runs "
                         "(FETCH_SIZE, then WRITE_SIZE) into profiles/pmc_traffic.json and exit")
    return ap.parse_args()


TRAFFIC_JSON = os.path.join(ROOT, "profiles", "pmc_traffic.json")
GATEUP_NAME = "gemm_kernel<_Float16, 3, 6, 2, 2>"   # fp16 operands, MT=3, NT=6 (balanced), U=2, SwiGLU
COPY_NAME = "neg_kernel"                            # torch.neg over 1 GiB of int16
COPY_BYTES = 1 << 30


def kernel_sources_digest() -> str:
    """Digest of the sources of the dominant kernel: a counter summary is
    only valid for the code it was taken on."""
    import hashlib
    h = hashlib.sha256()
    for f in ("gemm.hip", "sd_internal.h"):
        h.update(open(os.path.join(ROOT, "paper_2510_11331_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def traffic_from_profiles():
    """HBM bytes per launch of the gate/up GEMM from the committed rocprofv3
    counter summary (FETCH_SIZE + WRITE_SIZE, each scaled by the copy
    kernel's reading), or None if there is none for the current sources."""
    try:
        d = json.load(open(TRAFFIC_JSON))
        if d.get("sources_digest") != kernel_sources_digest():
            return None
        return float(d["gateup"]["bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def summarise_counters(fetch_csv: str, write_csv: str) -> None:
    import csv

    def per_kernel(path, counter):
        vals = {}
        with open(path) as f:
            for row in csv.DictReader(f):
                if row.get("Counter_Name") != counter:
                    continue
                name = short_kernel_name(row["Kernel_Name"])
                key = "copy" if COPY_NAME in name else "gateup" if GATEUP_NAME in name else None
                if key:
                    vals.setdefault(key, []).append(float(row["Counter_Value"]))
        return vals

    fe, wr = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")
    kib = COPY_BYTES / 1024
    f_scale = kib / float(np.median(fe["copy"]))
    w_scale = kib / float(np.median(wr["copy"]))
    fetch = float(np.median(fe["gateup"])) * f_scale * 1024
    write = float(np.median(wr["gateup"])) * w_scale * 1024
    out = {"kernel": GATEUP_NAME + " (target FFN gate/up, M=40, N=22016, K=4096)",
           "sources_digest": kernel_sources_digest(),
           "copy_kernel": {"bytes_read": COPY_BYTES, "bytes_written": COPY_BYTES,
                           "fetch_kib": float(np.median(fe["copy"])), "write_kib": float(np.median(wr["copy"])),
                           "fetch_scale": f_scale, "write_scale": w_scale},
           "gateup": {"launches": len(fe["gateup"]), "fetch_kib_raw": float(np.median(fe["gateup"])),
                      "write_kib_raw": float(np.median(wr["gateup"])),
                      "fetch_bytes": fetch, "write_bytes": write, "bytes_per_launch": fetch + write}}
    with open(TRAFFIC_JSON, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out, indent=1))


def _blas_threads() -> int:
    from threadpoolctl import threadpool_info
    return int(max([i.get("num_threads", 1) for i in threadpool_info()] or [1]))


def cpu_baseline(wl, B, gamma, emitted_per_step, budget_s=10.0, max_tasks=None):
    """The oracle (float64 NumPy, as it stands) on the host cores, on a
    bounded sample of the workload: the verify pass (forward_rows over
    gamma+1 rows with the workload's cached positions, LM head included) of
    every task (or of max_tasks of them, scaled to B) through a 1-layer and a
    2-layer cut of the target, which separates the per-layer cost from the
    head cost, and gamma draft forwards per task on the full draft.  Scaled to
    a full step: head + n_layers * layer + drafts."""
    from oracle import model as om
    t, d = wl.target, wl.draft
    ctx = wl.prompt_len or int(np.mean(wl.prompt_range))
    Bs = min(B, max_tasks or B)                       # tasks timed; the step time is scaled by B / Bs
    two = t.replace(n_layers=2)
    w = synth.model_weights(two, 1)
    m2 = om.Model(two, w)
    m1 = om.Model.__new__(om.Model)                   # same float64 weights, first layer only
    m1.s, m1.w, m1.ops, m1.bf16 = t.replace(n_layers=1), m2.w, m2.ops, m2.bf16
    md = om.Model(d, synth.model_weights(d, 2))
    rng = np.random.default_rng(0)

    def cache(m, seed):
        r = np.random.default_rng(seed)
        c = m.new_cache()
        for l in range(m.s.n_layers):
            c.K[l] = m.r(r.standard_normal((ctx, m.s.n_kv_heads, m.s.head_dim)))
            c.V[l] = m.r(r.standard_normal((ctx, m.s.n_kv_heads, m.s.head_dim)))
        return c

    def timed_verify(m):
        tot = 0.0
        for b in range(Bs):
            c = cache(m, b)
            rows = rng.integers(0, t.vocab, gamma + 1)
            t0 = time.perf_counter()
            m.forward_rows(c, rows)
            tot += time.perf_counter() - t0
        return tot

    # repeat the sample until about 10 s of oracle time has been measured
    reps, t1, t2, td, spent = 0, 0.0, 0.0, 0.0, 0.0
    while reps == 0 or (spent < budget_s and reps < 8):
        a, b2 = timed_verify(m1), timed_verify(m2)
        dd = 0.0
        for b in range(Bs):
            c = cache(md, 100 + b)
            for i in range(gamma):
                t0 = time.perf_counter()
                md.decode_row(c, int(rng.integers(0, d.vocab)), len(c))
                dd += time.perf_counter() - t0
        t1, t2, td, reps = t1 + a, t2 + b2, td + dd, reps + 1
        spent += a + b2 + dd
    t1, t2, td = t1 / reps * B / Bs, t2 / reps * B / Bs, td / reps * B / Bs
    layer = max(t2 - t1, 0.0)
    head = max(t1 - layer, 0.0)
    t_step = head + t.n_layers * layer + td
    cores = _blas_threads()
    return {"value": emitted_per_step * B / t_step, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"float64 NumPy oracle, {Bs} of {B} tasks: verify of {gamma + 1} rows with {ctx} cached "
                       f"positions through 1- and 2-layer cuts of the {t.n_layers}-layer target (LM head "
                       f"included) and {gamma} draft forwards per task; scaled to a full step = "
                       f"{t_step:.2f} s ({spent:.1f} s sampled over {reps} repetitions)"),
            "step_seconds": round(t_step, 4)}


def _unmangle_sd(n: str) -> str:
    """Readable form of a mangled libsd kernel name that the profiler left
    mangled (it does not know fp16 template arguments): _ZN2sd<len><name>I
    <args>E...  with args _Float16 (DF16_), float (f), unsigned short (t),
    ints (Li<n>E)."""
    import re
    m = re.match(r"_ZN2sd(\d+)", n)
    if not m:
        return n
    k = int(m.group(1))
    name = n[m.end():m.end() + k]
    rest = n[m.end() + k:]
    if not rest.startswith("I"):
        return "sd::" + name
    args, i = [], 1
    while i < len(rest) and rest[i] != "E":
        if rest.startswith("DF16_", i):
            args.append("_Float16"); i += 5
        elif rest[i] in "ft":
            args.append("float" if rest[i] == "f" else "unsigned short"); i += 1
        else:
            mm = re.match(r"Li(\d+)E", rest[i:])
            if not mm:
                return n
            args.append(mm.group(1)); i += mm.end()
    return f"sd::{name}<{', '.join(args)}>"


def short_kernel_name(n: str) -> str:
    """"void sd::gemm_kernel<...>(sd::GemmParams) [clone .kd]" -> "sd::gemm_kernel<...>"."""
    n = n.split(" [clone")[0].strip()
    if n.startswith("_Z"):
        return _unmangle_sd(n)
    if n.startswith("void "):
        n = n[5:]
    if n.endswith(")"):
        depth = 0
        for i in range(len(n) - 1, -1, -1):
            depth += n[i] == ")"
            depth -= n[i] == "("
            if depth == 0:
                n = n[:i]
                break
    return n


def counters_summary(path: str) -> None:
    """Markdown table of a rocprofv3 --pmc counter_collection.csv: per kernel
    and grid size, the dispatches, the median duration under counter
    collection, the median of every collected counter, and for the matrix
    FLOP counters (MfmaFlopsF16 / MfmaFlopsBF16) the achieved dense rate
    against MI355X's 2.5 PFLOP/s (fp16 and bf16 alike)."""
    import csv
    from collections import defaultdict
    vals, durs, counters = defaultdict(lambda: defaultdict(list)), defaultdict(dict), []
    with open(path) as f:
        for r in csv.DictReader(f):
            key = (short_kernel_name(r["Kernel_Name"]), int(r.get("Grid_Size", 0) or 0))
            c = r["Counter_Name"]
            if c not in counters:
                counters.append(c)
            vals[key][c].append(float(r["Counter_Value"]))
            durs[key][r["Dispatch_Id"]] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    flop = next((c for c in ("MfmaFlopsF16", "MfmaFlopsBF16") if c in counters), None)
    head = "| kernel (grid) | dispatches | median us | " + " | ".join(f"median {c}" for c in counters)
    if flop:
        head += " | MFMA TFLOP/s | of 2.5 PFLOP/s"
    print(head + " |")
    print("|---|---:|---:|" + "---:|" * len(counters) + ("---:|---:|" if flop else ""))
    for key in sorted(vals, key=lambda k: -sum(durs[k].values())):
        d = list(durs[key].values())
        us = float(np.median(d))
        row = f"| `{key[0]}` ({key[1]}) | {len(d)} | {us:.1f} | " + " | ".join(
            f"{float(np.median(vals[key][c])):.4g}" if vals[key][c] else "" for c in counters)
        if flop:
            fl = float(np.median(vals[key][flop])) if vals[key][flop] else 0.0
            tf = fl / (us * 1e-6) / 1e12 if us > 0 else 0.0
            row += f" | {tf:.0f} | {tf / 2500:.3f}"
        print(row + " |")


def trace_summary(path: str, warmup: int, steps: int) -> None:
    """Markdown summary of a rocprofv3 kernel trace of a default bench run.
    The timed steps are graph replays W .. W+K-1; a step runs from the first
    dispatch after the previous step's commit_kernel to its own
    commit_kernel (the prefill issues none)."""
    import csv
    from collections import defaultdict
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"],
                         int(r.get("Grid_Size_X", r.get("Grid_Size", 0)) or 0),
                         int(r.get("Workgroup_Size_X", r.get("Workgroup_Size", 0)) or 0),
                         int(r.get("Grid_Size_Y", 1) or 1)))
    rows.sort()

    short = short_kernel_name

    tot = defaultdict(list)
    for s, e, n, *_ in rows:
        tot[short(n)].append((e - s) / 1e3)
    all_us = sum(sum(v) for v in tot.values())
    print("## Whole run: every dispatch of the command\n")
    print("| kernel | calls | total ms | avg us | min us | max us | % |\n|---|---:|---:|---:|---:|---:|---:|")
    for n, v in sorted(tot.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{n[:90]}` | {len(v)} | {sum(v) / 1e3:.2f} | {np.mean(v):.2f} | {min(v):.2f} | {max(v):.2f} "
              f"| {100 * sum(v) / all_us:.1f} |")
    ends = [i for i, r in enumerate(rows) if "commit_kernel" in r[2]]
    spans = []
    for k in range(warmup, warmup + steps):
        if k < 1 or k >= len(ends):
            continue
        spans.append((ends[k - 1] + 1, ends[k]))
    if not spans:
        return
    dur = [rows[b][1] - rows[a][0] for a, b in spans]
    med = spans[int(np.argsort(dur)[len(dur) // 2])]
    a, b = med
    step = defaultdict(list)
    for s, e, n, gx, wg, gy in rows[a:b + 1]:
        step[f"{short(n)[:80]}  grid {gx}x{gy}, wg {wg}"].append((e - s) / 1e3)
    print(f"\n## One timed step (graph replay; median span of {len(spans)} timed steps): "
          f"{(rows[b][1] - rows[a][0]) / 1e3:.1f} us, {b - a + 1} dispatches, "
          f"kernel busy {sum(sum(v) for v in step.values()):.1f} us\n")
    print("| kernel (launch shape) | calls/step | total us | avg us | median us |\n|---|---:|---:|---:|---:|")
    for n, v in sorted(step.items(), key=lambda kv: -sum(kv[1])):
        print(f"| `{n}` | {len(v)} | {sum(v):.1f} | {np.mean(v):.2f} | {np.median(v):.2f} |")


def paper_flops_verify(J, h1, h2, kv, l):
    """Per-task FLOPs of a verify forward of 1 + l tokens over kv cached
    tokens (the decoding-stage form of eq. flops_v)."""
    return 4.0 * J * h1 * (1.0 + l) * (2.0 * h1 + kv + l + 1.0 + h2)


def paper_flops_draft(J, h1, h2, kv):
    """Per-task FLOPs of one draft decode forward over kv cached tokens (eq. flops_d, decoding stage)."""
    return 4.0 * J * h1 * (2.0 * h1 + kv + 1.0 + h2)


def linear_fit(x, y):
    """Least squares y = c1 x + c2; returns c1, c2, R^2, max relative residual."""
    x, y = np.asarray(x, dtype=np.float64), np.asarray(y, dtype=np.float64)
    A = np.stack([x, np.ones_like(x)], axis=1)
    (c1, c2), *_ = np.linalg.lstsq(A, y, rcond=None)
    pred = c1 * x + c2
    r2 = 1.0 - float(np.sum((y - pred) ** 2) / np.sum((y - y.mean()) ** 2))
    return float(c1), float(c2), r2, float(np.max(np.abs(pred - y) / y))


def replay_ms(graph, n):
    import torch
    graph.replay()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    ev[0].record()
    for k in range(n):
        graph.replay()
        ev[k + 1].record()
    torch.cuda.synchronize()
    return float(np.median([ev[k].elapsed_time(ev[k + 1]) for k in range(n)]))


def gateup_kernel_name(M: int, N: int) -> str:
    """Kernel the library launches for a bf16 SwiGLU gate/up projection of M
    rows and N = 2 d_ffn columns (the tile choices of plan_gemm / plan_rows)."""
    if M > 64 and N >= 8192:
        best, pad = 6, 1 << 30
        if M <= 640:
            for c in (4, 5, 6):
                rows = -(-M // (32 * c)) * 32 * c
                if rows <= pad:
                    best, pad = c, rows
        mtiles = -(-M // (32 * best))
        nf = 4 if N % 128 == 0 and mtiles * (N // 128) >= 128 else 2
        grid = mtiles * N // (32 * nf)
        waves = 8 if grid <= 256 and best != 8 else 4      # one workgroup per CU: 8 waves
        spare = 1 if waves == 8 and (best % 2 or nf % 2) else 0
        nb = (4 if 159 // (4 * best + 4 * nf + spare) >= 4 else 3) if grid <= 256 else 2   # LDS stages
        return f"gemm_rows_kernel<{best}, {nf}, 2, {nb}, {waves}>"
    if M > 64:
        return "gemm_kernel<_Float16, 4, 2, 2, 2>"
    mt = -(-M // 16)
    units = N // 32
    most = -(-units // 256) * 2
    if mt == 3 and units >= 256 and most <= 6:
        return f"gemm_kernel<_Float16, 3, {4 if most <= 4 else 6}, 2, 2> (balanced, 256 workgroups)"
    return f"gemm_kernel<_Float16, {mt}, {4 if mt == 3 and units < 512 else 2}, 2, 2>"


def fit_runtime(out_json: str) -> None:
    """Runtime model of the paper's serving scheduler refit on this GPU: the
    verify pass of the 7B-shape target and one decode forward of its draft,
    each captured as a HIP graph and replayed, over batch sizes b, cached
    contexts and speculation lengths l; F from the paper's FLOPs formulas."""
    import torch
    from paper_2510_11331_amd import SDEngine
    from paper_2510_11331_amd.engine import uniforms_device

    wl = synth.WORKLOADS["7b_b8"]
    t, d = wl.target, wl.draft
    ctxs, bs, ls = [256, 1024, 2048], [1, 4, 8, 16, 32], [1, 2, 4, 8]
    tg, dg = synth.StreamingWeights(t, 1), synth.StreamingWeights(d, 2)
    eng = SDEngine(t, d, tg, dg, max_slots=32, max_batch=32, gamma_max=8, max_ctx=max(ctxs) + 64,
                   prefill_rows=2048, temperature=1.0)
    tg.close(); dg.close()
    rows = []
    for ctx in ctxs:
        prompts = synth.prompts(32, [ctx] * 32, t.vocab)
        eng.prefill(list(range(32)), prompts, [32] * 32)
        for b in bs:
            u = uniforms_device(synth.uniform_table(42, list(range(b)), 1, 8)[0])
            bd = eng.batch(list(range(b)), 2)
            eng.draft_step(bd, 0, u)                 # the timed call is draft call 1 of a step
            gd = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gd):
                eng.draft_step(bd, 1, u)
            td = replay_ms(gd, 10)
            del gd
            for l in ls:
                bv = eng.batch(list(range(b)), l)
                for i in range(l):                   # verification follows the step's l draft calls
                    eng.draft_step(bv, i, u)
                gv = torch.cuda.CUDAGraph()
                with torch.cuda.graph(gv):
                    eng.verify(bv)
                tv = replay_ms(gv, 10)
                del gv
                rows.append({"ctx": ctx, "b": b, "l": l, "verify_ms": tv, "draft_ms": td})
                print(f"[fit] ctx {ctx} b {b} l {l}: verify {tv:.3f} ms, draft forward {td:.3f} ms",
                      file=sys.stderr, flush=True)
        for s in range(32):
            eng.release(s)
    eng.close()
    # P = ctx - 1 positions are cached after the prefill of prompt[:-1]
    xv = [paper_flops_verify(t.n_layers, t.d_model, t.d_ffn, r["ctx"] - 1, r["l"]) * r["b"] for r in rows]
    yv = [r["verify_ms"] * 1e-3 for r in rows]
    dr = [r for r in rows if r["l"] == 1]
    xd = [paper_flops_draft(d.n_layers, d.d_model, d.d_ffn, r["ctx"]) * r["b"] for r in dr]
    yd = [r["draft_ms"] * 1e-3 for r in dr]
    c1v, c2v, r2v, ev = linear_fit(xv, yv)
    c1d, c2d, r2d, ed = linear_fit(xd, yd)
    out = {"what": "T(b, F) = c1 F b + c2 (seconds) refit on one MI355X: 7B-shape bf16 target verify pass, "
                   "2-layer d1024 draft decode forward; graph replay; F from the paper's FLOPs formulas",
           "target": [t.n_layers, t.d_model, t.d_ffn], "draft": [d.n_layers, d.d_model, d.d_ffn],
           "c_verify": [c1v, c2v], "c_draft": [c1d, c2d],
           "fit_quality": {"verify_r2": r2v, "verify_max_rel_residual": ev, "draft_r2": r2d,
                           "draft_max_rel_residual": ed},
           "paper_table2": {"c_verify": [2.08e-14, 1.28e-2], "c_draft": [4.11e-13, 0.56e-3],
                            "hardware": "RTX 4500 (verify), RTX 3080 (draft)"},
           "points": rows}
    with open(out_json, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps({k: out[k] for k in ("c_verify", "c_draft", "fit_quality")}), flush=True)


def schedule_eval(fit_json: str) -> None:
    """The paper's scheduler (libsd sd_sched_*) with the runtime model refit on
    this GPU.  Predicted: the Section IV task set (100 tasks, input lengths
    uniform in [1, 512], every task given 2048 output tokens, acceptance rate
    0.8, speculation length up to 10, 16 GB draft memory) under the proposed
    plan (Algorithm 1 + the best speculation length) and the baseline
    policies of the paper, with this GPU's coefficients and with the
    paper's.  Measured: a 16-task ragged set run by the two-stream pipeline
    for each plan; steps 2..N are timed and compared with the model's latency
    of the same steps.  The engine processes prompts before step 1, so plans
    are made with the decoding-stage first step (prefill_separate), and one
    plan with the paper's first-step prefill pricing for comparison."""
    import torch
    from paper_2510_11331_amd import SDEngine, sched, generate

    fit = json.load(open(fit_json))
    base = {"draft": fit["draft"], "target": fit["target"]}
    ours = dict(base, c_draft=fit["c_draft"], c_verify=fit["c_verify"])
    paper = dict(base, c_draft=fit["paper_table2"]["c_draft"], c_verify=fit["paper_table2"]["c_verify"])

    def chunks(order, size):
        return [order[i:i + size] for i in range(0, len(order), size)]

    def best_over_l(cfg, lengths, batches, l_max):
        ts = [sched.latency(cfg, lengths, batches, l) for l in range(1, l_max + 1)]
        return int(np.argmin(ts)) + 1, float(min(ts))

    def policies(cfg, lengths, l_max):
        order = sorted(range(len(lengths)), key=lambda k: (lengths[k], k))
        p = sched.plan(cfg, lengths, l_max)
        fsl_b, fsl_t = sched.batching(cfg, lengths, 7)
        res = {"proposed (Algorithm 1 + best l)": (p["l"], len(p["batches"]), p["t_inf"]),
               "fixed l = 7 (FSL), Algorithm 1 batching": (7, len(fsl_b), fsl_t)}
        for name, bt in (("no batching", chunks(order, 1)), ("static batches of 8", chunks(order, 8)),
                         ("one batch (max batching)", [order])):
            l, t = best_over_l(cfg, lengths, bt, l_max)
            res[name] = (l, len(bt), t)
        # the proposed plan without the pipeline: batches one after the other
        serial = sum(sched.latency(cfg, lengths, [b], p["l"]) for b in p["batches"])
        res["proposed plan, no pipeline"] = (p["l"], len(p["batches"]), serial)
        return res, p

    rng = np.random.default_rng(7)
    lengths = [int(x) for x in rng.integers(1, 513, 100)]
    out = {"fit": {k: fit[k] for k in ("c_verify", "c_draft", "fit_quality")}, "predicted": {}}
    for label, cfg in (("mi355x_fit", ours), ("paper_table2", paper)):
        c = dict(cfg, alpha=0.8, o_max=2048, mem_budget=16e9)
        res, _ = policies(c, lengths, 10)
        out["predicted"][label] = {k: {"l": v[0], "batches": v[1], "t_inf_s": round(v[2], 4)} for k, v in res.items()}
        print(f"[schedule] predicted, {label} coefficients:", file=sys.stderr)
        for k, v in res.items():
            print(f"   {k:44s} l={v[0]:2d} batches={v[1]:3d} T_inf={v[2]:9.3f} s", file=sys.stderr, flush=True)

    # measured: 16 ragged tasks, random-init 7B-shape pair (acceptance ~0.45 per draft)
    wl = synth.WORKLOADS["7b_b8"]
    t, d = wl.target, wl.draft
    K, alpha, o_max, l_max = 16, 0.45, 48, 8
    rng = np.random.default_rng(11)
    lens = [int(x) for x in rng.integers(64, 1025, K)]
    tg, dg = synth.StreamingWeights(t, 1), synth.StreamingWeights(d, 2)
    reserve = (o_max + 2) * (l_max + 1)           # tokens a task may emit over the steps of any plan
    eng = SDEngine(t, d, tg, dg, max_slots=K, max_batch=K, gamma_max=l_max, max_ctx=1024 + reserve + 64,
                   prefill_rows=2048, temperature=1.0)
    tg.close(); dg.close()
    prompts = synth.prompts(K, lens, t.vocab)
    # the engine processes the prompts before the first step, so every step it
    # runs is a decoding step: plans are made with prefill_separate, and also,
    # for comparison, with the paper's first-step (prefill) pricing
    c = dict(ours, alpha=alpha, o_max=o_max, prefill_separate=True)
    c_paper = dict(c, prefill_separate=False)
    p = sched.plan(c, lens, l_max)
    p_paper = sched.plan(c_paper, lens, l_max)
    order = sorted(range(K), key=lambda k: (lens[k], k))
    l1, _ = best_over_l(c, lens, [order], l_max)
    plans = {"proposed": (p["batches"], p["l"]),
             "proposed, step-1 prefill pricing": (p_paper["batches"], p_paper["l"]),
             "one batch": ([order], l1), "fixed l = 7": (sched.batching(c, lens, 7)[0], 7)}
    c1 = dict(c, o_max=1)
    measured = {}
    for name, (batches, l) in plans.items():
        L = (1 - alpha ** (l + 1)) / (1 - alpha)
        N = int(np.ceil(o_max / L))
        pred = sched.latency(c, lens, batches, l) - sched.latency(c1, lens, batches, l)
        serial = sum(sched.latency(c, lens, [b], l) - sched.latency(c1, lens, [b], l) for b in batches)
        eng.prefill(list(range(K)), prompts, [reserve] * K)
        bts = [eng.batch(list(b), l) for b in batches]
        uts = [synth.uniform_table(42, list(b), N, l) for b in batches]
        generate(eng, bts, [u[:1] for u in uts], 1, two_streams=True)          # warm-up step
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        generate(eng, bts, [u[1:] for u in uts], N - 1, two_streams=True)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3
        measured[name] = {"l": l, "batches": [len(b) for b in batches], "decode_steps": N - 1,
                          "measured_ms": round(ms, 2), "predicted_ms": round(pred * 1e3, 2),
                          "predicted_serial_ms": round(serial * 1e3, 2)}
        print(f"[schedule] measured {name}: l={l} batches={[len(b) for b in batches]} {N - 1} decode steps: "
              f"{ms:.1f} ms (model, two-stage pipeline {pred * 1e3:.1f} ms; serial {serial * 1e3:.1f} ms)",
              file=sys.stderr, flush=True)
        for s in range(K):
            eng.release(s)
    eng.close()
    out["measured"] = {"tasks": K, "input_lengths": lens, "alpha": alpha, "o_max": o_max, "plans": measured}
    print(json.dumps(out), flush=True)


def oracle_e2e(name: str) -> dict:
    """The oracle's speculative decoding of a whole workload, task after task
    (prefill with batched rows, then SD steps until new_tokens are emitted):
    verified tokens per second with and without the prefill."""
    from oracle import model as om, sd as osd
    wl = synth.WORKLOADS[name]
    target = om.Model(wl.target, synth.model_weights(wl.target, 1))
    draft = om.Model(wl.draft, synth.model_weights(wl.draft, 2))
    prompts = synth.prompts(wl.batch, wl.prompt_len, wl.target.vocab)
    ut = synth.uniform_table(7, list(range(wl.batch)), wl.new_tokens + 2, wl.gamma)
    t_pre = t_dec = 0.0
    tokens = steps = 0
    for k in range(wl.batch):
        t0 = time.perf_counter()
        task = osd.SDTask(target, draft, prompts[k], batch_rows=True)
        t1 = time.perf_counter()
        while len(task.emitted) < wl.new_tokens:
            task.step(wl.gamma, ut[task.n_steps, k], wl.temperature, wl.greedy, batch_rows=True)
        t2 = time.perf_counter()
        t_pre, t_dec = t_pre + t1 - t0, t_dec + t2 - t1
        tokens, steps = tokens + len(task.emitted), steps + task.n_steps
        print(f"[oracle e2e] {name} task {k}: {task.n_steps} steps, {len(task.emitted)} tokens, "
              f"prefill {t1 - t0:.2f} s, decode {t2 - t1:.2f} s", file=sys.stderr, flush=True)
    return {"tokens": tokens, "task_steps": steps, "prefill_s": round(t_pre, 3), "decode_s": round(t_dec, 3),
            "tokens_per_s_decode": round(tokens / t_dec, 3), "tokens_per_s_with_prefill": round(tokens / (t_pre + t_dec), 3)}


def oracle_timing() -> None:
    """The oracle's step time on this host for every configuration, with all
    BLAS threads and with one (cpu_baseline's sample; up to 8 tasks timed and
    scaled to the batch).  One JSON line per configuration."""
    from threadpoolctl import threadpool_limits
    for name in ("tiny", "small"):
        r = oracle_e2e(name)
        print(json.dumps({"workload": name, "end_to_end": r, "threads": _blas_threads(),
                          "host_cpus": len(os.sched_getaffinity(0))}), flush=True)
    for name in ("tiny", "small", "7b_b1", "7b_b8", "7b_paged", "13b"):
        wl = synth.WORKLOADS[name]
        emitted = 1.0                                  # tokens per task per step scale the rate; report seconds
        multi = cpu_baseline(wl, wl.batch, wl.gamma, emitted, budget_s=5.0, max_tasks=8)
        print(f"[oracle] {name}: {multi['step_seconds']} s per step on {multi['cores']} threads", file=sys.stderr,
              flush=True)
        with threadpool_limits(limits=1):
            single = cpu_baseline(wl, wl.batch, wl.gamma, emitted, budget_s=5.0, max_tasks=8)
        print(json.dumps({"workload": name, "batch": wl.batch, "gamma": wl.gamma,
                          "step_s_all_threads": multi["step_seconds"], "threads": multi["cores"],
                          "step_s_one_thread": single["step_seconds"],
                          "host_cpus": len(os.sched_getaffinity(0)), "sample": multi["sample"]}), flush=True)


def reference_continuation(eng, slots, prompts, gamma, max_new):
    """Greedy verification emits the target's greedy continuation whatever
    the drafts: max_new unforced steps of a batch of the given gamma (the
    timed run's launch configuration, hence its rounding) give each task's
    continuation, [prompt + max_new tokens] per task."""
    from paper_2510_11331_amd import generate_graph, emitted_tokens
    ref = eng.batch(slots, gamma)
    acc0, out0 = generate_graph(eng, ref, synth.uniform_table(7, slots, max_new, gamma), max_new)
    em = emitted_tokens(acc0, out0)
    assert min(len(e) for e in em) >= max_new
    return np.array([list(prompts[k]) + em[k][:max_new] for k in range(len(slots))], dtype=np.int32)


def gamma_sweep(args) -> None:
    """The speculation-length sweep of a workload (7B B = 1: verify latency
    against gamma; 13B: gamma 2 / 4 / 8): for each gamma a fresh prefill of
    the same tasks, W warmup and K timed graph replays of the whole step,
    then the verify pass and the gamma draft calls alone (graph replay, p50)."""
    import torch
    from paper_2510_11331_amd import SDEngine, StepGraph, generate_graph
    wl = workload_of(args)
    gammas = [int(x) for x in args.sweep_gamma.split(",")]
    B, K, W = args.batch or wl.batch, args.steps, args.warmup
    t, d = wl.target, wl.draft
    assert not wl.prompt_range, "one batch of fixed-length prompts"
    g_max = max(gammas)
    forced = wl.alpha_forced is not None
    max_new = (K + W + 2) * (g_max + 1)
    tg, dg = synth.StreamingWeights(t, 1), synth.StreamingWeights(d, 2)
    eng = SDEngine(t, d, tg, dg, max_slots=B, max_batch=B, gamma_max=g_max,
                   max_ctx=wl.prompt_len + 2 * max_new + g_max + 16, prefill_rows=2048,
                   temperature=wl.temperature, greedy=wl.greedy)
    tg.close(); dg.close()
    slots = list(range(B))
    prompts = synth.prompts(B, wl.prompt_len, t.vocab)
    for gamma in gammas:
        eng.prefill(slots, prompts, [2 * max_new] * B)
        if forced:
            # the reference runs at the same gamma: the projections' tiling,
            # and so their rounding, depends on the number of verified rows
            cont = reference_continuation(eng, slots, prompts, gamma, max_new)
            for s_ in slots:
                eng.release(s_)
            eng.prefill(slots, prompts, [2 * max_new] * B)
        batch = eng.batch(slots, gamma)
        if forced:
            batch.set_force(cont, wl.alpha_forced)
        ut = synth.uniform_table(42, slots, W + K, gamma)
        graph = StepGraph(eng, batch)
        generate_graph(eng, batch, ut[:W], W, graph)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        acc, _ = generate_graph(eng, batch, ut[W:W + K], K, graph)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        del graph
        verify_ms, draft_ms = graph_latencies(eng, batch, ut[W + K - 1], K)
        flags = eng.check_flags()
        emitted = float((acc + 1).mean())
        line = {"workload": wl.name, "batch": B, "gamma": gamma, "steps": K, "ms_per_step": round(elapsed / K * 1e3, 3),
                "tokens_per_s": round(float((acc + 1).sum()) / elapsed, 1),
                "verify_ms_p50": round(float(np.median(verify_ms)), 4),
                "draft_ms_per_call": round(float(np.median(draft_ms)) / gamma, 4),
                "mean_emitted_per_step": round(emitted, 4), "device_flags": flags}
        if forced and wl.alpha_forced < 1:
            a = wl.alpha_forced
            line["alpha_forced"] = a
            line["emitted_per_step_eq_ol"] = round((1 - a ** (gamma + 1)) / (1 - a), 4)
        print(json.dumps(line), flush=True)
        for s_ in slots:
            eng.release(s_)
    eng.close()


def workload_of(args):
    """The named workload, with the forced acceptance rate overridden by --alpha."""
    import dataclasses
    wl = synth.WORKLOADS[args.workload]
    if args.alpha is not None:
        assert wl.alpha_forced is not None, "--alpha applies to a forced-acceptance workload"
        wl = dataclasses.replace(wl, alpha_forced=float(args.alpha))
    return wl


def copy_ceiling_gbs(nbytes: int = 1 << 30, reps: int = 10) -> float:
    """HBM rate of a plain device-to-device copy of nbytes (torch's copy
    kernel), bytes read plus bytes written per second: the practical ceiling
    a streaming kernel is compared with, beside the 8 TB/s datasheet peak."""
    import torch
    src = torch.ones(nbytes // 2, dtype=torch.int16, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2.0 * nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    return gbs


def graph_latencies(eng, batch, u_step, n):
    """Median-ready lists of n replay times (ms) of the verify pass and of the
    gamma draft calls of one batch, each captured as a HIP graph."""
    import torch
    from paper_2510_11331_amd.engine import uniforms_device
    u = uniforms_device(u_step)
    gv, gd = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    # capture order follows the step (draft calls, then verify); capturing
    # records launches and advances no slot
    with torch.cuda.graph(gd):
        for i in range(batch.gamma):
            eng.draft_step(batch, i, u)
    with torch.cuda.graph(gv):
        eng.verify(batch)
    out = []
    for g in (gv, gd):
        g.replay()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
        ev[0].record()
        for k in range(n):
            g.replay()
            ev[k + 1].record()
        torch.cuda.synchronize()
        out.append(np.array([ev[k].elapsed_time(ev[k + 1]) for k in range(n)]))
    del gv, gd
    return out


def main():
    args = parse()
    if args.traffic_from:
        summarise_counters(*args.traffic_from)
        return
    if args.counters_summary:
        counters_summary(args.counters_summary)
        return
    if args.trace_summary:
        trace_summary(args.trace_summary, args.warmup, args.steps)
        return
    if args.fit_runtime:
        fit_runtime(args.fit_runtime)
        return
    if args.schedule:
        schedule_eval(args.schedule)
        return
    if args.sweep_gamma:
        gamma_sweep(args)
        return
    if args.oracle_timing:
        oracle_timing()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus}); "
              "the single-GPU figure is the per-GPU share of the task-sharded design.", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2510_11331_amd import SDEngine, StepGraph, generate, generate_graph, emitted_tokens
    from paper_2510_11331_amd import _lib

    wl = workload_of(args)
    B = args.batch or wl.batch
    gamma = args.gamma or wl.gamma
    K, W = args.steps, args.warmup
    t, d = wl.target, wl.draft
    headline = args.workload == "7b_b8" and B == wl.batch and gamma == wl.gamma
    # the ragged paged workload runs two batches pipelined on two streams
    n_batches = 2 if wl.prompt_range else 1
    n_tasks = n_batches * B
    if wl.prompt_range:
        lens = [int(x) for x in synth.ragged_lengths(n_tasks, *wl.prompt_range)]
        prompt_desc = f"prompts uniform in [{wl.prompt_range[0]}, {wl.prompt_range[1]}] (mean {np.mean(lens):.0f})"
    else:
        lens = [wl.prompt_len] * n_tasks
        prompt_desc = f"prompt {wl.prompt_len}"
    max_new = (2 * K + W + 2) * (gamma + 1)
    forced = wl.alpha_forced is not None
    # a forced-acceptance workload first generates its reference continuation
    # (the target's greedy output) with up to max_new unforced steps
    ctx_need = max(lens) + (2 if forced else 1) * max_new + gamma + 16
    print(f"[bench] workload {wl.name} B={B}x{n_batches} gamma={gamma} steps={K} warmup={W}", file=sys.stderr,
          flush=True)

    t0 = time.time()
    tg, dg = synth.StreamingWeights(t, 1), synth.StreamingWeights(d, 2)
    eng = SDEngine(t, d, tg, dg, max_slots=n_tasks, max_batch=B, gamma_max=gamma, max_ctx=ctx_need,
                   prefill_rows=2048, temperature=wl.temperature, greedy=wl.greedy)
    tg.close(); dg.close()
    print(f"[bench] weights on device in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    prompts = synth.prompts(n_tasks, lens, t.vocab)

    def prefill_tasks():
        # in groups of 16, each reported (slow under counter collection); the
        # same grouping every time, so that a re-prefill caches the same bits
        for c in range(0, n_tasks, 16):
            group = list(range(c, min(c + 16, n_tasks)))
            eng.prefill(group, [prompts[k] for k in group], [(2 if forced else 1) * max_new] * len(group))
            print(f"[bench] prefilled tasks {group[0]}..{group[-1]}", file=sys.stderr, flush=True)

    t0 = time.time()
    prefill_tasks()
    print(f"[bench] prefill {n_tasks} tasks, {sum(lens)} tokens in {time.time() - t0:.2f}s", file=sys.stderr,
          flush=True)

    batches = [eng.batch(list(range(m * B, (m + 1) * B)), gamma) for m in range(n_batches)]
    if forced and not args.pmc_pass:
        # greedy verification emits the target's greedy continuation whatever
        # the drafts, so one unforced run gives each task's continuation; the
        # timed run then starts over with drafts forced to it w.p. alpha
        # (a counter pass skips it: forcing changes no kernel's shape)
        assert n_batches == 1 and wl.greedy
        t0 = time.time()
        cont = reference_continuation(eng, list(range(B)), prompts, gamma, max_new)
        for s_ in range(n_tasks):
            eng.release(s_)
        prefill_tasks()
        batches[0].set_force(cont, wl.alpha_forced)
        print(f"[bench] reference continuation of {max_new} tokens per task in {time.time() - t0:.1f}s; "
              f"drafts forced with probability {wl.alpha_forced}", file=sys.stderr, flush=True)
    uts = [synth.uniform_table(42, list(range(m * B, (m + 1) * B)), W + 2 * K, gamma) for m in range(n_batches)]
    batch, ut = batches[0], uts[0]
    if args.pmc_pass:
        src = torch.ones(COPY_BYTES // 2, dtype=torch.int16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst
        generate(eng, [batch], [ut[:2]], 2, two_streams=False)
        torch.cuda.synchronize()
        print("[bench] pmc pass done", file=sys.stderr, flush=True)
        return
    if n_batches == 1:
        graph = StepGraph(eng, batch)                  # one HIP graph replays every step
        generate_graph(eng, batch, ut[:W], W, graph)   # warmup
        torch.cuda.synchronize()
        # timed region: K graph replays, no host synchronisation inside
        t0 = time.perf_counter()
        acc, out = generate_graph(eng, batch, ut[W:W + K], K, graph)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        emitted = int((acc + 1).sum())
    else:
        # drafting of batch m+1 overlaps verification of batch m (two streams, events only)
        generate(eng, batches, [u[:W] for u in uts], W, two_streams=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        res_b = generate(eng, batches, [u[W:W + K] for u in uts], K, two_streams=True)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
        acc = res_b[0][0]
        emitted = int(sum((a_ + 1).sum() for a_, _ in res_b))
        # the same tasks from the same state on one stream ("SD w/o pipeline",
        # Section IV-A): re-prefilled, the same W + K steps with the same
        # uniforms, so the same trajectory (the streams change no result)
        for s_ in range(n_tasks):
            eng.release(s_)
        prefill_tasks()
        generate(eng, batches, [u[:W] for u in uts], W, two_streams=False)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        res_1 = generate(eng, batches, [u[W:W + K] for u in uts], K, two_streams=False)
        torch.cuda.synchronize()
        elapsed_one = time.perf_counter() - t0
        same = all(np.array_equal(a0, a1) and np.array_equal(o0, o1) for (a0, o0), (a1, o1) in zip(res_b, res_1))
        print(f"[bench] one stream: {K} steps in {elapsed_one:.3f}s (tokens identical: {same})", file=sys.stderr,
              flush=True)
    value = emitted / elapsed
    print(f"[bench] timed {K} steps in {elapsed:.3f}s, {emitted} tokens", file=sys.stderr, flush=True)

    # verify-step and draft-call latency: the verify pass alone (and the gamma
    # draft calls alone) captured as HIP graphs and replayed back to back,
    # HIP events on the replay stream around every replay.  A replay repeats
    # the same work (same rows, same K/V written at the same uncommitted
    # positions), so every replay is one verify step of this batch.
    verify_ms, draft_ms = graph_latencies(eng, batch, ut[W + K - 1], K)

    # instrumented pass: dispatch-stamped HIP events around the GEMM and
    # attention kernels.  Each step is queued behind a GPU sleep longer than
    # its host enqueue time, so the events time kernels, not launch latency.
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record(); torch.cuda._sleep(1_000_000); s1.record(); torch.cuda.synchronize()
    cycles_per_ms = 1_000_000 / max(s0.elapsed_time(s1), 1e-3)
    eng.profile(True)
    for n in range(K):
        torch.cuda._sleep(int(cycles_per_ms * 40))
        generate(eng, [batch], [ut[W + K + n:W + K + n + 1]], 1, two_streams=False)
    n_gu, ms_gu, bytes_gu = eng.profile_read(_lib.SD_PROF_GEMM_VERIFY_GATEUP)
    n_all, ms_all, bytes_all = eng.profile_read(_lib.SD_PROF_GEMM_VERIFY_ALL)
    n_at, ms_at, _ = eng.profile_read(_lib.SD_PROF_ATTN_VERIFY)
    eng.profile(False)
    flags = eng.check_flags()
    gu_ms = ms_gu / max(n_gu, 1)
    gu_bytes = bytes_gu / max(n_gu, 1)
    achieved = gu_bytes / (gu_ms * 1e-3) / 1e9
    # algorithmic bytes of one verify step: every weight read once (of the
    # embedding table only the B (gamma+1) rows the pass looks up), the
    # cached K/V of every task once per layer, the new K/V, logits /
    # probabilities; the verify latency was taken on batch 0 after its W + K
    # steps, so its context is the prompt plus the tokens those steps committed
    P = float(np.mean(lens[:B])) + float((acc + 1).mean()) * (W + K)
    kv_bytes = t.n_layers * 2 * t.n_kv_heads * t.head_dim * 2 * B * P
    weight_bytes = 2 * (t.n_params() - t.vocab * t.d_model) + 2 * B * (gamma + 1) * t.d_model
    step_bytes = weight_bytes + kv_bytes + 2 * B * (gamma + 1) * t.vocab * 4
    verify_p50 = float(np.median(verify_ms))
    copy_gbs = copy_ceiling_gbs()

    M = B * (gamma + 1)
    gu_name = gateup_kernel_name(M, 2 * t.d_ffn)
    shape_desc = (f"{t.n_layers}-layer d{t.d_model} target ({t.n_heads}/{t.n_kv_heads} heads, FFN {t.d_ffn}) + "
                  f"{d.n_layers}-layer d{d.d_model} draft")
    res = {
        "metric": METRIC if headline else f"verified tokens/sec + verify-step latency, {wl.name} B={B} gamma={gamma}",
        "value": round(value, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(elapsed / K * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: random-init N(0,0.02^2) bf16 weights, uniform-random prompt ids, SplitMix64 uniforms",
        "config": {"workload": f"{shape_desc}, B={B}" + (f" x {n_batches} batches on two streams" if n_batches > 1
                                                            else "") + f", gamma={gamma}, {prompt_desc}, "
                               + (f"greedy verification, drafts forced to the target's greedy continuation "
                                  f"w.p. {wl.alpha_forced}" if forced else
                                  "greedy" if wl.greedy else f"tau={wl.temperature}"),
                   "batch": B, "batches": n_batches, "gamma": gamma, "prompt_len": float(np.mean(lens)),
                   "temperature": 0.0 if wl.greedy else wl.temperature},
        "verify_ms_p50": round(verify_p50, 3),
        "verify_ms_p90": round(float(np.percentile(verify_ms, 90)), 3),
        "verify_hbm_gbs": round(step_bytes / (verify_p50 * 1e-3) / 1e9, 1),
        "verify_hbm_frac": round(step_bytes / (verify_p50 * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "copy_ceiling_gbs": round(copy_gbs, 1),
        "verify_frac_of_copy": round(step_bytes / (verify_p50 * 1e-3) / 1e9 / copy_gbs, 4),
        "verify_gemm_gbs": round(bytes_all / max(ms_all, 1e-9) * 1e-6, 1),
        "verify_attn_ms_per_layer": round(ms_at / max(n_at, 1), 4),
        "draft_ms_per_call": round(float(np.median(draft_ms)) / gamma, 4),
        "mean_accepted": round(float(acc.mean()), 4),
        "mean_emitted_per_step": round(float((acc + 1).mean()), 4),
        # eq. ol at the forced acceptance rate (chance matches of the draft aside)
        "emitted_per_step_eq_ol": (round((1 - wl.alpha_forced ** (gamma + 1)) / (1 - wl.alpha_forced), 4)
                                   if forced and wl.alpha_forced < 1 else None),
        "device_flags": flags,
        "roofline": {"kernel": f"{gu_name} (target FFN gate/up, M={M}, N={2 * t.d_ffn}, K={t.d_model})",
                     "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "frac_of_copy": round(achieved / copy_gbs, 4),
                     "traffic": traffic_from_profiles() if headline else None,
                     "launch_ms": round(gu_ms, 5), "algorithmic_bytes_per_launch": gu_bytes},
        "cpu_baseline": None,
    }
    if n_batches > 1:
        # two-stream overlap against the same steps on one stream, and the
        # pipeline latency of eq. time with the measured pass times: per
        # step, with the paper's per-step barrier (C_{n,0} = 0), M batches
        # of draft time T_d and verify time T_v take T_d + M T_v when
        # T_v >= T_d; one stream takes M (T_d + T_v)
        td_ms, tv_ms = float(np.median(draft_ms)), float(np.median(verify_ms))
        one_ms, two_ms = elapsed_one / K * 1e3, elapsed / K * 1e3
        c_d = c_v = 0.0
        for _ in range(n_batches):
            c_d += td_ms
            c_v = max(c_d, c_v) + tv_ms
        res["pipeline"] = {
            "two_streams_ms_per_step": round(two_ms, 3), "one_stream_ms_per_step": round(one_ms, 3),
            "same_tokens": bool(same), "draft_ms_per_batch_step": round(td_ms, 3),
            "verify_ms_per_batch_step": round(tv_ms, 3),
            "hidden_draft_fraction": round((one_ms - two_ms) / (n_batches * td_ms), 3),
            "eq_time_pipelined_ms_per_step": round(c_v, 3),
            "eq_time_serial_ms_per_step": round(n_batches * (td_ms + tv_ms), 3)}
    if not args.no_cpu_baseline and headline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        cb = cpu_baseline(wl, B, gamma, float((acc + 1).mean()))
        res["cpu_baseline"] = {k: (round(v, 4) if isinstance(v, float) else v) for k, v in cb.items()}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
