"""Oracle of the paper's serving scheduler (test infrastructure only).

Written from Sections II-C and II-D ("Inference Cost Model", "Serving
Latency Model") and Sections III-A and III-B ("Optimal Communication Resource
Allocation", "Optimal Batching and Speculation Length", Algorithm 1) of the paper, in float64,
with plain loops.  It shares no code with the scheduler in the HIP library.

Model (per task k: input length I_k; per batch m: I_m = max input length,
b_m = number of tasks; speculation length l; acceptance rate alpha):
  * expected tokens emitted per step L = (1 - alpha^(l+1)) / (1 - alpha)
    (eq. ol; alpha = 1 gives l + 1), steps N = ceil(O_max / L) (eq. step_n,
    every task given O_max);
  * FLOPs of the i-th draft forward of step n (eq. flops_d) and of the
    verify forward of step n (eq. flops_v), with the KV lengths
    I_m + ((n-1) L - 1) + i - 1 and I_m + (n-1) L - 1 (fractional, from the
    expected L, as printed);
  * runtime of one forward T(b, F) = c1 F b + c2 (eq. latency_b2); a draft
    step is the sum over its l forwards (eq. d_latency), a verify step one
    forward (eq. v_latency);
  * two-stage pipeline per step (eq. time): C^d_{n,m} = C^d_{n,m-1} + T^d_{n,m},
    C_{n,m} = max(C^d_{n,m}, C_{n,m-1}) + T^v_{n,m}, C_{n,0} = 0; the step
    takes C_{n,M} (eq. latency_infer_batch) and T_inf = sum_n C_{n,M}
    (eq. latency_inf);
  * draft memory of a batch: parameters J (8 h1^2 + 4 h1 h2) bytes
    (eq. memory_model) plus KV 4 J h1 (I_m + O_m) bytes per task
    (eq. memory_kv), against the budget Gamma_s;
  * uplink: w_k* proportional to I_k / log2(1 + p_k g_k / sigma^2)
    (eq. opt_w), all uploads finishing together at
    t* = sum_k lambda I_k / (B_w log2(1 + p_k g_k / sigma^2)).

Readings (the printed algorithm is inconsistent with the equations it
implements in places):
  S-1 the candidate latency of batch [j..i] (eq. t_ij1, Algorithm 1 line 15)
      is sum_n [ max(Y[j-1,n,0] + T^d_n, Y[j-1,n,1]) + T^v_n ], the order
      eq. time and eq. tt1 / tt2 require;
  S-2 the best boundary j* and S[i] are recorded for every feasible j,
      j = 1 included; a prefix with no feasible boundary makes the task set
      infeasible;
  S-3 ties go to the larger j (the printed ">=" comparison);
  S-4 the plan is read back by jumping i -> S[i] - 1;
  S-5 h1 = model width, h2 = FFN width, J = number of decoder blocks; the
      FLOPs formulas are the paper's (two FFN matrices); the fitted c1
      absorbs the constant factor of the SwiGLU FFN actually run.

Option cfg["prefill_separate"] (an engine that processes the prompts before
the first step, as the HIP path does): step 1 is a decoding-stage step like
the others, with the draft's first forward over one token and the verify
over 1 + l tokens, I_m - 1 tokens cached (the prompt minus the token the
step starts from); the prompt processing is not part of T_inf.
"""
from __future__ import annotations

import itertools
import math
from typing import Dict, List, Sequence, Tuple


def expected_emitted(alpha: float, l: int) -> float:
    """L = (1 - alpha^(l+1)) / (1 - alpha) (eq. ol); l + 1 at alpha = 1."""
    if alpha >= 1.0:
        return float(l + 1)
    return (1.0 - alpha ** (l + 1)) / (1.0 - alpha)


def n_steps(o_max: int, alpha: float, l: int) -> int:
    """Decoding steps to emit O_max tokens in expectation (eq. step_n)."""
    return int(math.ceil(o_max / expected_emitted(alpha, l)))


def flops_draft(J: int, h1: int, h2: int, I_m: float, i: int, n: int, L: float) -> float:
    """FLOPs of the i-th draft forward at step n for one task (eq. flops_d):
    the prefill of the I_m prompt tokens for i = n = 1, else one token with
    I^kv = I_m + ((n - 1) L - 1) + i - 1 cached tokens."""
    if n == 1 and i == 1:
        return 4.0 * J * h1 * I_m * (2.0 * h1 + I_m + h2)
    kv = I_m + ((n - 1) * L - 1.0) + i - 1
    return 4.0 * J * h1 * (2.0 * h1 + kv + 1.0 + h2)


def flops_verify(J: int, h1: int, h2: int, I_m: float, l: int, n: int, L: float) -> float:
    """FLOPs of the verify forward at step n for one task (eq. flops_v): the
    prefill of I_m + l tokens at n = 1, else 1 + l tokens with
    I^kv = I_m + (n - 1) L - 1 cached tokens."""
    if n == 1:
        return 4.0 * J * h1 * (I_m + l) * (2.0 * h1 + I_m + l + h2)
    kv = I_m + (n - 1) * L - 1.0
    return 4.0 * J * h1 * (1.0 + l) * (2.0 * h1 + kv + l + 1.0 + h2)


def runtime(c: Tuple[float, float], F: float, b: int) -> float:
    """T(b, F) = c1 F b + c2 (eq. latency_b2)."""
    return c[0] * F * b + c[1]


def flops_draft_decode(J: int, h1: int, h2: int, kv: float) -> float:
    """FLOPs of one draft forward of one token over kv cached tokens (the
    decoding-stage form of eq. flops_d)."""
    return 4.0 * J * h1 * (2.0 * h1 + kv + 1.0 + h2)


def flops_verify_decode(J: int, h1: int, h2: int, kv: float, l: int) -> float:
    """FLOPs of one verify forward of 1 + l tokens over kv cached tokens (the
    decoding-stage form of eq. flops_v)."""
    return 4.0 * J * h1 * (1.0 + l) * (2.0 * h1 + kv + l + 1.0 + h2)


def step_times(cfg: Dict, b: int, I_m: float, l: int, n: int, L: float) -> Tuple[float, float]:
    """(T^d_{n,m}, T^v_{n,m}) of a batch of b tasks with input length I_m
    (eq. d_latency, eq. v_latency)."""
    Jd, h1d, h2d = cfg["draft"]
    Jv, h1v, h2v = cfg["target"]
    td = 0.0
    if cfg.get("prefill_separate"):
        # every step is a decoding step; before step n the caches hold the
        # prompt minus one token plus (n - 1) L emitted tokens
        base = I_m - 1.0 + (n - 1) * L
        for i in range(1, l + 1):
            td += runtime(cfg["c_draft"], flops_draft_decode(Jd, h1d, h2d, base + i - 1), b)
        tv = runtime(cfg["c_verify"], flops_verify_decode(Jv, h1v, h2v, base, l), b)
        return td, tv
    for i in range(1, l + 1):
        td += runtime(cfg["c_draft"], flops_draft(Jd, h1d, h2d, I_m, i, n, L), b)
    tv = runtime(cfg["c_verify"], flops_verify(Jv, h1v, h2v, I_m, l, n, L), b)
    return td, tv


def draft_memory(cfg: Dict, b: int, I_m: float, o_max: int) -> float:
    """Peak draft memory of a batch: parameters (eq. memory_model) plus the
    KV of b tasks of at most I_m + O_max tokens (eq. memory_kv), in bytes."""
    J, h1, h2 = cfg["draft"]
    return J * (8.0 * h1 * h1 + 4.0 * h1 * h2) + 4.0 * J * h1 * (I_m + o_max) * b


def pipeline_latency(cfg: Dict, batches: Sequence[Sequence[int]], lengths: Sequence[int], l: int,
                     alpha: float, o_max: int) -> float:
    """T_inf of a plan: batches (lists of task indices) processed in the given
    order in the two-stage pipeline at every step (eq. time,
    latency_infer_batch, latency_inf)."""
    L = expected_emitted(alpha, l)
    N = n_steps(o_max, alpha, l)
    total = 0.0
    for n in range(1, N + 1):
        cd = 0.0          # completion of the first stage, batches so far
        c = 0.0           # completion of both stages, batches so far
        for batch in batches:
            I_m = max(lengths[k] for k in batch)
            td, tv = step_times(cfg, len(batch), I_m, l, n, L)
            cd = cd + td
            c = max(cd, c) + tv
        total += c
    return total


def dp_batching(cfg: Dict, lengths: Sequence[int], l: int, alpha: float, o_max: int,
                mem_budget: float = 0.0) -> Tuple[List[List[int]], float]:
    """Algorithm 1 (batching for a given speculation length l), readings
    S-1..S-4.  Returns the batches (task indices, in pipeline order) and the
    minimum T_inf found (Y[K, 0, 0])."""
    K = len(lengths)
    order = sorted(range(K), key=lambda k: (lengths[k], k))      # task_list
    I = [float(lengths[k]) for k in order]
    L = expected_emitted(alpha, l)
    N = n_steps(o_max, alpha, l)
    # Y[i][n] = (first-stage completion, second-stage completion) of the
    # first i sorted tasks at step n; Y[0][n] = (0, 0)
    Y = [[(0.0, 0.0)] * (N + 1) for _ in range(K + 1)]
    best_val = [0.0] * (K + 1)
    S = [0] * (K + 1)
    for i in range(1, K + 1):
        found = False
        for j in range(1, i + 1):
            b = i - j + 1
            if mem_budget > 0 and draft_memory(cfg, b, I[i - 1], o_max) > mem_budget:
                continue
            temp = 0.0
            rows = []
            for n in range(1, N + 1):
                td, tv = step_times(cfg, b, I[i - 1], l, n, L)
                s0 = Y[j - 1][n][0] + td
                s1 = max(s0, Y[j - 1][n][1]) + tv
                rows.append((s0, s1))
                temp += s1
            if not found or best_val[i] >= temp:
                found = True
                best_val[i] = temp
                S[i] = j
                Y[i] = [(0.0, 0.0)] + rows
        if not found:
            raise ValueError(f"no feasible batch ends at sorted task {i}")
    batches = []
    i = K
    while i > 0:
        j = S[i]
        batches.append([order[k] for k in range(j - 1, i)])
        i = j - 1
    batches.reverse()
    return batches, best_val[K]


def plan(cfg: Dict, lengths: Sequence[int], l_max: int, alpha: float, o_max: int,
         mem_budget: float = 0.0) -> Dict:
    """Problem P3: the speculation length in 1..l_max with the lowest T_inf
    of its Algorithm 1 batching (ties to the smaller l)."""
    by_l = []
    best = None
    for l in range(1, l_max + 1):
        batches, t = dp_batching(cfg, lengths, l, alpha, o_max, mem_budget)
        by_l.append(t)
        if best is None or t < best["t_inf"]:
            best = {"l": l, "batches": batches, "t_inf": t}
    best["t_inf_by_l"] = by_l
    return best


def brute_force_batching(cfg: Dict, lengths: Sequence[int], l: int, alpha: float, o_max: int,
                         mem_budget: float = 0.0) -> Tuple[List[List[int]], float]:
    """Minimum T_inf over every split of the sorted task list into
    contiguous batches (2^(K-1) plans; small K only)."""
    K = len(lengths)
    order = sorted(range(K), key=lambda k: (lengths[k], k))
    best = None
    for cuts in itertools.product([0, 1], repeat=K - 1):
        batches, cur = [], [order[0]]
        for pos, cut in enumerate(cuts, start=1):
            if cut:
                batches.append(cur)
                cur = []
            cur.append(order[pos])
        batches.append(cur)
        if mem_budget > 0 and any(draft_memory(cfg, len(bt), max(lengths[k] for k in bt), o_max) > mem_budget
                                  for bt in batches):
            continue
        t = pipeline_latency(cfg, batches, lengths, l, alpha, o_max)
        if best is None or t < best[1]:
            best = (batches, t)
    return best


def uplink_allocation(lengths: Sequence[int], snr: Sequence[float], lam: float, bw: float):
    """Optimal bandwidth shares (eq. opt_w) and the common upload time
    t* = sum_k lam I_k / (bw log2(1 + snr_k)) (eq. bandw1 solved)."""
    a = [I / math.log2(1.0 + s) for I, s in zip(lengths, snr)]
    tot = sum(a)
    return [x / tot for x in a], lam * tot / bw


def upload_times(lengths: Sequence[int], snr: Sequence[float], w: Sequence[float], lam: float, bw: float):
    """Per-task upload latency lam I_k / (w_k bw log2(1 + snr_k)) (eq. ul_latency_k)."""
    return [lam * I / (wk * bw * math.log2(1.0 + s)) for I, s, wk in zip(lengths, snr, w)]
