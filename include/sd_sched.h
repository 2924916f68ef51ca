/* Serving scheduler of the speculative-decoding system: host-side planning
 * of batches and speculation length from a runtime model (part of libsd).
 *
 * Everything here is host arithmetic in double precision; no call touches
 * the GPU.  Pointers are host pointers.  Return values are the SD_* codes of
 * sd.h (SD_OK, SD_EINVAL for bad arguments, SD_ENOMEM when the draft memory
 * budget admits no batching).  Outputs are written only on SD_OK.
 *
 * The model is the paper's (Sections II-C "Inference Cost Model" and II-D
 * "Serving Latency Model"):
 *   - a task k has input length I_k; every task is given O_max output
 *     tokens (the simplification of Section III-B, so every batch runs every
 *     step); a batch m of b_m tasks has I_m = max of its input lengths;
 *   - tokens emitted per step L = (1 - alpha^(l+1)) / (1 - alpha) (eq. ol;
 *     l + 1 at alpha = 1) and steps N = ceil(O_max / L) (eq. step_n);
 *   - per-task FLOPs of the i-th draft forward and of the verify forward at
 *     step n: eq. flops_d and eq. flops_v, with the (fractional) KV lengths
 *     I_m + ((n-1) L - 1) + i - 1 and I_m + (n-1) L - 1;
 *   - runtime of one forward T(b, F) = c1 F b + c2 (eq. latency_b2), the
 *     draft step the sum over its l forwards (eq. d_latency), the verify
 *     step one forward (eq. v_latency);
 *   - two-stage pipeline at every step (eq. time): C^d_{n,m} = C^d_{n,m-1}
 *     + T^d_{n,m}, C_{n,m} = max(C^d_{n,m}, C_{n,m-1}) + T^v_{n,m},
 *     C_{n,0} = 0; T_inf = sum_n C_{n,M} (eqs. latency_infer_batch,
 *     latency_inf);
 *   - draft memory of a batch J_d (8 h1^2 + 4 h1 h2) + 4 J_d h1 (I_m + O_max)
 *     b_m bytes (eqs. memory_model, memory_kv).
 * h1 is the model width, h2 the FFN width, J the number of decoder blocks.
 */
#ifndef SD_SCHED_H
#define SD_SCHED_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int n_layers;   /* J  */
    int d_model;    /* h1 */
    int d_ffn;      /* h2 */
} sd_sched_model;

typedef struct {
    sd_sched_model draft, target;
    double c1_draft, c2_draft;     /* draft forward: T = c1 F b + c2 (seconds)  */
    double c1_verify, c2_verify;   /* verify forward                            */
    double alpha;                  /* acceptance rate, 0 <= alpha <= 1          */
    int o_max;                     /* output tokens given to every task, >= 1   */
    double mem_budget;             /* draft memory budget in bytes; <= 0: none  */
    int prefill_separate;          /* 1: the prompts are processed before step
                                      1 (as sd_prefill does), so step 1 is a
                                      decoding-stage step like the others: the
                                      draft forwards over one token, the verify
                                      over 1 + l tokens, with I_m - 1 + (n-1) L
                                      tokens cached before step n; prompt
                                      processing is not part of T_inf.
                                      0: the paper's first step (eqs. flops_d,
                                      flops_v at n = 1).                        */
} sd_sched_cfg;

/* Expected inference latency T_inf (seconds) of a plan: task k (input length
 * input_len[k] >= 1) is in batch batch_of[k] (0 .. n_batches-1; every batch
 * non-empty), batches are processed in index order at every step, with
 * speculation length l >= 1.  The memory budget is not checked here. */
int sd_sched_latency(const sd_sched_cfg *cfg, int K, const int32_t *input_len, int n_batches,
                     const int32_t *batch_of, int l, double *t_inf);

/* Batching for a given speculation length l (Section III-B, Algorithm 1).
 * Tasks are sorted by input length (ties by index); a batch is a run of the
 * sorted order.  Dynamic program over the sorted prefix: Y[i][n] = (first-
 * stage, second-stage) completion at step n of the plan chosen for the
 * first i tasks; for each i every last batch [j..i] that fits the memory
 * budget is scored sum_n [max(Y[j-1][n][0] + T^d_n, Y[j-1][n][1]) + T^v_n]
 * (the order of eq. time; the printed eq. t_ij1 places T^d elsewhere), the
 * lowest score wins with ties to the larger j, and the plan is read back by
 * jumping from i to j - 1.  Outputs: batch_of[K] (batch index of every
 * task, batches in pipeline order = ascending input length), *n_batches, and
 * *t_inf, the plan's T_inf.  SD_ENOMEM if some sorted prefix has no batch
 * within the budget.  Cost O(K^2 N l). */
int sd_sched_batching(const sd_sched_cfg *cfg, int K, const int32_t *input_len, int l, int32_t *batch_of,
                      int *n_batches, double *t_inf);

/* Speculation length (Section III-B, problem P3): the batching of
 * sd_sched_batching for every l in 1..l_max, keeping the lowest T_inf (ties
 * to the smaller l).  Outputs as sd_sched_batching plus *l_best and, if
 * t_inf_by_l is not null, T_inf of every l in t_inf_by_l[l_max]. */
int sd_sched_plan(const sd_sched_cfg *cfg, int K, const int32_t *input_len, int l_max, int32_t *batch_of,
                  int *n_batches, int *l_best, double *t_inf, double *t_inf_by_l);

/* Uplink bandwidth shares (Section III-A, eq. opt_w): w_k proportional to
 * I_k / log2(1 + snr_k) with sum w_k = 1, so that every upload of
 * lambda_bits I_k bits over w_k bandwidth_hz finishes at the same time
 * *t_com = sum_k lambda_bits I_k / (bandwidth_hz log2(1 + snr_k)).
 * snr_k = p_k g_k / sigma^2 > 0. */
int sd_sched_uplink(int K, const int32_t *input_len, const double *snr, double lambda_bits, double bandwidth_hz,
                    double *w, double *t_com);

#ifdef __cplusplus
}
#endif

#endif /* SD_SCHED_H */
