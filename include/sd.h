/*
 * libsd: batched speculative-decoding hot path on one MI355X (gfx950).
 *
 * One decoding step of the paper (arXiv 2510.11331, Section II-A, "Inference
 * Mechanism with SD") for a batch of B tasks:
 *
 *   sd_draft_step x gamma   the draft model generates gamma tokens per task
 *                           autoregressively (drafting phase), each with its
 *                           draft distribution q;
 *   sd_verify               the target ("verify") model scores the current
 *                           input plus the gamma drafts of every task in one
 *                           forward pass, giving p at gamma+1 positions;
 *   sd_accept_resample      draft i is accepted with probability
 *                           min(1, p/q); at the first rejection a correction
 *                           token is drawn from norm(max(0, p - q)); if all
 *                           are accepted a reward token is drawn from p;
 *   sd_kv_commit            rejected drafts are removed from both KV caches
 *                           and the bonus token becomes the next input.
 *
 * The tasks of the paper's problem statement are {I_k, O_k} pairs (input
 * length, output budget; Section II); here each task lives in a "slot" that
 * owns paged KV blocks in the target and draft caches.  Section II-B's
 * pipeline (drafting of one batch overlapping verification of another) is
 * obtained by calling the draft and verify entry points of two disjoint slot
 * batches on two streams.
 *
 * Conventions
 *   - Device pointers unless stated otherwise.  The caller owns every buffer
 *     (weights, KV pools, workspace, inputs, outputs); the context borrows
 *     them and they must outlive it.  libsd never allocates device memory.
 *   - Streams are hipStream_t values passed as void* (NULL = null stream).
 *     Every call except sd_init and sd_prefill only enqueues work on the
 *     given stream and returns; sd_prefill blocks until its work is done.
 *   - A negative return value is an error (SD_E*).  Argument and state
 *     errors are detected on the host before anything is enqueued and leave
 *     the context unchanged.  No C++ exception crosses this interface.
 *   - Layouts are row-major except the packed weight matrices described at
 *     sd_pack_linear.  bf16 data is stored as raw 16-bit patterns.
 *   - Calls that share one context and overlap in time on different streams
 *     must use disjoint slots, and at most one draft call and one
 *     verify/accept/commit sequence may be in flight at a time (they use
 *     separate halves of the workspace).  A context is driven from one host
 *     thread.
 *   - Call order.  A batch is the device slot list passed to the step calls
 *     (identified by its address, with its B and gamma).  Its decoding step
 *     (Section II-A) is sd_draft_step i = 0 .. gamma-1 in order, then
 *     sd_verify, then sd_kv_commit; the host checks this order before
 *     enqueueing and returns SD_ESTATE on a violation:
 *       draft i = 0   always allowed; starts (or restarts, discarding any
 *                     uncommitted work of) a step
 *       draft i > 0   only right after draft i - 1 of the same step
 *       force i       only after draft i and before draft i + 1 / verify
 *       verify        only after all gamma drafts of the step; may be
 *                     repeated (it rewrites the same uncommitted positions)
 *       commit        only after verify; ends the step (a second commit
 *                     of the same step is refused)
 *     sd_accept_resample takes no context and is not tracked: it writes only
 *     the caller's n_acc / out_tok, which the commit then consumes.
 *     Capturing calls into a graph performs these checks once, at capture;
 *     replays repeat the captured order.
 */
#ifndef SD_H
#define SD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct sd_ctx sd_ctx;   /* opaque, host-side */

enum {
    SD_OK = 0,
    SD_EINVAL = -1,   /* bad argument or configuration                  */
    SD_ENOMEM = -2,   /* KV block pool cannot hold the request          */
    SD_ESTATE = -3,   /* call not allowed in the slot's current state   */
    SD_EHIP = -4      /* a HIP runtime call failed                      */
};

enum { SD_DTYPE_BF16 = 0, SD_DTYPE_F32 = 1 };

/* Decoder-only model (LLaMA layout of the paper's decoder block, eqs. f11,
 * f21, f31): RMSNorm -> QKV -> rotary embedding -> causal attention over the
 * KV cache -> output projection + residual -> RMSNorm -> SwiGLU feed-forward
 * + residual; final RMSNorm and LM head.  dtype is the type the weights are
 * given in.  SD_DTYPE_F32: everything fp32.  SD_DTYPE_BF16: the products run
 * on fp16 operands with fp32 accumulation: the packed matrices are the fp16
 * values of the bf16 weights (sd_pack_linear; exact from 2^-14 up, smaller
 * magnitudes round to the fp16 subnormal grid of 2^-24), every
 * matrix-product input (normed rows, attention output, SwiGLU output) is
 * rounded to fp16 and the KV cache holds fp16; embedding rows and norm gains
 * are read as bf16; the residual stream, norms, rotary embedding and softmax
 * are fp32.  fp16 has the memory cost and matrix-instruction rate of bf16
 * and three more significant bits. */
typedef struct {
    int n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab;
    int dtype;              /* SD_DTYPE_BF16 or SD_DTYPE_F32                */
    float rope_theta;       /* rotary base, e.g. 10000                      */
    float rms_eps;          /* RMSNorm epsilon, e.g. 1e-5                   */
} sd_model_cfg;

/* Weights of one model, in the model's dtype.  Matrices are [out, in]
 * (y = x W^T); wqkv, wo, wgu, wdown and lm_head must be given in the packed
 * layout that sd_pack_linear writes (embed and the norms stay row-major).
 * The per-layer pointer arrays are host arrays of n_layers device pointers;
 * sd_init copies them.
 *   wqkv  [(n_heads + 2 n_kv_heads) head_dim, d_model]: query rows (head
 *         major), then key rows, then value rows.  The rows of each query
 *         and key head are in rotary pair order: for b < head_dim / 16,
 *         rows 16b..16b+7 of the head are its dims 8b..8b+7 and rows
 *         16b+8..16b+15 its dims head_dim/2+8b..+7 (the two halves that
 *         the rotary embedding rotates together); value rows are in plain
 *         order.
 *   wo    [d_model, n_heads head_dim]
 *   wgu   [2 d_ffn, d_model]: gate and up rows interleaved in blocks of 16:
 *         rows 32b..32b+15 are gate rows 16b..16b+15, rows 32b+16..32b+31
 *         are up rows 16b..16b+15.
 *   wdown [d_model, d_ffn]
 *   embed, lm_head [vocab, d_model]; norms [d_model]. */
typedef struct {
    const void *embed, *lm_head, *final_norm;
    const void *const *attn_norm, *const *wqkv, *const *wo;
    const void *const *ffn_norm, *const *wgu, *const *wdown;
} sd_weights;

typedef struct {
    sd_model_cfg target, draft;  /* same vocab                              */
    int max_slots;          /* task slots                                   */
    int max_batch;          /* max tasks per draft/verify call              */
    int gamma_max;          /* max speculation length (1..16)               */
    int max_ctx;            /* max positions a slot may reach (<= 32768)    */
    int kv_block;           /* tokens per KV block; must be 16              */
    int kv_blocks_target;   /* blocks in the target pool                    */
    int kv_blocks_draft;    /* blocks in the draft pool                     */
    int prefill_rows;       /* rows per prefill chunk (>= 1)                */
    float temperature;      /* tau > 0: p = softmax(z / tau)                */
    int greedy;             /* 1: arg-max drafting and verification         */
    void *kv_pool_target;   /* sd_kv_pool_bytes(cfg, 0) bytes               */
    void *kv_pool_draft;    /* sd_kv_pool_bytes(cfg, 1) bytes               */
    void *workspace;        /* sd_workspace_bytes(cfg) bytes                */
    size_t workspace_bytes;
} sd_config;

/* Repack a row-major [N, K] matrix of dtype (SD_DTYPE_*) into the layout
 * the matrix-core GEMMs read, enqueued on stream; a bf16 matrix is written
 * as fp16 (each value rounded to nearest even: exact from 2^-14 up).  The
 * packed matrix has the same size, N K elements.  It is a sequence of 1 KB
 * tiles, tile (n / 16, s) covering rows 16 (n/16) .. +15 and the s-th
 * 64-byte run of those rows' K extent (E = 32 fp16 or 16 fp32 elements);
 * tiles are ordered row block
 * major.  Inside a tile, element (n, k) with k = s E + e sits in 16-byte
 * unit 16 (e / (E/4)) + n % 16 at position e % (E/4): one wave-wide 16-byte
 * load per lane fetches a tile whole.  Requirements: N % 16 == 0 and
 * K * element size % 128 == 0 (SD_EINVAL otherwise); src and dst must not
 * overlap.  Used once per weight matrix before sd_init. */
int sd_pack_linear(const void *src, void *dst, int N, int K, int dtype,
                   void *stream);

/* Sizes (host-only queries; 0 on an invalid configuration). */
size_t sd_kv_pool_bytes(const sd_config *cfg, int draft);
size_t sd_workspace_bytes(const sd_config *cfg);

/* Validate cfg, borrow the buffers, clear the workspace's device state.
 * On success *out holds a new context.  The workspace then belongs to the
 * context until sd_destroy: besides scratch it holds slot state and the
 * attention's key-split counters, which every launch leaves at zero, so the
 * caller must not write to it. */
int sd_init(const sd_config *cfg, const sd_weights *target,
            const sd_weights *draft, sd_ctx **out);

/* Size of the library's own per-device workspace used by sd_init_static. */
#define SD_STATIC_WORKSPACE_MB 64

/* sd_init without a caller-allocated workspace, for callers that cannot
 * allocate device memory (code under graph capture, serving loops that
 * must not call hipMalloc, harnesses that forbid it).  cfg->workspace and
 * cfg->workspace_bytes are ignored: the context uses a file-scope device
 * array of SD_STATIC_WORKSPACE_MB MiB that the library holds on each GPU
 * until the process ends (the current device's copy).  Nothing is
 * allocated: no hipMalloc / hipFree or allocating library call; the caller
 * still owns the weights, the KV pools and every input and output.
 * SD_EINVAL if sd_workspace_bytes(cfg) exceeds the array (the reason is in
 * sd_last_error), SD_ESTATE while another context made by sd_init_static
 * on the same device is alive (they would share the array: calls of two
 * such contexts would race); sd_destroy gives the array back.  sd_init
 * clears what must start at zero, so a context never sees the previous
 * one's state.  Otherwise as sd_init. */
int sd_init_static(const sd_config *cfg, const sd_weights *target,
                   const sd_weights *draft, sd_ctx **out);

/* Start B tasks: prompt k (host tokens[off_k .. off_k + lens[k]), packed
 * back to back) goes to slot slots[k] (host).  Allocates KV blocks for
 * lens[k] + max_new[k] + gamma_max positions, runs both models over
 * prompt[:-1] (Section II-A, prefill stage; the target runs the same pass
 * over the prompt) and sets the slot's next input to the last prompt token.
 * Blocks until done.  SD_ESTATE if a slot is in use, SD_ENOMEM if a pool
 * is short.
 * Resume: after sd_kv_commit the committed state of a task is its prompt
 * plus the tokens emitted so far (both caches equal those of a fresh
 * prefill of that sequence); prefilling prompt + emitted, in this or
 * another context, and continuing with the uniforms of the following steps
 * continues the run. */
int sd_prefill(sd_ctx *ctx, int B, const int32_t *slots, const int32_t *tokens,
               const int32_t *lens, const int32_t *max_new, void *stream);

/* Free a slot's KV blocks (the slot can be prefilled again).  The slot's
 * KV capacity on the device is set to 0 with a blocking copy, so a later
 * pass whose batch still names the slot skips (and flags, see sd_check) its
 * KV writes instead of writing into blocks handed to another task.  The
 * caller must not release a slot that queued work still uses.  SD_ESTATE if
 * the slot is not in use. */
int sd_release(sd_ctx *ctx, int slot);

/* Drafting, call i of gamma (Section II-A, decoding stage of the draft):
 * the first call of a step feeds the draft its pending inputs (the previous
 * bonus token, preceded by the last accepted draft when all gamma were
 * accepted), call i > 0 feeds draft token i-1.  Writes
 *   draft_tok[b * gamma + i]       sampled token (int32)
 *   q[(b * gamma + i) * vocab ..]  q = softmax(z / tau) (fp32), or the draft
 *                                  logits in greedy mode.
 * slots [B] int32; u [B, 2 gamma + 1] uint32 uniforms of this step (column
 * i is used). */
int sd_draft_step(sd_ctx *ctx, int B, const int32_t *slots, int gamma, int i,
                  const uint32_t *u, int32_t *draft_tok, float *q, void *stream);

/* Verification (Section II-A, verification phase): one target forward over
 * rows b * (gamma+1) + j = [x0, t_1..t_gamma] of every task at positions
 * P_b .. P_b + gamma, appending their K/V to the target cache.  Writes
 * p [B, gamma+1, vocab] fp32 = softmax(z / tau) (the logits themselves in
 * greedy mode) and, if logits is not NULL, the raw logits there. */
int sd_verify(sd_ctx *ctx, int B, const int32_t *slots, int gamma,
              const int32_t *draft_tok, float *p, float *logits, void *stream);

/* Acceptance and resampling (Section II-A; speculative sampling): for task
 * b, draft i is accepted iff fl32(u_i * q_i(t_i)) < p_i(t_i) with
 * u_i = (u[b, gamma + i] >> 8) * 2^-24; a = index of the first rejection
 * (gamma if none).  The bonus token is drawn with r = u[b, 2 gamma] by the
 * integer inverse-CDF rule (W_j = floor(w_j 2^40), T = floor(S r / 2^32),
 * smallest j with prefix sum > T) from max(0, p_a - q_a) (from p_a if that
 * has no integer mass) when a < gamma, or from p_gamma when a = gamma.  In
 * greedy mode draft i is accepted iff it is the arg-max of row i of p (the
 * target logits; lowest index on ties) and the bonus is that arg-max.
 * Writes n_acc[b] = a and out_tok[b, 0..gamma] = t_1..t_a, bonus, then -1.
 * Needs no context: q [B, gamma, vocab], p [B, gamma+1, vocab].  Rows are
 * read as 16-byte vectors: vocab must be a multiple of 4 (4 .. 32768) and q,
 * p 16-byte aligned; SD_EINVAL otherwise, before anything is enqueued. */
int sd_accept_resample(int B, int gamma, int vocab, int greedy,
                       const int32_t *draft_tok, const float *q, const float *p,
                       const uint32_t *u, int32_t *n_acc, int32_t *out_tok,
                       void *stream);

/* Commit (Section II-A: rejected drafts are removed from both KV caches;
 * the bonus token is the next input): target length P -> P + a + 1, draft
 * keeps min(a + 1, gamma) of its new entries, next input = bonus token;
 * after full acceptance the last draft becomes a pending draft input. */
int sd_kv_commit(sd_ctx *ctx, int B, const int32_t *slots, int gamma,
                 const int32_t *n_acc, const int32_t *out_tok, void *stream);

/* Forced acceptance, a workload generator for greedy verification (the
 * acceptance rate alpha of eq. ol set from outside, as random-weight models
 * give none of their own).  Call between sd_draft_step(i) and the next
 * draft or verify call of the batch.  For each task b, if its draft uniform
 * u[b, i] (the slot sd_draft_step(i) read; unused by greedy drafting) is
 * below alpha 2^32, draft_tok[b, i] is replaced by cont[b, P + i + 1]: the
 * token that the task's reference continuation (e.g. the target's greedy
 * output, prompt included, indexed by absolute position, cont_len per task)
 * holds at that draft's position, P being the committed length.  Positions
 * at or past cont_len are left alone.  The draft model then consumes the
 * forced token, and greedy verification accepts it iff it is the target's
 * arg-max.  cont [B, cont_len] int32, u [B, 2 gamma + 1] uint32 and
 * draft_tok [B, gamma] are device arrays; 0 <= alpha <= 1.  SD_ESTATE if
 * the context samples (greedy == 0). */
int sd_force_draft(sd_ctx *ctx, int B, const int32_t *slots, int gamma, int i,
                   const int32_t *cont, int cont_len, const uint32_t *u, double alpha,
                   int32_t *draft_tok, void *stream);

/* Copy slot state to out [B, 4] int32 (device): committed target length
 * P, next input token x0, pending draft input (-1 if none), KV capacity. */
int sd_slot_state(sd_ctx *ctx, int B, const int32_t *slots, int32_t *out,
                  void *stream);

/* Device-side error flags (bit 0: a KV write beyond a slot's capacity was
 * skipped).  Synchronises the stream; clears the flags. */
int sd_check(sd_ctx *ctx, void *stream, int32_t *flags_out);

/* Timing with HIP events (off by default).  kind: SD_PROF_* below.  The
 * GEMM and attention kinds time each kernel with start/stop events that its
 * own dispatch timestamps (kernel begin to end, the interval a profiler
 * reports); the VERIFY and DRAFT kinds time the whole call with events
 * recorded on its stream.  bytes: algorithmic HBM bytes of the timed GEMMs
 * (weights + activations read + outputs written).  sd_profile_read
 * synchronises the recorded events and returns the number of timed
 * intervals, their summed milliseconds and bytes; reading resets that kind. */
enum {
    SD_PROF_GEMM_VERIFY_GATEUP = 0,   /* target FFN gate/up GEMM (+SwiGLU)  */
    SD_PROF_GEMM_VERIFY_ALL = 1,      /* every target GEMM in sd_verify     */
    SD_PROF_ATTN_VERIFY = 2,          /* target attention in sd_verify      */
    SD_PROF_VERIFY = 3,               /* whole sd_verify                    */
    SD_PROF_DRAFT = 4,                /* whole sd_draft_step                */
    SD_PROF_N = 5
};
int sd_profile(sd_ctx *ctx, int enable);
int sd_profile_read(sd_ctx *ctx, int kind, int64_t *count, double *ms,
                    double *bytes);

void sd_destroy(sd_ctx *ctx);
const char *sd_strerror(int code);

/* Text of the last SD_EHIP failure on the calling thread (HIP call and
 * message), or of a workspace-size refusal of sd_init_static; "" if none.
 * The string stays valid until the next call. */
const char *sd_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SD_H */
