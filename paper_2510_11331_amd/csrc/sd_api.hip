// libsd host runtime: configuration checks, workspace layout, the host KV
// block allocator, and the launch sequences of the prefill, draft and verify
// passes and of the acceptance / commit step.  See include/sd.h.
#include "sd.h"
#include "sd_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <deque>
#include <mutex>
#include <new>
#include <unordered_map>
#include <vector>

namespace sd {
size_t attention_lds_bytes(int hd, int esz, int qmax);
}

using namespace sd;

namespace {

constexpr int KV_BLOCK = 16;
constexpr int MAX_KSPLIT = 6;   // K splits of a residual projection (partial sums in the workspace)
constexpr int SKINNY_MAX_KSPLIT = 4;   // of those on the skinny GEMM

struct ModelRT {
  sd_model_cfg c{};
  size_t esz = 2;
  const void *embed = nullptr, *lm_head = nullptr, *final_norm = nullptr;
  std::vector<const void*> attn_norm, wqkv, wo, ffn_norm, wgu, wdown;
  unsigned char* pool = nullptr;
  int n_blocks = 0;
  float2* rope_tab = nullptr;   // [rope_pos, head_dim/2] rotary (cos, sin), in the workspace
  int rope_pos = 0;
  size_t layer_bytes = 0;   // bytes of one layer's pool
  int nqkv() const { return (c.n_heads + 2 * c.n_kv_heads) * c.head_dim; }
  int nq() const { return c.n_heads * c.head_dim; }
  int G() const { return c.n_heads / c.n_kv_heads; }
};

struct Lane {
  int rows = 0;                 // row capacity
  int32_t *row_tok = nullptr, *row_pos = nullptr, *row_slot = nullptr, *row_blk = nullptr, *rowblocks = nullptr;
  int32_t* row_bt = nullptr;    // [decode row blocks, mbps] block-table rows of a decode pass's tasks
  int rb_cap = 0;
  float *x = nullptr, *q = nullptr, *logits = nullptr;
  void *xn = nullptr, *att = nullptr, *hmid = nullptr;
  float* part = nullptr;        // [MAX_KSPLIT, part_rows, d] K-split partial sums
  int part_rows = 0;
  float *attn_o = nullptr, *attn_ml = nullptr;
  int32_t* attn_cnt = nullptr;  // [attn_items] split arrival counters (zero between launches)
  size_t attn_o_cap = 0, attn_ml_cap = 0;
  int attn_items = 0;           // (row block, kv head) items the split partials hold
};

struct Slot {
  bool active = false;
  std::vector<int> tblocks, dblocks;
};

// Where one batch (the device slot list passed to the step calls) stands in
// its current step: the decoding step of Section II-A is gamma draft calls
// in order, then verification, then the commit that trims both caches.
struct Phase {
  int B = 0, gamma = 0;
  int drafted = 0;        // draft calls 0 .. drafted-1 of this step are done
  bool verified = false;  // the verify pass of this step has been enqueued
};

// One timed interval: either the span of a whole call (events recorded on
// the stream around it) or one kernel (events stamped by its own dispatch),
// counted under every kind in the mask.
struct ProfRec {
  unsigned mask = 0;
  bool kernel = false;
  hipEvent_t a = nullptr, b = nullptr;
  double bytes = 0;
};

}  // namespace

struct sd_ctx {
  sd_config cfg{};
  ModelRT tgt, dft;
  int mbps = 0;                 // max blocks per slot
  int32_t *state = nullptr, *bt_t = nullptr, *bt_d = nullptr, *err = nullptr;
  Lane lv, ld;                  // verify / prefill lane, draft lane
  int keys_per_split = 64, attn_splits = 1;
  std::vector<Slot> slots;
  std::vector<int> free_t, free_d;
  std::unordered_map<const void*, Phase> phases;   // by device slot-list address
  int static_dev = -1;          // device whose static workspace this context holds (sd_init_static)
  bool prof = false;
  std::vector<ProfRec> recs;
};

namespace {

thread_local char g_last_error[320] = "";

int hip_fail(hipError_t e, const char* what, int line) {
  snprintf(g_last_error, sizeof(g_last_error), "sd_api.hip:%d %s: %s", line, what, hipGetErrorString(e));
  return SD_EHIP;
}

#define HIPCHK(x)                                                  \
  do {                                                             \
    hipError_t e_ = (x);                                           \
    if (e_ != hipSuccess) return hip_fail(e_, #x, __LINE__);       \
  } while (0)

size_t esize(int dtype) { return dtype == SD_DTYPE_F32 ? 4 : 2; }

bool model_ok(const sd_model_cfg& m) {
  if (m.n_layers < 1 || m.d_model < 1 || m.n_heads < 1 || m.n_kv_heads < 1 || m.d_ffn < 1 || m.vocab < 1)
    return false;
  if (m.dtype != SD_DTYPE_BF16 && m.dtype != SD_DTYPE_F32) return false;
  if (m.head_dim != 64 && m.head_dim != 128) return false;
  if (m.n_heads * m.head_dim != m.d_model) return false;
  if (m.n_heads % m.n_kv_heads) return false;
  if ((m.n_heads / m.n_kv_heads) * 2 > ATTN_QMAX) return false;
  const size_t e = esize(m.dtype);
  // GEMM K dims stream in 256-byte chunks; N dims come in 16-column tiles
  if ((m.d_model * e) % GEMM_CHUNK || (m.d_ffn * e) % GEMM_CHUNK) return false;
  if (m.vocab % 16 || m.d_ffn % 16 || m.vocab > 32768) return false;   // row kernels hold <= 32768 entries
  if (!(m.rope_theta > 0.f) || !(m.rms_eps > 0.f)) return false;
  return true;
}

bool cfg_ok(const sd_config* c) {
  if (!c) return false;
  if (!model_ok(c->target) || !model_ok(c->draft)) return false;
  if (c->target.vocab != c->draft.vocab) return false;
  if (c->max_slots < 1 || c->max_batch < 1 || c->max_batch > c->max_slots) return false;
  if (c->gamma_max < 1 || c->gamma_max > 16) return false;
  if (c->kv_block != KV_BLOCK) return false;
  if (c->max_ctx < 2 || c->max_ctx > MAX_CTX || c->kv_blocks_target < 1 || c->kv_blocks_draft < 1) return false;
  if (c->prefill_rows < 1) return false;
  if (!(c->temperature > 0.f)) return false;
  if ((c->target.n_heads / c->target.n_kv_heads) * (c->gamma_max + 1) > ATTN_QMAX) return false;
  return true;
}

size_t pool_bytes(const sd_model_cfg& m, int blocks) {
  return (size_t)m.n_layers * blocks * 2 * m.n_kv_heads * KV_BLOCK * m.head_dim * esize(m.dtype);
}

int keys_per_split(int max_ctx) {
  // aim for at most 12 key splits per (row block, kv head)
  const int chunks = (max_ctx + 63) / 64;
  const int per = std::max(1, (chunks + 11) / 12);
  return per * 64;
}

struct Alloc {
  unsigned char* base;   // null: size only
  size_t off = 0;
  template <typename P>
  P* take(size_t bytes) {
    off = (off + 255) & ~(size_t)255;
    P* r = base ? (P*)(base + off) : nullptr;
    off += bytes;
    return r;
  }
};

struct Dims {
  int d = 0, nqkv = 0, nq = 0, F = 0, V = 0, KV = 0, hd = 0, G = 1;
  size_t esz = 2;
};

Dims dims_max(const sd_model_cfg& a, const sd_model_cfg* b) {
  Dims r;
  auto upd = [&](const sd_model_cfg& m) {
    r.d = std::max(r.d, m.d_model);
    r.nqkv = std::max(r.nqkv, (m.n_heads + 2 * m.n_kv_heads) * m.head_dim);
    r.nq = std::max(r.nq, m.n_heads * m.head_dim);
    r.F = std::max(r.F, m.d_ffn);
    r.V = std::max(r.V, m.vocab);
    r.KV = std::max(r.KV, m.n_kv_heads);
    r.hd = std::max(r.hd, m.head_dim);
    r.G = std::max(r.G, m.n_heads / m.n_kv_heads);
    r.esz = std::max(r.esz, esize(m.dtype));
  };
  upd(a);
  if (b) upd(*b);
  return r;
}

// lane buffers; decode_rb = row blocks of a decode pass, qmax_dec = query vectors per row block
void lay_lane(Alloc& al, Lane& ln, int rows, const Dims& D, int decode_rb, int qmax_dec, int splits,
              int logits_rows, int prefill_rb, int mbps) {
  rows = (rows + GEMM_MROWS - 1) / GEMM_MROWS * GEMM_MROWS;   // operands are read in whole 64-row blocks
  ln.rows = rows;
  ln.row_tok = al.take<int32_t>(sizeof(int32_t) * rows);
  ln.row_pos = al.take<int32_t>(sizeof(int32_t) * rows);
  ln.row_slot = al.take<int32_t>(sizeof(int32_t) * rows);
  ln.row_blk = al.take<int32_t>(sizeof(int32_t) * rows);
  ln.rb_cap = prefill_rb;
  ln.rowblocks = al.take<int32_t>(sizeof(int32_t) * 2 * std::max(1, prefill_rb));
  ln.row_bt = al.take<int32_t>(sizeof(int32_t) * (size_t)decode_rb * mbps);
  ln.x = al.take<float>(sizeof(float) * rows * D.d);
  ln.xn = al.take<void>(D.esz * rows * D.d);
  ln.q = al.take<float>(sizeof(float) * rows * D.nq);
  ln.att = al.take<void>(D.esz * rows * D.nq);
  ln.hmid = al.take<void>(D.esz * rows * D.F);
  ln.part_rows = std::min(rows, 640);   // the largest pass whose residual projections split K
  ln.part = al.take<float>(sizeof(float) * MAX_KSPLIT * ln.part_rows * D.d);
  ln.logits = logits_rows ? al.take<float>(sizeof(float) * logits_rows * D.V) : nullptr;
  ln.attn_items = decode_rb * D.KV;
  ln.attn_o_cap = (size_t)ln.attn_items * splits * qmax_dec * D.hd;
  ln.attn_ml_cap = (size_t)ln.attn_items * splits * qmax_dec * 2;
  ln.attn_o = al.take<float>(sizeof(float) * ln.attn_o_cap);
  ln.attn_ml = al.take<float>(sizeof(float) * ln.attn_ml_cap);
  ln.attn_cnt = al.take<int32_t>(sizeof(int32_t) * std::max(1, ln.attn_items));
}

// prefill rows per attention row block: as many as fit the 64 query vectors
// of a workgroup and the default 64 KB of dynamic LDS
int prefill_qb(const sd_model_cfg& m) {
  const int G = m.n_heads / m.n_kv_heads;
  int qb = std::max(1, ATTN_QMAX / G);
  if (m.dtype == SD_DTYPE_BF16) return qb;   // the matrix kernel's LDS does not grow with the rows
  while (qb > 1 && attention_lds_bytes(m.head_dim, esize(m.dtype), qb * G) > 64 * 1024) --qb;
  return qb;
}

size_t layout(const sd_config* c, sd_ctx* ctx) {
  Alloc al{ctx ? (unsigned char*)c->workspace : nullptr};
  const int mbps = (c->max_ctx + KV_BLOCK - 1) / KV_BLOCK;
  int32_t* state = al.take<int32_t>(sizeof(int32_t) * ST_N * c->max_slots);
  int32_t* bt_t = al.take<int32_t>(sizeof(int32_t) * (size_t)c->max_slots * mbps);
  int32_t* bt_d = al.take<int32_t>(sizeof(int32_t) * (size_t)c->max_slots * mbps);
  int32_t* err = al.take<int32_t>(sizeof(int32_t) * 4);
  float2* tab_t = al.take<float2>(sizeof(float2) * (size_t)mbps * KV_BLOCK * (c->target.head_dim / 2));
  float2* tab_d = al.take<float2>(sizeof(float2) * (size_t)mbps * KV_BLOCK * (c->draft.head_dim / 2));
  const int kps = keys_per_split(c->max_ctx);
  const int splits = (c->max_ctx + kps - 1) / kps;
  const Dims Dt = dims_max(c->target, &c->draft);
  const Dims Dd = dims_max(c->draft, nullptr);
  const int rows_v = std::max(c->max_batch * (c->gamma_max + 1), c->prefill_rows);
  const int qb = std::min(prefill_qb(c->target), prefill_qb(c->draft));
  const int prefill_rb = c->prefill_rows / qb + c->max_slots + 1;
  Lane lv, ld;
  lay_lane(al, lv, rows_v, Dt, c->max_batch, (c->gamma_max + 1) * Dt.G, splits, 0, prefill_rb, mbps);
  lay_lane(al, ld, 2 * c->max_batch, Dd, c->max_batch, 2 * Dd.G, splits, c->max_batch, 0, mbps);
  if (ctx) {
    ctx->mbps = mbps;
    ctx->state = state;
    ctx->bt_t = bt_t;
    ctx->bt_d = bt_d;
    ctx->err = err;
    ctx->tgt.rope_tab = tab_t;
    ctx->dft.rope_tab = tab_d;
    ctx->tgt.rope_pos = ctx->dft.rope_pos = mbps * KV_BLOCK;
    ctx->lv = lv;
    ctx->ld = ld;
    ctx->keys_per_split = kps;
    ctx->attn_splits = splits;
  }
  return (al.off + 255) & ~(size_t)255;
}

// ---------------------------------------------------------------- profiling

// kinds < 0 are ignored; kernel = true: r.a / r.b go to the kernel's launch
void prof_begin(sd_ctx* ctx, hipStream_t s, ProfRec& r, int kind, int kind2, double bytes, bool kernel) {
  r = ProfRec{};
  unsigned mask = (kind >= 0 ? 1u << kind : 0u) | (kind2 >= 0 ? 1u << kind2 : 0u);
  if (!ctx->prof || !mask) return;
  if (hipEventCreate(&r.a) != hipSuccess) return;
  if (hipEventCreate(&r.b) != hipSuccess) {
    hipEventDestroy(r.a);
    r.a = nullptr;
    return;
  }
  if (!kernel && hipEventRecord(r.a, s) != hipSuccess) {
    hipEventDestroy(r.a);
    hipEventDestroy(r.b);
    r.a = r.b = nullptr;
    return;
  }
  r.mask = mask;
  r.kernel = kernel;
  r.bytes = bytes;
}

void prof_end(sd_ctx* ctx, hipStream_t s, ProfRec& r) {
  if (!r.mask) return;
  if (!r.kernel) hipEventRecord(r.b, s);
  ctx->recs.push_back(r);
}

// ---------------------------------------------------------------- GEMM planning

struct GemmPlan {
  int nt, mt, kw, gx, ksplit, gz;
  int tu;   // > 0: balanced column tiles dealt in units of tu tiles over gx = 256 workgroups
};

// One column tile of 16*nt columns per workgroup, kw waves splitting K inside
// it (interleaved step groups).  Chosen from sweeps on MI355X with packed
// operands and weights streamed from HBM, at the verify and draft shapes of
// the 7B-, 13B- and small configurations (M = 5 ... 320):
//   * 4 waves per workgroup throughout (8 or 16 were never better by more
//     than noise, often worse);
//   * QKV: 48-column tiles when that gives 192 ... 320 workgroups (7B width:
//     one per CU, 20 us against 25 us for 32-column tiles), else 16-column;
//   * 3-tile row blocks (33-48 rows, bf16): gate/up (SwiGLU) in balanced
//     mode, one workgroup per CU with the gate/up tile pairs dealt out
//     evenly (up to 3 pairs; 7B gate/up 38.4 -> 35.5 us): at these rows the
//     activation re-reads from L2 that a 32-column tile costs per weight
//     byte are what limit the shape.  The LM head gained nothing from it
//     (8 tiles per workgroup), nor the down projection from 64-column tiles
//     split 4 ways over K (the RMSNorm adding 4 partial sums cost more);
//   * other SwiGLU gate/up: 64-column tiles for 3-tile row blocks with < 512
//     column pairs (fewer activation re-reads), else 32-column;
//   * residual projections (O, down) with an RMSNorm after them (split_ok)
//     and one row block: K split over workgroups until there are ~256 of
//     them, 32-column tiles when every wave still gets >= 4 step groups
//     (64-column for a single 16-row tile: four times fewer activation
//     loads per weight load; 7B B = 1 verify pass 3.55 -> 3.20 ms, against
//     3.24 with 32 columns), else 16-column; the partial sums go through the
//     workspace to the RMSNorm, which adds them to the residual stream.
//     Without split_ok the output is added in place;
//   * LM head and other stores: 64-column tiles for 3-tile row blocks, else
//     32-column (4-tile row blocks take at most 32 columns);
//   * several 64-row blocks (B >= 32 verify, prefill): 32-column tiles.
// K is never split with a cross-workgroup reduction inside the GEMM: that
// needs a device-scope release per workgroup, which costs more than it saves.
GemmPlan plan_gemm(int M, int N, int K, size_t esz, int epi, bool split_ok = false) {
  GemmPlan g{};
  g.gz = (M + GEMM_MROWS - 1) / GEMM_MROWS;
  g.mt = g.gz > 1 ? 4 : (M + 15) / 16;
  g.ksplit = 1;
  g.kw = 4;
  g.tu = 0;
  const int groups = (int)(K * esz / 64) / GEMM_U;   // k-step groups of one wave step
  auto pick = [&](int nt) { return N % (16 * nt) == 0; };
  // balanced mode: tiles of tu over 256 workgroups, at most nt_max per workgroup
  auto balanced = [&](int tu, int nt_max) {
    if (g.gz != 1 || g.mt != 3 || esz != 2 || N % (16 * tu)) return 0;
    const int units = N / (16 * tu), most = (units + 255) / 256 * tu;
    if (units < 256 || most > nt_max) return 0;
    return most <= 4 ? 4 : nt_max;
  };
  if (g.gz > 1) {
    g.nt = pick(2) ? 2 : 1;
  } else if (epi == EPI_SWIGLU && balanced(2, 6)) {
    g.nt = balanced(2, 6);
    g.tu = 2;
  } else if (epi == EPI_SWIGLU) {
    g.nt = (g.mt == 3 && pick(4) && N / 32 < 512) ? 4 : 2;
  } else if (epi == EPI_QKV) {
    g.nt = (g.mt <= 3 && pick(3) && N / 48 >= 192 && N / 48 <= 320) ? 3 : 1;
  } else if (epi == EPI_RESID && split_ok) {
    auto splits = [&](int nt) {
      const int gx = N / (16 * nt);
      return std::min(std::min(SKINNY_MAX_KSPLIT, std::max(1, (256 + gx - 1) / gx)), std::max(1, groups / 4));
    };
    g.nt = 1;
    if (pick(2) && groups / splits(2) >= 4 * g.kw) g.nt = 2;
    if (g.mt == 1 && pick(4) && groups / splits(4) >= 4 * g.kw) g.nt = 4;
    g.ksplit = splits(g.nt);
  } else if (g.mt == 3 && pick(4)) {
    g.nt = 4;
  } else {
    g.nt = pick(2) ? 2 : 1;
  }
  g.gx = g.tu ? 256 : N / (16 * g.nt);
  const int gps = (groups + g.ksplit - 1) / g.ksplit;
  // the QKV epilogue assigns output rows by wave and needs exactly 4 waves
  if (epi != EPI_QKV) g.kw = std::max(1, std::min(g.kw, gps / 2));
  return g;
}

// Passes of several 64-row blocks (bf16) run the wide projections (QKV,
// gate/up, LM head: N >= 8192) on the row-tiled GEMM with 32 mf-row tiles,
// mf in 4..6 with the fewest padding rows (ties to the taller tile; 192-row
// tiles for prefill chunks), and 128-column tiles where they leave at least
// 128 workgroups, else 64-column.  Measured at the 7B B = 32
// and 13B B = 64 verify shapes (weights streamed from HBM): 13B gate/up at
// M = 320 109 us against 205 us on the skinny GEMM, LM head 108 against 245.
// The residual projections (N = d_model) from 128 to 640 rows run on
// 128 x 128 row tiles with K split when the caller can add partial sums
// (split_ok; *ks receives the split): 7B at M = 160: O 14.6-15.6 us and down
// 29.8-32.3 us, against about 22 and 64 on the skinny GEMM; 13B at M = 320:
// O 24.8 us, down 58.3, against 40.8 and 93.2 unsplit.  The split is chosen
// for the grid (column tiles x row tiles x splits): the largest split up to
// MAX_KSPLIT that keeps it within 512 workgroups (two per CU), or, when that
// grid would leave CUs with one workgroup and others with two (257 to 447
// workgroups), the largest that keeps it within 256 (one per CU), if that
// still splits.  Measured against the fixed four-way split (weights streamed
// from HBM): 13B down at M = 192 / 256 / 448 / 512: 44.4 / 53.9 / 77.1 / 88.5
// us against 58.6 / 70.4 / 107.8 / 125.2 (O: 20.6 / 24.5 / 30.8 / 36.8
// against 23.9 / 28.3 / 43.2 / 50.7); 7B down at M = 320 / 576: 40.6 / 59.5
// against 45.4 / 87.6.  Without a split they run on 128 x 64 tiles from 256
// to 640 rows and on the skinny GEMM below.  Returns false where the skinny
// GEMM runs.
int resid_ksplit(int M, int N) {
  const int tiles = (N / 128) * ((M + 127) / 128);
  int k512 = 0, k256 = 0;
  for (int k = 1; k <= MAX_KSPLIT; ++k) {
    if (tiles * k <= 512) k512 = k;
    if (tiles * k <= 256) k256 = k;
  }
  const int g = tiles * k512;
  return g > 256 && g < 448 && k256 >= 2 ? k256 : k512;
}

bool plan_rows(int M, int N, int K, int dtype, int epi, bool split_ok, int* mf, int* nf, int* ks) {
  *ks = 1;
  // a split range holds at least one stage (GEMM_CHUNK bytes of K)
  const int ks_res = std::min(resid_ksplit(M, N), K * 2 / GEMM_CHUNK);
  if (epi == EPI_RESID && dtype == SD_DTYPE_BF16 && split_ok && M >= 128 && M <= 640 && N % 128 == 0 &&
      ks_res >= 2) {
    *mf = 4;
    *nf = 4;
    *ks = ks_res;
    return true;
  }
  if (epi == EPI_RESID && dtype == SD_DTYPE_BF16 && M >= 256 && M <= 640 && N % 64 == 0) {
    *mf = 4;
    *nf = 2;
    return true;
  }
  if (dtype != SD_DTYPE_BF16 || M <= GEMM_MROWS || epi == EPI_PART || epi == EPI_RESID || N < 8192) return false;
  int best = 6, pad = 1 << 30;
  if (M <= 640) {
    for (int c : {4, 5, 6}) {
      const int rows = (M + 32 * c - 1) / (32 * c) * 32 * c;
      if (rows <= pad) {
        pad = rows;
        best = c;
      }
    }
  }
  *mf = best;
  // 128-column tiles while they leave at least 128 workgroups, else 64
  // (7B QKV at M = 160: 96 -> 192 workgroups, 60.8 -> 55.3 us in the sweep)
  const int mtiles = (M + 32 * best - 1) / (32 * best);
  *nf = N % 128 == 0 && mtiles * (N / 128) >= 128 ? 4 : 2;
  if (N % (32 * *nf)) return false;
  return true;
}

// Launch one projection.  part != null allows the K-split form for EPI_RESID:
// then *nsplit receives the number of partial sums written to part
// ([nsplit, M, ldo]) instead of being added to out, and the caller's RMSNorm
// adds them; otherwise *nsplit = 0.
int gemm(sd_ctx* ctx, const ModelRT& m, int epi, const void* A, const void* W, int M, int N, int K,
         float* out, int ldo, void* out_t, hipStream_t s, int prof_kind, int prof_kind2,
         const RopeParams* rope = nullptr, float* part = nullptr, int* nsplit = nullptr) {
  int mf = 0, nf = 0, rks = 1;
  const bool rows = plan_rows(M, N, K, m.c.dtype, epi, part != nullptr, &mf, &nf, &rks);
  GemmPlan g = plan_gemm(M, N, K, m.esz, epi, part != nullptr && !rows);
  if (!rows && !g.tu && N % (16 * g.nt)) return SD_EINVAL;
  const int ksplit = rows ? rks : g.ksplit;
  if (nsplit) *nsplit = 0;
  if (ksplit > 1) {
    epi = EPI_PART;
    out = part;
    if (nsplit) *nsplit = ksplit;
  }
  GemmParams p{};
  p.A = A;
  p.W = W;
  p.M = M;
  p.N = N;
  p.K = K;
  p.out = out;
  p.ldo = ldo;
  p.out_t = out_t;
  p.tile_unit = rows ? 0 : g.tu;
  p.ksplit = rows ? rks : 0;
  if (rope) p.rope = *rope;
  const double out_bytes = epi == EPI_SWIGLU ? (double)M * (N / 2) * m.esz
                           : epi == EPI_QKV  ? (double)M * (m.nq() * 4 + (N - m.nq()) * m.esz)
                           : epi == EPI_PART ? (double)M * N * 4 * ksplit
                                             : (double)M * N * 4 * (epi == EPI_RESID ? 2 : 1);
  const double bytes = (double)N * K * m.esz + (double)M * K * m.esz + out_bytes;
  ProfRec r1;
  prof_begin(ctx, s, r1, prof_kind, prof_kind2, bytes, true);
  if (rows)
    HIPCHK(launch_gemm_rows(epi, mf, nf, p, s, r1.a, r1.b));
  else
    HIPCHK(launch_gemm(m.c.dtype == SD_DTYPE_F32 ? 1 : 0, epi, g.nt, g.mt, g.kw, g.gx, g.ksplit, g.gz, p, s, r1.a,
                       r1.b));
  prof_end(ctx, s, r1);
  return SD_OK;
}

// One forward pass of a model over the rows set up by `rows` (or already in
// the lane for prefill).  lm_M > 0: final norm over rows r*lm_stride+lm_off
// and LM head into `logits` [lm_M, V].
int forward(sd_ctx* ctx, ModelRT& m, Lane& ln, RowsParams rows, int M, int nrb, const int32_t* rowblocks,
            int R, int attn_splits, int qmax, int lm_M, int lm_stride, int lm_off, float* logits,
            const int32_t* bt, bool verify, hipStream_t s) {
  const sd_model_cfg& c = m.c;
  const int dt = c.dtype == SD_DTYPE_F32 ? 1 : 0;
  const int d = c.d_model;
  rows.M = M;
  rows.embed = m.embed;
  rows.gain = m.attn_norm[0];
  rows.x = ln.x;
  rows.xn = ln.xn;
  rows.d = d;
  rows.V = c.vocab;
  rows.eps = c.rms_eps;
  rows.row_tok = ln.row_tok;
  rows.row_pos = ln.row_pos;
  rows.row_slot = ln.row_slot;
  rows.row_blk = ln.row_blk;
  rows.block_table = bt;
  rows.mbps = ctx->mbps;
  rows.row_bt = rowblocks ? nullptr : ln.row_bt;
  rows.state = ctx->state;
  rows.err = ctx->err;
  rows.n_slots = ctx->cfg.max_slots;
  HIPCHK(launch_rows_embed(dt, rows, s));
  const int pk_all = verify ? SD_PROF_GEMM_VERIFY_ALL : -1;
  int ns = 0;                   // K-split partial sums pending in ln.part
  for (int l = 0; l < c.n_layers; ++l) {
    RopeParams rp{};
    rp.q = ln.q;
    rp.kv = m.pool + (size_t)l * m.layer_bytes;
    rp.tab = m.rope_tab;
    rp.row_pos = ln.row_pos;
    rp.row_blk = ln.row_blk;
    rp.H = c.n_heads;
    rp.KV = c.n_kv_heads;
    rp.hd = c.head_dim;
    rp.nblk = m.n_blocks;
    int rc = gemm(ctx, m, EPI_QKV, ln.xn, m.wqkv[l], M, m.nqkv(), d, nullptr, 0, nullptr, s, pk_all, -1, &rp);
    if (rc) return rc;
    AttnParams ap{};
    ap.q = ln.q;
    ap.kv = rp.kv;
    ap.block_table = bt;
    ap.row_bt = rowblocks ? nullptr : ln.row_bt;
    ap.mbps = ctx->mbps;
    ap.nblk = m.n_blocks;
    ap.row_pos = ln.row_pos;
    ap.row_slot = ln.row_slot;
    ap.rowblocks = rowblocks;
    ap.R = R;
    ap.nrb = nrb;
    ap.H = c.n_heads;
    ap.KV = c.n_kv_heads;
    ap.hd = c.head_dim;
    // split the keys when the (row block, kv head) items leave more than half
    // of the 256 compute units idle, into at most as many splits as keep the
    // grid within one workgroup per CU (every split has keys to read: a
    // second round of workgroups would double the pass); the last split of
    // an item to finish merges them (16-bit caches), or a second kernel
    // does (fp32)
    int splits = attn_splits;
    const int items = nrb * c.n_kv_heads;
    if (items >= ATTN_SPLIT_BELOW) splits = 1;
    else if (splits > 1) splits = std::min(splits, std::max(1, 256 / items));
    const int kps = (ctx->cfg.max_ctx + 63) / 64 * 64;
    ap.splits = splits;
    ap.keys_per_split = splits > 1 ? std::max(ctx->keys_per_split, (kps / splits + 63) / 64 * 64) : kps;
    ap.splits = splits > 1 ? (kps + ap.keys_per_split - 1) / ap.keys_per_split : 1;
    ap.scale = 1.0f / sqrtf((float)c.head_dim);
    ap.out = ln.att;
    ap.part_o = ln.attn_o;
    ap.part_ml = ln.attn_ml;
    ap.cnt = ln.attn_cnt;
    ap.qmax = qmax;
    if (ap.splits > 1 && (items > ln.attn_items || (size_t)items * ap.splits * qmax * c.head_dim > ln.attn_o_cap))
      return SD_EINVAL;   // the lane holds the partials of its decode passes only
    ProfRec ra;
    prof_begin(ctx, s, ra, verify ? SD_PROF_ATTN_VERIFY : -1, -1, 0, true);
    HIPCHK(launch_attention(dt, ap, s, ra.a, ra.b));
    prof_end(ctx, s, ra);
    // residual projections may leave K-split partial sums in ln.part for the
    // RMSNorm after them to add
    const bool can_split = M <= ln.part_rows;
    rc = gemm(ctx, m, EPI_RESID, ln.att, m.wo[l], M, d, m.nq(), ln.x, d, nullptr, s, pk_all, -1, nullptr,
              can_split ? ln.part : nullptr, &ns);
    if (rc) return rc;
    NormParams np{ln.x, ns ? ln.part : nullptr, ns, m.ffn_norm[l], ln.xn, M, d, 1, 0, M, c.rms_eps};
    HIPCHK(launch_rmsnorm(dt, np, s));
    rc = gemm(ctx, m, EPI_SWIGLU, ln.xn, m.wgu[l], M, 2 * c.d_ffn, d, nullptr, 0, ln.hmid, s, pk_all,
              verify ? SD_PROF_GEMM_VERIFY_GATEUP : -1);
    if (rc) return rc;
    const bool norm_next = l + 1 < c.n_layers || lm_M > 0;
    rc = gemm(ctx, m, EPI_RESID, ln.hmid, m.wdown[l], M, d, c.d_ffn, ln.x, d, nullptr, s, pk_all, -1, nullptr,
              can_split && norm_next ? ln.part : nullptr, &ns);
    if (rc) return rc;
    if (l + 1 < c.n_layers) {
      NormParams nn{ln.x, ns ? ln.part : nullptr, ns, m.attn_norm[l + 1], ln.xn, M, d, 1, 0, M, c.rms_eps};
      HIPCHK(launch_rmsnorm(dt, nn, s));
    }
  }
  if (lm_M > 0) {
    NormParams fn{ln.x, ns ? ln.part : nullptr, ns, m.final_norm, ln.xn, lm_M, d, lm_stride, lm_off, M,
                  c.rms_eps};
    HIPCHK(launch_rmsnorm(dt, fn, s));
    int rc = gemm(ctx, m, EPI_STORE, ln.xn, m.lm_head, lm_M, c.vocab, d, logits, c.vocab, nullptr, s,
                  pk_all, -1);
    if (rc) return rc;
  }
  return SD_OK;
}

bool model_ptrs_ok(const sd_weights* w, int L) {
  if (!w || !w->embed || !w->lm_head || !w->final_norm) return false;
  if (!w->attn_norm || !w->wqkv || !w->wo || !w->ffn_norm || !w->wgu || !w->wdown) return false;
  for (int l = 0; l < L; ++l)
    if (!w->attn_norm[l] || !w->wqkv[l] || !w->wo[l] || !w->ffn_norm[l] || !w->wgu[l] || !w->wdown[l])
      return false;
  return true;
}

void load_model(ModelRT& m, const sd_model_cfg& c, const sd_weights* w, void* pool, int blocks) {
  m.c = c;
  m.esz = esize(c.dtype);
  m.embed = w->embed;
  m.lm_head = w->lm_head;
  m.final_norm = w->final_norm;
  m.attn_norm.assign(w->attn_norm, w->attn_norm + c.n_layers);
  m.wqkv.assign(w->wqkv, w->wqkv + c.n_layers);
  m.wo.assign(w->wo, w->wo + c.n_layers);
  m.ffn_norm.assign(w->ffn_norm, w->ffn_norm + c.n_layers);
  m.wgu.assign(w->wgu, w->wgu + c.n_layers);
  m.wdown.assign(w->wdown, w->wdown + c.n_layers);
  m.pool = (unsigned char*)pool;
  m.n_blocks = blocks;
  m.layer_bytes = pool_bytes(c, blocks) / c.n_layers;
}

bool batch_ok(sd_ctx* ctx, int B, const void* slots, int gamma) {
  return ctx && B >= 1 && B <= ctx->cfg.max_batch && slots && gamma >= 1 && gamma <= ctx->cfg.gamma_max;
}

// Order of the step calls of one batch (host-side, checked before anything
// is enqueued).  The batch is identified by its device slot list; a list
// seen with another B or gamma starts a new record.
//   draft i = 0      always allowed: starts (or restarts, discarding the
//                    uncommitted work) a step
//   draft i > 0      after draft i - 1 of the same step, not after verify
//   force i          after draft i, before draft i + 1 and verify
//   verify           after all gamma drafts of the step (may be repeated:
//                    it rewrites the same uncommitted positions)
//   commit           after verify; ends the step
// Acceptance (sd_accept_resample) needs no context and is not tracked: it
// only writes the caller's n_acc / out_tok, which the commit consumes.
Phase& phase_of(sd_ctx* ctx, const void* slots, int B, int gamma) {
  Phase& ph = ctx->phases[slots];
  if (ph.B != B || ph.gamma != gamma) ph = Phase{B, gamma, 0, false};
  return ph;
}

}  // namespace

// ---------------------------------------------------------------- static workspace

// The workspace of sd_init_static: a file-scope device array (each GPU the
// library runs on holds its own copy until the process ends).  Host code
// never uses the array's name as an address: its device address on each
// device comes from hipGetSymbolAddress, once per device, with that device
// current, and is kept in g_static_ptr.  A context holds its device's
// array from sd_init_static to sd_destroy; the array keeps the last
// context's contents and sd_init clears the parts that must start at zero.
constexpr size_t STATIC_WS_BYTES = (size_t)SD_STATIC_WORKSPACE_MB << 20;
constexpr int STATIC_MAX_DEV = 64;
__device__ __align__(256) unsigned char scratch[STATIC_WS_BYTES];
std::mutex g_static_mu;
void* g_static_ptr[STATIC_MAX_DEV] = {};
bool g_static_held[STATIC_MAX_DEV] = {};

// ============================================================== C ABI

extern "C" {

size_t sd_kv_pool_bytes(const sd_config* cfg, int draft) {
  if (!cfg_ok(cfg)) return 0;
  return draft ? pool_bytes(cfg->draft, cfg->kv_blocks_draft) : pool_bytes(cfg->target, cfg->kv_blocks_target);
}

size_t sd_workspace_bytes(const sd_config* cfg) {
  if (!cfg_ok(cfg)) return 0;
  return layout(cfg, nullptr);
}

int sd_init(const sd_config* cfg, const sd_weights* target, const sd_weights* draft, sd_ctx** out) {
  if (!out) return SD_EINVAL;
  *out = nullptr;
  if (!cfg_ok(cfg)) return SD_EINVAL;
  if (!model_ptrs_ok(target, cfg->target.n_layers) || !model_ptrs_ok(draft, cfg->draft.n_layers))
    return SD_EINVAL;
  if (!cfg->kv_pool_target || !cfg->kv_pool_draft || !cfg->workspace) return SD_EINVAL;
  if (cfg->workspace_bytes < layout(cfg, nullptr)) return SD_EINVAL;
  if (((uintptr_t)cfg->workspace | (uintptr_t)cfg->kv_pool_target | (uintptr_t)cfg->kv_pool_draft) & 255)
    return SD_EINVAL;
  sd_ctx* ctx = new (std::nothrow) sd_ctx();
  if (!ctx) return SD_EINVAL;
  ctx->cfg = *cfg;
  load_model(ctx->tgt, cfg->target, target, cfg->kv_pool_target, cfg->kv_blocks_target);
  load_model(ctx->dft, cfg->draft, draft, cfg->kv_pool_draft, cfg->kv_blocks_draft);
  layout(cfg, ctx);
  ctx->slots.resize(cfg->max_slots);
  for (int b = cfg->kv_blocks_target - 1; b >= 0; --b) ctx->free_t.push_back(b);
  for (int b = cfg->kv_blocks_draft - 1; b >= 0; --b) ctx->free_d.push_back(b);
  // device state: invalid slots, no errors; rotary tables
  // (kernels, synchronous here)
  hipStream_t s = nullptr;
  bool ok = launch_fill_i32((int32_t*)cfg->workspace, 0, layout(cfg, nullptr) / 4, s) == hipSuccess &&
            launch_rope_table(ctx->tgt.rope_tab, ctx->tgt.rope_pos, cfg->target.head_dim / 2,
                              cfg->target.rope_theta, s) == hipSuccess &&
            launch_rope_table(ctx->dft.rope_tab, ctx->dft.rope_pos, cfg->draft.head_dim / 2,
                              cfg->draft.rope_theta, s) == hipSuccess &&
            hipStreamSynchronize(s) == hipSuccess;
  if (!ok) {
    delete ctx;
    return SD_EHIP;
  }
  *out = ctx;
  return SD_OK;
}

int sd_init_static(const sd_config* cfg, const sd_weights* target, const sd_weights* draft, sd_ctx** out) {
  if (!out) return SD_EINVAL;
  *out = nullptr;
  if (!cfg_ok(cfg)) return SD_EINVAL;
  const size_t need = layout(cfg, nullptr);
  if (need > STATIC_WS_BYTES) {
    snprintf(g_last_error, sizeof(g_last_error),
             "sd_init_static: the configuration needs a %zu-byte workspace, the static one holds %zu", need,
             STATIC_WS_BYTES);
    return SD_EINVAL;
  }
  int dev = -1;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= STATIC_MAX_DEV) return SD_EINVAL;
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (g_static_held[dev]) return SD_ESTATE;    // another live context uses this device's array
  if (!g_static_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "hipGetSymbolAddress(scratch)",
                                               __LINE__);
    g_static_ptr[dev] = p;
  }
  sd_config c = *cfg;
  c.workspace = g_static_ptr[dev];
  c.workspace_bytes = STATIC_WS_BYTES;
  const int rc = sd_init(&c, target, draft, out);
  if (rc == SD_OK) {
    (*out)->static_dev = dev;
    g_static_held[dev] = true;
  }
  return rc;
}

int sd_prefill(sd_ctx* ctx, int B, const int32_t* slots, const int32_t* tokens, const int32_t* lens,
               const int32_t* max_new, void* stream) {
  if (!ctx || B < 1 || !slots || !tokens || !lens || !max_new) return SD_EINVAL;
  const sd_config& c = ctx->cfg;
  hipStream_t s = (hipStream_t)stream;
  std::vector<char> seen(c.max_slots, 0);
  size_t need_t = 0, need_d = 0;
  for (int k = 0; k < B; ++k) {
    if (slots[k] < 0 || slots[k] >= c.max_slots || seen[slots[k]]) return SD_EINVAL;
    seen[slots[k]] = 1;
    if (lens[k] < 1 || max_new[k] < 1) return SD_EINVAL;
    if ((long)lens[k] + max_new[k] + c.gamma_max > c.max_ctx) return SD_EINVAL;
    if (ctx->slots[slots[k]].active) return SD_ESTATE;
    const int nb = (lens[k] + max_new[k] + c.gamma_max + KV_BLOCK - 1) / KV_BLOCK;
    need_t += nb;
    need_d += nb;
  }
  size_t off = 0;
  for (int k = 0; k < B; ++k) {
    for (int i = 0; i < lens[k]; ++i)
      if (tokens[off + i] < 0 || tokens[off + i] >= c.target.vocab) return SD_EINVAL;
    off += lens[k];
  }
  if (need_t > ctx->free_t.size() || need_d > ctx->free_d.size()) return SD_ENOMEM;

  // allocate blocks and build the host images of state and block tables
  std::vector<int32_t> st(ST_N * B), bt(ctx->mbps * (size_t)B * 2, 0);
  off = 0;
  for (int k = 0; k < B; ++k) {
    Slot& sl = ctx->slots[slots[k]];
    const int nb = (lens[k] + max_new[k] + c.gamma_max + KV_BLOCK - 1) / KV_BLOCK;
    sl.tblocks.clear();
    sl.dblocks.clear();
    for (int i = 0; i < nb; ++i) {
      sl.tblocks.push_back(ctx->free_t.back());
      ctx->free_t.pop_back();
      sl.dblocks.push_back(ctx->free_d.back());
      ctx->free_d.pop_back();
      bt[(size_t)k * ctx->mbps + i] = sl.tblocks[i];
      bt[(size_t)(B + k) * ctx->mbps + i] = sl.dblocks[i];
    }
    st[k * ST_N + ST_LEN] = lens[k] - 1;
    st[k * ST_N + ST_X0] = tokens[off + lens[k] - 1];
    st[k * ST_N + ST_PEND] = -1;
    st[k * ST_N + ST_CAP] = nb * KV_BLOCK;
    off += lens[k];
  }
  auto undo = [&]() {
    for (int k = 0; k < B; ++k) {
      Slot& sl = ctx->slots[slots[k]];
      for (int b : sl.tblocks) ctx->free_t.push_back(b);
      for (int b : sl.dblocks) ctx->free_d.push_back(b);
      sl.tblocks.clear();
      sl.dblocks.clear();
    }
  };
  for (int k = 0; k < B; ++k) {
    if (hipMemcpyAsync(ctx->state + (size_t)slots[k] * ST_N, &st[k * ST_N], sizeof(int32_t) * ST_N,
                       hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(ctx->bt_t + (size_t)slots[k] * ctx->mbps, &bt[(size_t)k * ctx->mbps],
                       sizeof(int32_t) * ctx->mbps, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(ctx->bt_d + (size_t)slots[k] * ctx->mbps, &bt[(size_t)(B + k) * ctx->mbps],
                       sizeof(int32_t) * ctx->mbps, hipMemcpyHostToDevice, s) != hipSuccess) {
      undo();
      return hip_fail(hipGetLastError(), "prefill state upload", __LINE__);
    }
  }

  // rows: prompt[:-1] of every task, in chunks of prefill_rows
  struct RowRec { int32_t tok, pos, slot; };
  std::vector<RowRec> all;
  off = 0;
  for (int k = 0; k < B; ++k) {
    for (int i = 0; i + 1 < lens[k]; ++i) all.push_back({tokens[off + i], i, slots[k]});
    off += lens[k];
  }
  Lane& ln = ctx->lv;
  // host staging kept alive until the final synchronize; a deque keeps references stable
  std::deque<std::vector<int32_t>> keep;
  int rc = SD_OK;
  for (size_t c0 = 0; c0 < all.size() && rc == SD_OK; c0 += c.prefill_rows) {
    const int M = (int)std::min(all.size() - c0, (size_t)c.prefill_rows);
    keep.emplace_back(3 * (size_t)M);
    std::vector<int32_t>& rows = keep.back();
    for (int r = 0; r < M; ++r) {
      rows[r] = all[c0 + r].tok;
      rows[M + r] = all[c0 + r].pos;
      rows[2 * M + r] = all[c0 + r].slot;
    }
    if (hipMemcpyAsync(ln.row_tok, rows.data(), sizeof(int32_t) * M, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(ln.row_pos, rows.data() + M, sizeof(int32_t) * M, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(ln.row_slot, rows.data() + 2 * M, sizeof(int32_t) * M, hipMemcpyHostToDevice, s) !=
            hipSuccess) {
      rc = hip_fail(hipGetLastError(), "prefill row upload", __LINE__);
      break;
    }
    for (int which = 0; which < 2 && rc == SD_OK; ++which) {
      ModelRT& m = which == 0 ? ctx->tgt : ctx->dft;
      const int qb = prefill_qb(m.c);
      keep.emplace_back();
      std::vector<int32_t>& rbv = keep.back();
      for (int r = 0; r < M;) {
        int e = r + 1;
        while (e < M && e - r < qb && rows[2 * M + e] == rows[2 * M + r]) ++e;
        rbv.push_back(r);
        rbv.push_back(e - r);
        r = e;
      }
      const int nrb = (int)rbv.size() / 2;
      if (nrb > ln.rb_cap) { rc = SD_EINVAL; break; }
      // each model's row blocks go to their own half of the row-block buffer region in turn;
      // the copy is ordered after the previous model's kernels on the same stream
      if (hipMemcpyAsync(ln.rowblocks, rbv.data(), sizeof(int32_t) * rbv.size(), hipMemcpyHostToDevice, s) !=
          hipSuccess) {
        rc = hip_fail(hipGetLastError(), "prefill row-block upload", __LINE__);
        break;
      }
      RowsParams rp{};
      rp.mode = ROWS_PREFILL;
      rc = forward(ctx, m, ln, rp, M, nrb, ln.rowblocks, 0, 1, qb * m.G(), 0, 1, 0, nullptr,
                   which == 0 ? ctx->bt_t : ctx->bt_d, false, s);
    }
  }
  {
    const hipError_t e = hipStreamSynchronize(s);
    if (e != hipSuccess) rc = hip_fail(e, "prefill synchronize", __LINE__);
  }
  if (rc != SD_OK) {
    undo();
    return rc;
  }
  for (int k = 0; k < B; ++k) ctx->slots[slots[k]].active = true;
  return SD_OK;
}

int sd_release(sd_ctx* ctx, int slot) {
  if (!ctx || slot < 0 || slot >= ctx->cfg.max_slots) return SD_EINVAL;
  Slot& sl = ctx->slots[slot];
  if (!sl.active) return SD_ESTATE;
  // capacity 0 on the device: a later pass that still names the slot skips
  // (and flags) every KV write instead of writing into blocks that another
  // task may be given next
  const int32_t zero = 0;
  HIPCHK(hipMemcpy(ctx->state + (size_t)slot * ST_N + ST_CAP, &zero, sizeof(int32_t), hipMemcpyHostToDevice));
  for (int b : sl.tblocks) ctx->free_t.push_back(b);
  for (int b : sl.dblocks) ctx->free_d.push_back(b);
  sl.tblocks.clear();
  sl.dblocks.clear();
  sl.active = false;
  return SD_OK;
}

int sd_draft_step(sd_ctx* ctx, int B, const int32_t* slots, int gamma, int i, const uint32_t* u,
                  int32_t* draft_tok, float* q, void* stream) {
  if (!batch_ok(ctx, B, slots, gamma) || i < 0 || i >= gamma || !u || !draft_tok || !q) return SD_EINVAL;
  Phase& ph = phase_of(ctx, slots, B, gamma);
  if (i > 0 && (ph.drafted != i || ph.verified)) return SD_ESTATE;
  hipStream_t s = (hipStream_t)stream;
  ModelRT& m = ctx->dft;
  Lane& ln = ctx->ld;
  const bool first = i == 0;
  const int R = first ? 2 : 1;
  const int M = B * R;
  RowsParams rp{};
  rp.mode = first ? ROWS_DRAFT_FIRST : ROWS_DRAFT_NEXT;
  rp.B = B;
  rp.gamma = gamma;
  rp.step_i = i;
  rp.slots = slots;
  rp.draft_tok = draft_tok;
  ProfRec pr;
  prof_begin(ctx, s, pr, SD_PROF_DRAFT, -1, 0, false);
  int rc = forward(ctx, m, ln, rp, M, B, nullptr, R, ctx->attn_splits, R * m.G(), B, R, R - 1, ln.logits,
                   ctx->bt_d, false, s);
  if (rc) return rc;
  DraftSampleParams dp{};
  dp.z = ln.logits;
  dp.q = q;
  dp.draft_tok = draft_tok;
  dp.u = u;
  dp.B = B;
  dp.V = m.c.vocab;
  dp.gamma = gamma;
  dp.i = i;
  dp.inv_tau = 1.0f / ctx->cfg.temperature;
  dp.greedy = ctx->cfg.greedy;
  HIPCHK(launch_draft_sample(dp, s));
  prof_end(ctx, s, pr);
  ph.drafted = i + 1;
  ph.verified = false;
  return SD_OK;
}

int sd_verify(sd_ctx* ctx, int B, const int32_t* slots, int gamma, const int32_t* draft_tok, float* p,
              float* logits, void* stream) {
  if (!batch_ok(ctx, B, slots, gamma) || !draft_tok || !p) return SD_EINVAL;
  Phase& ph = phase_of(ctx, slots, B, gamma);
  if (ph.drafted != gamma) return SD_ESTATE;
  hipStream_t s = (hipStream_t)stream;
  ModelRT& m = ctx->tgt;
  Lane& ln = ctx->lv;
  const int R = gamma + 1;
  const int M = B * R;
  RowsParams rp{};
  rp.mode = ROWS_VERIFY;
  rp.B = B;
  rp.gamma = gamma;
  rp.slots = slots;
  rp.draft_tok = draft_tok;
  float* z = logits ? logits : p;
  ProfRec pr;
  prof_begin(ctx, s, pr, SD_PROF_VERIFY, -1, 0, false);
  int rc = forward(ctx, m, ln, rp, M, B, nullptr, R, ctx->attn_splits, R * m.G(), M, 1, 0, z, ctx->bt_t,
                   true, s);
  if (rc) return rc;
  SoftmaxParams sp{z, p, M, m.c.vocab, 1.0f / ctx->cfg.temperature, ctx->cfg.greedy};
  HIPCHK(launch_softmax(sp, s));
  prof_end(ctx, s, pr);
  ph.verified = true;
  return SD_OK;
}

int sd_accept_resample(int B, int gamma, int vocab, int greedy, const int32_t* draft_tok, const float* q,
                       const float* p, const uint32_t* u, int32_t* n_acc, int32_t* out_tok, void* stream) {
  if (B < 1 || gamma < 1 || gamma > 64 || vocab < 4 || vocab > 32768 || !draft_tok || !q || !p || !u || !n_acc ||
      !out_tok)
    return SD_EINVAL;
  // rows of q and p are read as float4: 16-byte aligned starts and whole float4s
  if ((vocab & 3) || (((uintptr_t)q | (uintptr_t)p) & 15)) return SD_EINVAL;
  AcceptParams ap{};
  ap.B = B;
  ap.gamma = gamma;
  ap.V = vocab;
  ap.greedy = greedy ? 1 : 0;
  ap.draft_tok = draft_tok;
  ap.q = q;
  ap.p = p;
  ap.u = u;
  ap.n_acc = n_acc;
  ap.out_tok = out_tok;
  ap.err = nullptr;
  HIPCHK(launch_accept(ap, (hipStream_t)stream));
  return SD_OK;
}

int sd_kv_commit(sd_ctx* ctx, int B, const int32_t* slots, int gamma, const int32_t* n_acc,
                 const int32_t* out_tok, void* stream) {
  if (!batch_ok(ctx, B, slots, gamma) || !n_acc || !out_tok) return SD_EINVAL;
  Phase& ph = phase_of(ctx, slots, B, gamma);
  if (!ph.verified) return SD_ESTATE;
  CommitParams cp{B, gamma, ctx->cfg.max_slots, slots, n_acc, out_tok, ctx->state, ctx->err};
  HIPCHK(launch_commit(cp, (hipStream_t)stream));
  ph.drafted = 0;
  ph.verified = false;
  return SD_OK;
}

int sd_force_draft(sd_ctx* ctx, int B, const int32_t* slots, int gamma, int i, const int32_t* cont, int cont_len,
                   const uint32_t* u, double alpha, int32_t* draft_tok, void* stream) {
  if (!batch_ok(ctx, B, slots, gamma) || i < 0 || i >= gamma || !cont || cont_len < 1 || !u || !draft_tok ||
      !(alpha >= 0.0 && alpha <= 1.0))
    return SD_EINVAL;
  if (!ctx->cfg.greedy) return SD_ESTATE;   // the draft uniforms are in use when sampling
  const Phase& ph = phase_of(ctx, slots, B, gamma);
  if (ph.drafted != i + 1 || ph.verified) return SD_ESTATE;
  ForceParams fp{};
  fp.B = B;
  fp.gamma = gamma;
  fp.i = i;
  fp.n_slots = ctx->cfg.max_slots;
  fp.slots = slots;
  fp.state = ctx->state;
  fp.cont = cont;
  fp.cont_len = cont_len;
  fp.u = u;
  fp.threshold = (uint64_t)std::llround(alpha * 4294967296.0);
  fp.draft_tok = draft_tok;
  HIPCHK(launch_force_draft(fp, (hipStream_t)stream));
  return SD_OK;
}

int sd_slot_state(sd_ctx* ctx, int B, const int32_t* slots, int32_t* out, void* stream) {
  if (!ctx || B < 1 || !slots || !out) return SD_EINVAL;
  // gather via the commit-free path: one tiny copy per row on the stream
  hipStream_t s = (hipStream_t)stream;
  std::vector<int32_t> hs(B);
  HIPCHK(hipMemcpyAsync(hs.data(), slots, sizeof(int32_t) * B, hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  for (int b = 0; b < B; ++b) {
    if (hs[b] < 0 || hs[b] >= ctx->cfg.max_slots) return SD_EINVAL;
    HIPCHK(hipMemcpyAsync(out + (size_t)b * ST_N, ctx->state + (size_t)hs[b] * ST_N, sizeof(int32_t) * ST_N,
                          hipMemcpyDeviceToDevice, s));
  }
  return SD_OK;
}

int sd_check(sd_ctx* ctx, void* stream, int32_t* flags_out) {
  if (!ctx) return SD_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  int32_t f = 0;
  HIPCHK(hipMemcpyAsync(&f, ctx->err, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  HIPCHK(hipStreamSynchronize(s));
  HIPCHK(launch_fill_i32(ctx->err, 0, 1, s));
  HIPCHK(hipStreamSynchronize(s));
  if (flags_out) *flags_out = f;
  return SD_OK;
}

int sd_profile(sd_ctx* ctx, int enable) {
  if (!ctx) return SD_EINVAL;
  ctx->prof = enable != 0;
  return SD_OK;
}

int sd_profile_read(sd_ctx* ctx, int kind, int64_t* count, double* ms, double* bytes) {
  if (!ctx || kind < 0 || kind >= SD_PROF_N) return SD_EINVAL;
  int64_t n = 0;
  double t = 0, by = 0;
  std::vector<ProfRec> keep;
  for (ProfRec& r : ctx->recs) {
    if (!(r.mask & (1u << kind))) {
      keep.push_back(r);
      continue;
    }
    float e = 0.f;
    if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&e, r.a, r.b) == hipSuccess) {
      ++n;
      t += e;
      by += r.bytes;
    }
    r.mask &= ~(1u << kind);
    if (r.mask) {
      keep.push_back(r);
    } else {
      hipEventDestroy(r.a);
      hipEventDestroy(r.b);
    }
  }
  ctx->recs.swap(keep);
  if (count) *count = n;
  if (ms) *ms = t;
  if (bytes) *bytes = by;
  return SD_OK;
}

void sd_destroy(sd_ctx* ctx) {
  if (!ctx) return;
  if (ctx->static_dev >= 0) {
    std::lock_guard<std::mutex> lock(g_static_mu);
    g_static_held[ctx->static_dev] = false;
  }
  for (ProfRec& r : ctx->recs) {
    hipEventDestroy(r.a);
    hipEventDestroy(r.b);
  }
  delete ctx;
}

int sd_pack_linear(const void* src, void* dst, int N, int K, int dtype, void* stream) {
  if (!src || !dst || N < 16 || K < 1 || (dtype != SD_DTYPE_BF16 && dtype != SD_DTYPE_F32)) return SD_EINVAL;
  if (N % 16 || ((size_t)K * esize(dtype)) % GEMM_CHUNK) return SD_EINVAL;
  HIPCHK(launch_pack_linear(dtype == SD_DTYPE_F32 ? 1 : 0, src, dst, N, K, (hipStream_t)stream));
  return SD_OK;
}

const char* sd_last_error(void) { return g_last_error; }

const char* sd_strerror(int code) {
  switch (code) {
    case SD_OK: return "ok";
    case SD_EINVAL: return "invalid argument or configuration";
    case SD_ENOMEM: return "KV block pool exhausted";
    case SD_ESTATE: return "call not allowed in the slot's current state";
    case SD_EHIP: return "HIP runtime error";
    default: return "unknown error";
  }
}

}  // extern "C"
