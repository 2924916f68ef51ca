// Internal declarations shared by the libsd kernels and host runtime.
// Written for gfx950 (CDNA4): 64-lane wavefronts, bf16 MFMA, 160 KB LDS/CU.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stddef.h>
#include <stdint.h>

namespace sd {

// ---------------------------------------------------------------- numerics

typedef uint16_t bf16_t;  // raw bf16 bit pattern in memory
// IEEE binary16.  A bf16 model is computed with fp16 operands: its packed
// weight matrices are converted to fp16 once (sd_pack_linear; exact for
// every bf16 value of magnitude >= 2^-14, smaller ones round to fp16's
// subnormal grid of 2^-24), and its matrix-product inputs and KV cache are
// rounded to fp16 (11 significant bits against bf16's 8), at the same memory
// cost and matrix-instruction rate.  Embedding rows and norm gains stay bf16.
typedef _Float16 f16_t;

__device__ __forceinline__ float bf2f(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }

// round to nearest even (inputs are finite)
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// fp16 bit pattern of f, rounded to nearest even (v_cvt_f16_f32)
__device__ __forceinline__ uint16_t f2h(float f) { return __builtin_bit_cast(uint16_t, (f16_t)f); }
__device__ __forceinline__ float h2f(uint16_t h) { return (float)__builtin_bit_cast(f16_t, h); }

// MFMA-tile layout of a matrix-product operand X[R, K] (weights R = N,
// activations R = M rows padded to 16): a k-step is 64 bytes of a row
// (32 bf16 or 16 fp32); tile (r / 16, k-step s) is 1 KB holding, for lane
// l = 16 * (k-group) + r % 16, the 16 bytes of row r, k-group (k % step) /
// (elements per 16 bytes).  Every 16-byte lane load of an operand fragment
// is then part of one contiguous 1 KB block.
// Element offset of the K (kv = 0) or V (kv = 1) tile of (kv head h, block b)
// in one layer's pool.  The pool is head-major, [kv heads][blocks][K|V][16 x hd],
// so the blocks of one task and head, allocated in order, form one run.
__host__ __device__ __forceinline__ size_t kv_tile_off(int h, int b, int kv, int nblk, int hd) {
  return (((size_t)h * nblk + b) * 2 + kv) * 16 * (size_t)hd;
}

// Element offset of key (token t, dim d) inside one 16-token block of one kv
// head.  bf16 caches use the layout of the attention's matrix instruction:
// for each of the hd/32 k-steps s, a 1 KB run of 64 16-byte units, unit
// 16 g + t holding dims g (hd/4) + 8 s .. + 8 (g < 4), so every key load of
// a wave is contiguous.  fp32 caches are token-major ([16][hd]).
template <typename T> __host__ __device__ __forceinline__ int kv_key_off(int t, int d, int hd) {
  if constexpr (sizeof(T) == 2) {
    const int q = hd / 4, g = d / q, s = (d % q) / 8;
    return ((s * 4 + g) * 16 + t) * 8 + (d & 7);
  } else {
    return t * hd + d;
  }
}

// Element offset of value (token t, dim d) inside one 16-token V tile.  bf16
// caches: for each 32-dim group the 16 x 32 slice is ordered
// [dim % 16][t / 4][(d / 16) % 2][t % 4], so that the 4 consecutive tokens of
// two dims 16 apart are one 16-byte unit and a wave load of 64 such units is
// one contiguous 1 KB.  fp32 caches: transposed, [hd][16].
template <typename T> __host__ __device__ __forceinline__ int kv_val_off(int t, int d, int hd) {
  if constexpr (sizeof(T) == 2) {
    return ((((d >> 5) * 16 + (d & 15)) * 4 + (t >> 2)) * 2 + ((d >> 4) & 1)) * 4 + (t & 3);
  } else {
    return d * 16 + t;
  }
}

template <typename T> struct Tile {
  static constexpr int EPL = 16 / (int)sizeof(T);   // elements per lane unit
  static constexpr int EPK = 4 * EPL;                // elements per k-step
  __host__ __device__ __forceinline__ static size_t off(int r, int k, int K) {
    const int ks = K / EPK;
    const int lane = ((k % EPK) / EPL) * 16 + (r & 15);
    return (((size_t)(r >> 4) * ks + k / EPK) * 64 + lane) * EPL + (k % EPL);
  }
};

template <typename T> struct Store;
template <> struct Store<bf16_t> {
  __device__ __forceinline__ static float load(const bf16_t* p, size_t i) { return bf2f(p[i]); }
  __device__ __forceinline__ static void store(bf16_t* p, size_t i, float v) { p[i] = f2bf(v); }
};
template <> struct Store<f16_t> {
  __device__ __forceinline__ static float load(const f16_t* p, size_t i) { return (float)p[i]; }
  __device__ __forceinline__ static void store(f16_t* p, size_t i, float v) { p[i] = (f16_t)v; }
};
template <> struct Store<float> {
  __device__ __forceinline__ static float load(const float* p, size_t i) { return p[i]; }
  __device__ __forceinline__ static void store(float* p, size_t i, float v) { p[i] = v; }
};

// ---------------------------------------------------------------- row modes

enum RowMode { ROWS_PREFILL = 0, ROWS_VERIFY = 1, ROWS_DRAFT_FIRST = 2, ROWS_DRAFT_NEXT = 3 };

// per-slot device state, int32 x 4
enum { ST_LEN = 0, ST_X0 = 1, ST_PEND = 2, ST_CAP = 3, ST_N = 4 };

enum { ERR_KV_OVERFLOW = 1, ERR_BAD_TOKEN = 2, ERR_BAD_ACCEPT = 4 };

// ---------------------------------------------------------------- kernel params

struct RowsParams {
  int mode, B, gamma, step_i, M;
  const int32_t* slots;      // [B] (not prefill)
  const int32_t* draft_tok;  // [B, gamma]
  int32_t* state;            // [slots, ST_N]
  int32_t* row_tok;          // [M]
  int32_t* row_pos;          // [M]; -1 = inactive row
  int32_t* row_slot;         // [M]
  int32_t* row_blk;          // [M] KV block the row's K/V go to; -1 = none (inactive, or over capacity)
  const int32_t* block_table;  // [slots, mbps] of the model run over the rows
  int mbps;
  int32_t* row_bt;           // null (prefill), or [B, mbps]: task b's block-table row, copied for the
                             // attention of the pass (row block b), which then needs no slot lookup
  const void* embed;         // [V, d]
  const void* gain;          // [d]
  float* x;                  // [M, d]
  void* xn;                  // [M, d] in the MFMA-tile layout
  int d, V, n_slots;
  float eps;
  int32_t* err;
};

struct NormParams {
  float* x;           // [rows_in, d] residual stream
  const float* part;  // null, or [nsplit, rows_in, d] partial sums added to x first (in split order)
  int nsplit;
  const void* gain;   // [d]
  void* xn;           // [M, d] in the MFMA-tile layout
  int M, d, src_stride, src_off;  // output row r reads input row r*src_stride + src_off
  int rows_in;
  float eps;
};


// Rotary embedding (rotate-half pairs (i, i + hd/2), angle pos * theta^(-2i/hd))
// and KV append, done by the epilogue of the QKV projection.  Query and key
// rows of the fused weight are in pair order (see sd_weights), so the two
// halves of a pair meet in one lane.
struct RopeParams {
  float* q;                    // [M, H hd] fp32, rotary applied
  void* kv;                    // layer base of the pool (kv_tile_off), V tiles as [hd][16]
  const float2* tab;           // [positions, hd/2] (cos, sin), fp64 angles rounded to fp32
  const int32_t* row_pos;      // [M]; -1 = inactive row
  const int32_t* row_blk;      // [M] KV block of the row's position; -1 = not written
  int H, KV, hd, nblk;         // nblk: blocks in the pool
};

struct GemmParams {
  const void* A;      // [M, K] activations, MFMA-tile layout (rows padded to the M block)
  const void* W;      // [N, K] weights, MFMA-tile layout
  int M, N, K;
  float* out;         // STORE: out[m * ldo + n]; RESID: out[m * ldo + n] += acc
  int ldo;
  void* out_t;        // SWIGLU: out_t[M, N/2] in the MFMA-tile layout
  RopeParams rope;    // QKV: rotary embedding of q and k, K/V appended to the cache
  int mblocks;        // > 1: 1-D grid of (column tile, M block) pairs, XCD-aware (see gemm.hip)
  int tile_unit;      // > 0: balanced column tiles, dealt in units of tile_unit tiles (see gemm.hip)
  int ksplit;         // row-tiled GEMM: K in ksplit ranges; with PART, range r's partial sums go to
                      // out[(r M + m) ldo + n] (0 or 1: no split)
};

struct AttnParams {
  const float* q;            // [M, H hd] (rotary applied)
  const void* kv;            // layer base of the pool (kv_tile_off)
  const int32_t* block_table;
  const int32_t* row_bt;     // null, or [nrb, mbps]: row block rb's block-table row (decode passes)
  int mbps, nblk;            // block-table width, blocks in the pool
  const int32_t* row_pos;
  const int32_t* row_slot;
  const int32_t* rowblocks;  // [nrb, 2] = (row0, nrows), or null: rowblock i = rows [i*R, i*R+R)
  int R, nrb, H, KV, hd;
  int keys_per_split, splits;
  float scale;
  void* out;                 // [M, H hd] model dtype, MFMA-tile layout
  float* part_o;             // [nrb*KV, splits, Qmax, hd]
  float* part_ml;            // [nrb*KV, splits, Qmax, 2]
  int qmax;                  // max query vectors per (rowblock, kv head)
  int* cnt;                  // [nrb*KV] arrivals of an item's key splits (16-bit caches; zero between launches)
};

struct SoftmaxParams {
  const float* z;   // [M, V]
  float* p;         // [M, V] (may alias z)
  int M, V;
  float inv_tau;
  int greedy;
};

struct DraftSampleParams {
  const float* z;          // [B, V] draft logits
  float* q;                // [B, gamma, V]
  int32_t* draft_tok;      // [B, gamma]
  const uint32_t* u;       // [B, 2 gamma + 1]
  int B, V, gamma, i;
  float inv_tau;
  int greedy;
};

struct AcceptParams {
  int B, gamma, V, greedy;
  const int32_t* draft_tok;  // [B, gamma]
  const float* q;            // [B, gamma, V]
  const float* p;            // [B, gamma+1, V]
  const uint32_t* u;         // [B, 2 gamma + 1]
  int32_t* n_acc;            // [B]
  int32_t* out_tok;          // [B, gamma+1]
  int32_t* err;              // may be null
};

struct CommitParams {
  int B, gamma, n_slots;
  const int32_t* slots;
  const int32_t* n_acc;
  const int32_t* out_tok;
  int32_t* state;
  int32_t* err;
};

struct ForceParams {
  int B, gamma, i, n_slots;
  const int32_t* slots;
  const int32_t* state;
  const int32_t* cont;     // [B, cont_len] token at each absolute position
  int cont_len;
  const uint32_t* u;       // [B, 2 gamma + 1]; slot i decides
  uint64_t threshold;      // forced iff u < threshold (alpha * 2^32)
  int32_t* draft_tok;      // [B, gamma]
};

// PART: K split over gridDim.y workgroups; split y stores its partial sum to
// out[(y * M + m) * ldo + n], the residual add happens in the next RMSNorm
enum GemmEpi { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_QKV = 3, EPI_PART = 4 };

// ---------------------------------------------------------------- launchers
// dtype: 0 bf16, 1 fp32 (same values as SD_DTYPE_*)

hipError_t launch_rows_embed(int dtype, const RowsParams& p, hipStream_t s);
hipError_t launch_rmsnorm(int dtype, const NormParams& p, hipStream_t s);
// Kernel launch; with a start event the launch carries (start, stop) events
// that the dispatch itself timestamps (kernel begin / end), as profilers do.
template <typename K, typename... A>
inline void launch_k(K kern, dim3 grid, dim3 block, uint32_t shm, hipStream_t s, hipEvent_t e0, hipEvent_t e1,
                     A... args) {
  if (e0 || e1) hipExtLaunchKernelGGL(kern, grid, block, shm, s, e0, e1, 0, args...);
  else hipLaunchKernelGGL(kern, grid, block, shm, s, args...);
}

// Row-tiled bf16 GEMM for passes of several 64-row blocks: 32 mf x 32 nf
// output tiles, mf in {4, 5, 6, 8}, nf in {2, 4}; epi: STORE, RESID, SWIGLU
// or QKV (no K split).  N must be a multiple of 32 nf.
hipError_t launch_gemm_rows(int epi, int mf, int nf, const GemmParams& p, hipStream_t s, hipEvent_t e0 = nullptr,
                            hipEvent_t e1 = nullptr);
// Host-side check of a skinny GEMM launch (launch_gemm rejects what fails it)
bool gemm_config_ok(int dtype, int epi, int nt, int mt, int kw, int grid_x, int ksplit, int grid_z,
                    const GemmParams& p);
hipError_t launch_gemm(int dtype, int epi, int nt, int mt, int kw, int grid_x, int ksplit, int grid_z,
                       const GemmParams& p, hipStream_t s, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// tab[pos * half + i] = (cos, sin) of pos * theta^(-i/half), pos < n_pos, i < half
hipError_t launch_rope_table(float2* tab, int n_pos, int half, double theta, hipStream_t s);
hipError_t launch_attention(int dtype, const AttnParams& p, hipStream_t s, hipEvent_t e0 = nullptr,
                            hipEvent_t e1 = nullptr);
hipError_t launch_softmax(const SoftmaxParams& p, hipStream_t s);
hipError_t launch_draft_sample(const DraftSampleParams& p, hipStream_t s);
hipError_t launch_accept(const AcceptParams& p, hipStream_t s);
hipError_t launch_commit(const CommitParams& p, hipStream_t s);
hipError_t launch_force_draft(const ForceParams& p, hipStream_t s);
hipError_t launch_fill_i32(int32_t* p, int32_t v, size_t n, hipStream_t s);
hipError_t launch_pack_linear(int dtype, const void* src, void* dst, int N, int K, hipStream_t s);

// GEMM geometry (shared by host planning and the kernel)
constexpr int GEMM_U = 2;              // 64-byte k-steps per wave step of the GEMM
constexpr int GEMM_CHUNK = 64 * GEMM_U; // K dims must be a multiple of this many bytes
constexpr int GEMM_MROWS = 64;         // rows per M block (4 MFMA row tiles)

// attention geometry
constexpr int ATTN_KEYS = 64;          // keys per LDS chunk
constexpr int ATTN_QMAX = 64;          // max query vectors per workgroup
constexpr int ATTN_BT_CAP = 2048;      // KV blocks of one key range staged in LDS (32768 positions)
constexpr int ATTN_MAX_SPLITS = 12;    // key splits per item the matrix kernel merges itself
constexpr int ATTN_SPLIT_BELOW = 128;  // decode passes with fewer (row block, kv head) items split the keys
constexpr int MAX_CTX = ATTN_BT_CAP * 16;   // positions a slot may reach

}  // namespace sd
