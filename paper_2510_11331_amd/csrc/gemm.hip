// Skinny GEMM for the projections of the draft and verify passes:
// out[M, N] = A[M, K] * W[N, K]^T with M = rows of the pass (a few to a few
// dozen in decoding, up to 64 per block in prefill), fp32 accumulation.
//
// The pass is bound by streaming W from HBM, so the kernel is organised
// around that stream:
//   * W and A are stored in the MFMA-tile layout (W packed once by
//     sd_pack_linear, A written that way by the producing kernels), so every
//     fragment load of a wave is one contiguous 1 KB block;
//   * a workgroup owns one column tile (16*NT output columns = 16*NT rows
//     of W; NT in {1, 2, 3, 4}, wider tiles re-read the activations less
//     often) and splits K over its KW waves (up to 4), interleaved in
//     groups of U k-steps; each wave streams its share of the tile straight
//     into registers, one step group ahead of the MFMAs;
//   * or, in balanced mode (one M block), the grid is one workgroup per CU
//     and the N / 16 column tiles are dealt out evenly, up to NT = 6 per
//     workgroup: at 33-48 rows the activation re-reads from L2 then cost a
//     third as much, and no CU holds more work than another by more than
//     one deal unit;
//   * the matching activation fragments are loaded the same way (they are
//     small and stay in L2), so the main loop has no LDS traffic and no
//     barriers; it has no branches either (padding rows and groups past a
//     wave's share are out-of-range buffer loads that return zero), so
//     vmcnt only ever waits for the older step group;
//   * bf16 models (operands in fp16, see f16_t): one v_mfma_f32_16x16x32_f16
//     per 16-byte unit; fp32: four v_mfma_f32_16x16x4_f32;
//   * the KW partial tiles are added in wave order through LDS in one round
//     (deterministic); K is never split across workgroups (a cross-workgroup
//     reduction needs a device-scope release per workgroup, which costs more
//     than it recovers at these sizes);
//   * for projections with few column tiles, K may also be split over
//     gridDim.y workgroups that store fp32 partial sums; the RMSNorm that
//     follows adds them to the residual stream in split order (no
//     cross-workgroup synchronisation, deterministic);
//   * epilogues: store fp32, add into the fp32 residual stream, SwiGLU over
//     interleaved gate/up rows (written in the model dtype), or, for the QKV
//     projection, the rotary embedding of q and k (rows in rotary pair
//     order: the two halves of a pair sit 8 columns apart in one tile and
//     meet through a lane exchange) with q stored in fp32 and k, v appended
//     to the paged KV cache.
#include "sd_internal.h"

#include <algorithm>
#include <type_traits>

namespace sd {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Mfma;
template <> struct Mfma<f16_t> {
  __device__ __forceinline__ static f32x4 step(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
  }
};
template <> struct Mfma<float> {
  __device__ __forceinline__ static f32x4 step(u32x4 a, u32x4 b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
};

__device__ __forceinline__ float silu(float g) { return g / (1.0f + expf(-g)); }

// register budget the compiler plans for: narrow tiles as for 16 waves
// (128 VGPRs, several workgroups per CU), wider ones as for 8 (256 VGPRs);
// a launch runs at most 4 waves
template <int MT, int NT> struct GemmBounds {
  static constexpr int threads = (MT * NT <= 4 && MT < 4 && NT < 4) ? 1024 : 512;
};

// Buffer resource over `bytes` bytes at p: raw (unswizzled) addressing with
// range checking, so a load at an offset >= bytes returns zero and reads no
// memory.  The main loop uses such offsets for padding rows and for step
// groups past a wave's share instead of branches: a load under a branch makes
// the compiler wait for every outstanding load before the next MFMA, which
// serialises the stream.
constexpr uint32_t OOB = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
// 16-byte buffer load; NT: non-temporal (streamed once, not kept in the caches)
template <bool NT> __device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, NT ? 2 : 0));
}

// QKV projection epilogue, shared by both GEMM kernels.  Output columns are
// the fused [q heads | k heads | v heads] rows of the weight, q and k in
// rotary pair order: column r16 < 8 of a 16-column tile of a q or k head is
// dim 8 b + r16 of the head, column r16 + 8 its partner dim hd/2 + 8 b + r16,
// so the two halves of a pair meet in one lane exchange (r16 ^ 8).
// qkv_column classifies column c0 + r16 of this lane once per tile: kind (0
// q, 1 k, 2 v), the q column, the rotary frequency index f, and the K/V
// element offset of (token 0, block 0); a row adds its block and token.
template <typename T>
__device__ __forceinline__ void qkv_column(const RopeParams& rp, int c0, int r16, int& kind, int& qcol, int& f,
                                           size_t& kvb) {
  const int hd = rp.hd, half = hd / 2, Nq = rp.H * hd, Nqk = Nq + rp.KV * hd;
  kind = c0 < Nq ? 0 : c0 < Nqk ? 1 : 2;
  qcol = 0;
  f = 0;
  kvb = 0;
  if (c0 < Nqk) {
    const int h = c0 / hd;
    f = 8 * ((c0 % hd) / 16) + (r16 & 7);
    const int d = r16 < 8 ? f : f + half;
    if (h < rp.H) qcol = h * hd + d;
    else kvb = kv_tile_off(h - rp.H, 0, 0, rp.nblk, hd) + kv_key_off<T>(0, d, hd);
  } else {
    const int cv = c0 + r16 - Nqk;
    kvb = kv_tile_off(cv / hd, 0, 1, rp.nblk, hd) + kv_val_off<T>(0, cv % hd, hd);
  }
}

// Rotary embedding of row m (position pos, KV block blk or -1) for the NT
// tiles of a lane: o = this lane's projection, pr = its pair partner's, cs =
// (cos, sin) of the lane's frequency; q goes to rp.q (fp32), k and v are
// appended to the cache (skipped when blk < 0: over capacity, flagged).
template <typename T, int NT>
__device__ __forceinline__ void qkv_store(const RopeParams& rp, int m, int pos, int blk, int r16, const float (&o)[NT],
                                          const float (&pr)[NT], const float2 (&cs)[NT], const int (&kind)[NT],
                                          const int (&qcol)[NT], const size_t (&kvb)[NT]) {
  const int off = pos & 15;
  T* kv = (T*)rp.kv;
  const size_t brow = (size_t)max(blk, 0) * 32 * rp.hd;   // block offset inside a head's run
  const size_t Nq = (size_t)rp.H * rp.hd;
#pragma unroll
  for (int j = 0; j < NT; ++j) {
    const float a = r16 < 8 ? o[j] : pr[j], b = r16 < 8 ? pr[j] : o[j];
    const float y = r16 < 8 ? a * cs[j].x - b * cs[j].y : a * cs[j].y + b * cs[j].x;
    if (kind[j] == 0) rp.q[(size_t)m * Nq + qcol[j]] = y;
    else if (blk < 0) continue;
    else if (kind[j] == 1) Store<T>::store(kv, kvb[j] + brow + kv_key_off<T>(off, 0, rp.hd), y);
    else Store<T>::store(kv, kvb[j] + brow + kv_val_off<T>(off, 0, rp.hd), o[j]);
  }
}

// Both operands are in the MFMA-tile layout (Tile<T>): fragment (tile t,
// k-step s) of a lane is the 16-byte unit 64 (t * ksteps + s) + lane, so a
// wave's load of one fragment is a contiguous 1 KB block.  The k-steps of a
// workgroup's K range are taken in groups of U; wave w takes groups w, w + KW,
// w + 2 KW, ..., so the waves of a workgroup read adjacent memory at any time.
// Each wave keeps the next group's loads in flight while it multiplies the
// current one (two register stages; scheduling barriers keep the compiler
// from pulling the loads next to their uses).
template <typename T, int MT, int NT, int U, int EPI>
__global__ __launch_bounds__((GemmBounds<MT, NT>::threads)) void gemm_kernel(GemmParams p) {

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int KW = blockDim.x >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const int ksteps = (int)((size_t)p.K * sizeof(T) / 64);
  // K * sizeof(T) is a multiple of 64 U (checked by the host); split y of
  // gridDim.y takes step groups [gb, gb + groups)
  const int gall = ksteps / U, gsp = (gall + gridDim.y - 1) / gridDim.y;
  const int gb = min((int)blockIdx.y * gsp, gall), groups = min(gsp, gall - gb);
  const int nw = max(0, (groups - wave + KW - 1) / KW);   // groups of this wave
  // Several M blocks (p.mblocks > 1, 1-D grid): workgroup w runs on XCD w % 8
  // (round-robin dispatch), so the M blocks of one column tile are given
  // consecutive slots of one XCD; they run together and all but the first
  // find the tile's weights in that XCD's L2 (plain loads, not streamed).
  // Otherwise blockIdx.x is the column tile and blockIdx.z the M block.
  int bx = blockIdx.x, bz = blockIdx.z;
  if (p.mblocks > 1) {
    const int w = blockIdx.x, j = w >> 3;
    bz = j % p.mblocks;
    bx = (j / p.mblocks) * 8 + (w & 7);
  }
  const bool stream_w = p.mblocks <= 1;
  // Balanced mode (p.tile_unit > 0): the N / 16 column tiles, in units of
  // tile_unit tiles (2 for SwiGLU: a gate tile and its up tile), are dealt
  // to the gridDim.x workgroups as evenly as possible, a contiguous run per
  // workgroup of at most NT tiles.  Loads of tiles past the run fall outside
  // the buffer range: they return zero and read nothing.
  int tile0 = bx * NT, ntile = NT;
  if (p.tile_unit > 0) {
    const int units = p.N / (16 * p.tile_unit), G = gridDim.x;
    const int base = units / G, extra = units % G;
    tile0 = (bx * base + min(bx, extra)) * p.tile_unit;
    ntile = (base + (bx < extra ? 1 : 0)) * p.tile_unit;
  }
  const int n0 = tile0 * 16;
  const int m0 = bz * MT * 16;
  const uint32_t tile_bytes = (uint32_t)ksteps * 1024u;
  const __amdgpu_buffer_rsrc_t wr = buf_rsrc((const char*)p.W + (size_t)tile0 * tile_bytes, ntile * tile_bytes);
  const __amdgpu_buffer_rsrc_t ar = buf_rsrc((const char*)p.A + (size_t)bz * MT * tile_bytes, MT * tile_bytes);

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // activation rows at or past M are padding: never read (their outputs are dropped)
  uint32_t aoff[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) aoff[t] = m0 + 16 * t + r16 < p.M ? (uint32_t)t * tile_bytes + lane * 16u : OOB;
  u32x4 ws[2][NT][U], as[2][MT][U];
  auto load = [&]<int S>(int i) {              // i-th step group of this wave's share
    const bool ok = i < nw;
    const uint32_t kb = (uint32_t)((gb + i * KW + wave) * U) * 1024u;
    // weights are read once: non-temporal loads keep them from evicting the
    // activations, which every workgroup re-reads from L2
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const uint32_t o = ok ? j * tile_bytes + kb + u * 1024u + lane * 16u : OOB;
        ws[S][j][u] = stream_w ? buf_load16<true>(wr, o) : buf_load16<false>(wr, o);
      }
#pragma unroll
    for (int t = 0; t < MT; ++t)
#pragma unroll
      for (int u = 0; u < U; ++u) as[S][t][u] = buf_load16<false>(ar, ok ? aoff[t] + kb + u * 1024u : OOB);
    __builtin_amdgcn_sched_barrier(0);
  };
  auto compute = [&]<int S>() {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < MT; ++t)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[t][j] = Mfma<T>::step(as[S][t][u], ws[S][j][u], acc[t][j]);
    __builtin_amdgcn_sched_barrier(0);
  };

  // QKV runs exactly 4 waves, so wave w finishes the rows 16 i + 4 g + w of
  // the block; their positions, KV blocks and rotary (cos, sin) are loaded
  // at the start of the stream, so the epilogue waits on nothing
  int qpos[EPI == EPI_QKV ? MT : 1], qblk[EPI == EPI_QKV ? MT : 1];
  if constexpr (EPI == EPI_QKV) {
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int m = m0 + 16 * i + 4 * g + wave;
      qpos[i] = m < p.M ? p.rope.row_pos[m] : -1;
      qblk[i] = m < p.M ? p.rope.row_blk[m] : -1;
    }
  }

  // QKV: what column n0 + 16 j + r16 of this lane is (independent of the row)
  int qkind[EPI == EPI_QKV ? NT : 1], qcol[EPI == EPI_QKV ? NT : 1], qf[EPI == EPI_QKV ? NT : 1];
  size_t qkvb[EPI == EPI_QKV ? NT : 1];
  float2 qcs[EPI == EPI_QKV ? MT : 1][NT];

  // groups past nw load zeros (no memory access) and add nothing
  load.template operator()<0>(0);
  if constexpr (EPI == EPI_QKV) {
    // the rotary (cos, sin) of this lane's rows are loaded once both register
    // stages are in flight: the wait for the row positions (loaded first)
    // then overlaps the first step group's, and the table loads complete
    // during the stream instead of after it
    load.template operator()<1>(1);
    const int half = p.rope.hd / 2;
#pragma unroll
    for (int j = 0; j < NT; ++j) qkv_column<T>(p.rope, n0 + 16 * j, r16, qkind[j], qcol[j], qf[j], qkvb[j]);
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j)
        qcs[i][j] = qpos[i] >= 0 && qkind[j] < 2 ? p.rope.tab[(size_t)qpos[i] * half + qf[j]] : float2{1.f, 0.f};
    __builtin_amdgcn_sched_barrier(0);
    for (int i = 0; i < nw; i += 2) {
      compute.template operator()<0>();
      load.template operator()<0>(i + 2);
      compute.template operator()<1>();
      load.template operator()<1>(i + 3);
    }
  } else {
    for (int i = 0; i < nw; i += 2) {
      load.template operator()<1>(i + 1);
      compute.template operator()<0>();
      load.template operator()<0>(i + 2);
      compute.template operator()<1>();
    }
  }

  // Reduction over the KW (<= 4) wave partials, in wave order 0, 1, 2, 3
  // (deterministic).  Finishing units are a gate/up tile pair (SwiGLU) or a
  // tile; with at least 4 of them each wave finishes whole units (one LDS
  // round, 16 bytes per lane), else each finishes output rows.
  constexpr int TPU = EPI == EPI_SWIGLU ? 2 : 1;        // tiles per unit
  constexpr int UPR = NT / TPU;                         // units per row tile
  if constexpr (EPI == EPI_QKV || MT * UPR < 4) {
    // every wave publishes its partial tile set; wave w finishes the output
    // rows (i, v) with (4 i + v) % KW == w (for QKV the rows whose
    // positions, KV blocks and rotary inputs it prefetched)
    __shared__ float red[4][MT * NT * 4][64];     // [wave][element][lane]
    // residual values of this wave's rows, loaded before the reduction (a
    // load behind the store of the previous row would wait for it)
    float rres[EPI == EPI_RESID ? MT : 1][4][EPI == EPI_RESID ? NT : 1];
    if constexpr (EPI == EPI_RESID) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          if ((4 * i + v) % KW != wave) continue;
          const int m = m0 + 16 * i + 4 * g + v;
#pragma unroll
          for (int j = 0; j < NT; ++j)
            rres[i][v][j] = m < p.M && j < ntile ? p.out[(size_t)m * p.ldo + n0 + 16 * j + r16] : 0.f;
        }
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) red[wave][(i * NT + j) * 4 + v][lane] = acc[i][j][v];
    __syncthreads();
    if constexpr (EPI == EPI_QKV) {
      // first use of the prefetched rotary inputs before any store: the wait
      // for them is taken here, not behind the epilogue's stores (the memory
      // counter also counts stores)
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        asm volatile("" : "+v"(qpos[i]), "+v"(qblk[i]));
#pragma unroll
        for (int j = 0; j < NT; ++j) asm volatile("" : "+v"(qcs[i][j].x), "+v"(qcs[i][j].y));
      }
    }
    // output element (i, j, v) is row m0 + 16 i + 4 g + v, column n0 + 16 j + r16
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        if ((4 * i + v) % KW != wave) continue;
        const int m = m0 + 16 * i + 4 * g + v;
        float o[NT];
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          float t = red[0][(i * NT + j) * 4 + v][lane];
          for (int w = 1; w < KW; ++w) t += red[w][(i * NT + j) * 4 + v][lane];
          o[j] = t;
        }
        if constexpr (EPI == EPI_QKV) {
          // the rotary partner of column r16 is column r16 ^ 8 of the same
          // tile (exchanged while the whole wave is still converged)
          float pr[NT];
#pragma unroll
          for (int j = 0; j < NT; ++j) pr[j] = __shfl_xor(o[j], 8);
          if (m >= p.M || qpos[i] < 0) continue;   // padding row, or no pending draft token
          qkv_store<T, NT>(p.rope, m, qpos[i], qblk[i], r16, o, pr, qcs[i], qkind, qcol, qkvb);
        } else if constexpr (EPI == EPI_SWIGLU) {
          if (m >= p.M) continue;
          // tiles (2k, 2k+1) are the gate and up rows of the same 16 outputs
          const int F = p.N / 2;
#pragma unroll
          for (int j = 0; j < NT; j += 2)
            if (j < ntile) Store<T>::store((T*)p.out_t, Tile<T>::off(m, n0 / 2 + 8 * j + r16, F), silu(o[j]) * o[j + 1]);
        } else {
          if (m >= p.M) continue;
          const size_t row = EPI == EPI_PART ? (size_t)blockIdx.y * p.M + m : (size_t)m;
#pragma unroll
          for (int j = 0; j < NT; ++j) {
            if (j >= ntile) continue;
            float* dst = p.out + row * p.ldo + n0 + 16 * j + r16;
            if constexpr (EPI == EPI_RESID) *dst = rres[i][v][j] + o[j];
            else *dst = o[j];
          }
        }
      }
  } else {
    // unit u (row tile i, unit k of it) is finished by wave u % KW; the
    // other waves leave their partial of its tiles in LDS slot
    // (w - f - 1) mod 4
    __shared__ f32x4 red[MT * NT][3][64];           // [tile][slot][lane]
    // residual values of the units this wave finishes, loaded before the
    // reduction so that their latency overlaps it
    float rres[EPI == EPI_RESID ? MT : 1][EPI == EPI_RESID ? UPR : 1][4];
    if constexpr (EPI == EPI_RESID) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int k = 0; k < UPR; ++k) {
          if ((i * UPR + k) % KW != wave || k * TPU >= ntile) continue;
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int m = m0 + 16 * i + 4 * g + v;
            rres[i][k][v] = m < p.M ? p.out[(size_t)m * p.ldo + n0 + 16 * k + r16] : 0.f;
          }
        }
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int f = (i * UPR + j / TPU) % KW;
        if (wave != f && j < ntile) red[i * NT + j][(wave - f - 1) & 3][lane] = acc[i][j];
      }
    __syncthreads();
    // the sum of a tile in wave order 0, 1, 2, 3; this wave's own partial
    // from registers, the others from their slots
    auto total = [&](const f32x4& own, int tile) {
      f32x4 t = own;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if (w >= KW) break;
        f32x4 pw;
        if (w == wave) pw = own;
        else pw = red[tile][(w - wave - 1) & 3][lane];
        t = w == 0 ? pw : t + pw;
      }
      return t;
    };
    // output element (i, j, v) is row m0 + 16 i + 4 g + v, column n0 + 16 j + r16
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int k = 0; k < UPR; ++k) {
        if ((i * UPR + k) % KW != wave || k * TPU >= ntile) continue;
        if constexpr (EPI == EPI_SWIGLU) {
          // tiles (2k, 2k+1) are the gate and up rows of the same 16 outputs
          const f32x4 gt = total(acc[i][2 * k], i * NT + 2 * k), up = total(acc[i][2 * k + 1], i * NT + 2 * k + 1);
          const int F = p.N / 2;
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int m = m0 + 16 * i + 4 * g + v;
            if (m < p.M) Store<T>::store((T*)p.out_t, Tile<T>::off(m, n0 / 2 + 16 * k + r16, F), silu(gt[v]) * up[v]);
          }
        } else {
          const f32x4 o = total(acc[i][k], i * NT + k);
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int m = m0 + 16 * i + 4 * g + v;
            if (m >= p.M) continue;
            const size_t row = EPI == EPI_PART ? (size_t)blockIdx.y * p.M + m : (size_t)m;
            float* dst = p.out + row * p.ldo + n0 + 16 * k + r16;
            if constexpr (EPI == EPI_RESID) *dst = rres[i][k][v] + o[v];
            else *dst = o[v];
          }
        }
      }
  }
}

// Wait until at most N vector memory operations of this wave are
// outstanding (vmcnt only; the LDS and export counters are not waited on).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Row-tiled GEMM for passes with more than one 64-row block (batched
// verify at B >= 32, prefill): there every weight byte meets hundreds of
// rows, so the operands are staged once per workgroup in LDS and shared.
// A workgroup of 4 waves (2 x 2) owns a BM x BN = 32 MF x 32 NF output tile;
// wave (wm, wn) owns the 16 MF x 16 NF sub-tile at (wm 16 MF, wn 16 NF).
// With 8 waves (one workgroup per CU) waves w and w + 4 own the same
// sub-tile and take the first and the second k-step of each stage; the
// second adds its sums to the first's through LDS at the end.
// K advances in stages of two k-steps (64 fp16); a stage is the
// 2 (BM + BN) / 16 1 KB fragments, which the waves load straight into
// one of NB LDS buffers (buffer loads with an LDS destination: lane i's
// 16 bytes land at the buffer's fragment base + 16 i, no registers held).
// NB - 1 stages are in flight while one is multiplied: at the top of stage
// st a wave waits until its own loads of stage st have landed (at most
// NB - 2 stages of its loads outstanding), then one barrier makes every
// wave's loads visible and frees the buffer stage st - 1 used, which then
// receives stage st + NB - 1.  Every stage issues the same number of loads
// (past the last stage, at an out-of-range offset: they read nothing), so
// the count the wait uses holds to the end.  The barrier is a plain
// s_barrier with a compiler memory clobber: a fenced one would wait for
// every load in flight.  Rows at or past M load zeros (range-checked buffer
// loads).  Tile order: the row tiles of one column tile take consecutive
// slots of one XCD (1-D grid, round-robin dispatch over 8 XCDs), so its
// weights are fetched from HBM once and re-read from that XCD's L2.
template <int MF, int NF, int EPI, int NB, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void gemm_rows_kernel(GemmParams p) {
  using T = f16_t;
  static_assert(WAVES == 4 || WAVES == 8, "4 waves, or 8 that split each stage's two k-steps");
  constexpr int BM = 32 * MF, BN = 32 * NF;
  constexpr int FA = 2 * BM / 16, FW = 2 * BN / 16;   // fragments per stage
  constexpr int LA = (FA + WAVES - 1) / WAVES, LW = (FW + WAVES - 1) / WAVES;   // loads per wave
  constexpr int SPARE = (WAVES * LA > FA || WAVES * LW > FW) ? 1 : 0;          // their overflow slot
  constexpr int FS = FA + FW + SPARE;
  static_assert(NB >= 2 && (NB - 2) * (LA + LW) < 64, "stages in flight");
  extern __shared__ __align__(16) unsigned char smem[];
  u32x4* lds = (u32x4*)smem;                          // [NB][FS][64]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = (wave >> 1) & 1;
  const int r16 = lane & 15, g = lane >> 4;
  const int ksteps = p.K * 2 / 64, stages = ksteps / 2;
  const int gx = p.N / BN, gz = (p.M + BM - 1) / BM;
  // K split: the R = gz ks (row tile, K range) pairs of a column tile take
  // consecutive slots of one XCD, as the row tiles alone do without a split
  const int ks = max(p.ksplit, 1), R = gz * ks;
  int bx, r;
  {
    const int w = blockIdx.x;
    if (gx % 8 == 0) {
      const int j = w >> 3;
      r = j % R;
      bx = (j / R) * 8 + (w & 7);
    } else {
      bx = w % gx;
      r = w / gx;
    }
  }
  const int bz = r % gz, split = r / gz;
  const int sps = (stages + ks - 1) / ks;              // stages of one K range
  const int s_lo = min(split * sps, stages), s_hi = min(s_lo + sps, stages);
  const uint32_t tile_bytes = (uint32_t)ksteps * 1024u;
  const __amdgpu_buffer_rsrc_t wr = buf_rsrc((const char*)p.W + (size_t)bx * (BN / 16) * tile_bytes, (BN / 16) * tile_bytes);
  const __amdgpu_buffer_rsrc_t ar = buf_rsrc((const char*)p.A + (size_t)bz * (BM / 16) * tile_bytes, (BM / 16) * tile_bytes);
  const int mvalid = p.M - bz * BM;                   // rows of this tile below M

  // this wave's share of stage st: A fragments f = WAVES k + wave (k < LA), W
  // fragments f = WAVES k + wave (k < LW); fragment f = 2 t + u is (16-row
  // tile t, k-step u of the stage).  Indices past the stage's fragments load
  // nothing (out-of-range offset) into the overflow slot, so every wave
  // issues the same count
  auto gload = [&](int st) {
    const bool ok = st < s_hi;
    u32x4* base = lds + (size_t)(st % NB) * FS * 64;
#pragma unroll
    for (int k = 0; k < LA; ++k) {
      const int f = WAVES * k + wave, t = f >> 1, u = f & 1;
      const bool real = FA % WAVES == 0 || f < FA;       // known true when the loads divide evenly
      const uint32_t off = real && ok && 16 * t + r16 < mvalid
                               ? (uint32_t)t * tile_bytes + (uint32_t)(2 * st + u) * 1024u + lane * 16u
                               : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ar, (__attribute__((address_space(3))) void*)(base + (real ? f : FA + FW) * 64),
                                               16, off, 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < LW; ++k) {
      const int f = WAVES * k + wave, t = f >> 1, u = f & 1;
      const bool real = FW % WAVES == 0 || f < FW;
      const uint32_t off = real && ok ? (uint32_t)t * tile_bytes + (uint32_t)(2 * st + u) * 1024u + lane * 16u : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (__attribute__((address_space(3))) void*)(base + (real ? FA + f : FA + FW) * 64),
                                               16, off, 0, 0, 0);
    }
  };

  f32x4 acc[MF][NF];
#pragma unroll
  for (int i = 0; i < MF; ++i)
#pragma unroll
    for (int j = 0; j < NF; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int st = 0; st < NB - 1; ++st) gload(s_lo + st);
  for (int st = s_lo; st < s_hi; ++st) {
    wait_vmcnt<(NB - 2) * (LA + LW)>();
    asm volatile("s_barrier" ::: "memory");
    gload(st + NB - 1);
    const u32x4* base = lds + (size_t)(st % NB) * FS * 64;
    // 4 waves: both k-steps of the stage; 8 waves: wave group w / 4 takes k-step w / 4
#pragma unroll
    for (int uu = 0; uu < 8 / WAVES; ++uu) {
      const int u = WAVES == 8 ? wave >> 2 : uu;
      u32x4 a[MF], b[NF];
#pragma unroll
      for (int i = 0; i < MF; ++i) a[i] = base[(2 * (wm * MF + i) + u) * 64 + lane];
#pragma unroll
      for (int j = 0; j < NF; ++j) b[j] = base[(FA + 2 * (wn * NF + j) + u) * 64 + lane];
#pragma unroll
      for (int i = 0; i < MF; ++i)
#pragma unroll
        for (int j = 0; j < NF; ++j) acc[i][j] = Mfma<T>::step(a[i], b[j], acc[i][j]);
    }
  }
  wait_vmcnt<0>();                                    // the trailing out-of-range loads
  if constexpr (WAVES == 8) {
    // waves 4-7 hand their k-step-1 sums to waves 0-3 through LDS (the stage
    // buffers, free once every wave is past the loop); waves 0-3 then finish
    float* red = (float*)smem + (size_t)(wave & 3) * MF * NF * 4 * 64;
    __syncthreads();
    if (wave >= 4) {
#pragma unroll
      for (int i = 0; i < MF; ++i)
#pragma unroll
        for (int j = 0; j < NF; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) red[((i * NF + j) * 4 + v) * 64 + lane] = acc[i][j][v];
    }
    __syncthreads();
    if (wave >= 4) return;
#pragma unroll
    for (int i = 0; i < MF; ++i)
#pragma unroll
      for (int j = 0; j < NF; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[i][j][v] += red[((i * NF + j) * 4 + v) * 64 + lane];
  }

  // epilogue: element (i, j, v) is row bz BM + wm 16 MF + 16 i + 4 g + v,
  // column n0 + 16 j + r16 with n0 the first column of the wave's sub-tile.
  // Every load of the epilogue (residual values; row positions, KV blocks
  // and rotary inputs) is issued for all of the lane's rows before the first
  // store: a load after a store to a possibly aliasing address would wait
  // for that store, one round trip per row.
  const int n0 = bx * BN + wn * 16 * NF;
  const int mrow0 = bz * BM + wm * 16 * MF + 4 * g;    // + 16 i + v
  if constexpr (EPI == EPI_QKV) {
    int qkind[NF], qcol[NF], qf[NF];
    size_t qkvb[NF];
#pragma unroll
    for (int j = 0; j < NF; ++j) qkv_column<T>(p.rope, n0 + 16 * j, r16, qkind[j], qcol[j], qf[j], qkvb[j]);
    const int half = p.rope.hd / 2;
    auto store_rows = [&](int i, const int (&pos)[4], const int (&blk)[4], const float2 (&cs)[4][NF]) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float o[NF], pr[NF];
#pragma unroll
        for (int j = 0; j < NF; ++j) o[j] = acc[i][j][v];
#pragma unroll
        for (int j = 0; j < NF; ++j) pr[j] = __shfl_xor(o[j], 8);
        if (pos[v] >= 0)   // a row at or past M has pos -1
          qkv_store<T, NF>(p.rope, mrow0 + 16 * i + v, pos[v], blk[v], r16, o, pr, cs[v], qkind, qcol, qkvb);
      }
    };
    auto load_rows = [&](int i, int (&pos)[4], int (&blk)[4]) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = mrow0 + 16 * i + v;
        pos[v] = m < p.M ? p.rope.row_pos[m] : -1;
        blk[v] = m < p.M ? p.rope.row_blk[m] : -1;
      }
    };
    auto load_cs = [&](const int (&pos)[4], float2 (&c)[4][NF]) {
#pragma unroll
      for (int v = 0; v < 4; ++v)
#pragma unroll
        for (int j = 0; j < NF; ++j)
          c[v][j] = qkind[j] < 2 ? p.rope.tab[(size_t)max(pos[v], 0) * half + qf[j]] : float2{1.f, 0.f};
    };
    if constexpr (NB > 2) {
      // one workgroup per CU: registers to spare, so the positions of all
      // the lane's rows are loaded at once and the rotary inputs one 16-row
      // tile ahead of the stores
      int pos[MF][4], blk[MF][4];
#pragma unroll
      for (int i = 0; i < MF; ++i) load_rows(i, pos[i], blk[i]);
      float2 cs[2][4][NF];
      load_cs(pos[0], cs[0]);
#pragma unroll
      for (int i = 0; i < MF; ++i) {
        if (i + 1 < MF) load_cs(pos[i + 1], cs[(i + 1) & 1]);
        store_rows(i, pos[i], blk[i], cs[i & 1]);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      // two workgroups per CU (large grids, e.g. prefill): registers are
      // short, so one row at a time; its loads then wait behind the previous
      // row's stores, which the long main loop of these shapes hides
#pragma unroll
      for (int i = 0; i < MF; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int m = mrow0 + 16 * i + v;
          float o[NF], pr[NF];
#pragma unroll
          for (int j = 0; j < NF; ++j) o[j] = acc[i][j][v];
#pragma unroll
          for (int j = 0; j < NF; ++j) pr[j] = __shfl_xor(o[j], 8);
          if (m >= p.M) continue;
          const int pos = p.rope.row_pos[m];
          if (pos < 0) continue;
          const int blk = p.rope.row_blk[m];
          float2 cs[NF];
#pragma unroll
          for (int j = 0; j < NF; ++j) cs[j] = qkind[j] < 2 ? p.rope.tab[(size_t)pos * half + qf[j]] : float2{1.f, 0.f};
          qkv_store<T, NF>(p.rope, m, pos, blk, r16, o, pr, cs, qkind, qcol, qkvb);
        }
    }
  } else if constexpr (EPI == EPI_RESID) {
    float r[MF][4][NF];
#pragma unroll
    for (int i = 0; i < MF; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = mrow0 + 16 * i + v;
#pragma unroll
        for (int j = 0; j < NF; ++j) r[i][v][j] = m < p.M ? p.out[(size_t)m * p.ldo + n0 + 16 * j + r16] : 0.f;
      }
#pragma unroll
    for (int i = 0; i < MF; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = mrow0 + 16 * i + v;
        if (m >= p.M) continue;
#pragma unroll
        for (int j = 0; j < NF; ++j) p.out[(size_t)m * p.ldo + n0 + 16 * j + r16] = r[i][v][j] + acc[i][j][v];
      }
  } else {
#pragma unroll
    for (int i = 0; i < MF; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = mrow0 + 16 * i + v;
        if (m >= p.M) continue;
        if constexpr (EPI == EPI_SWIGLU) {
          const int F = p.N / 2;
#pragma unroll
          for (int j = 0; j < NF; j += 2)
            Store<T>::store((T*)p.out_t, Tile<T>::off(m, n0 / 2 + 8 * j + r16, F), silu(acc[i][j][v]) * acc[i][j + 1][v]);
        } else {
          const size_t row = EPI == EPI_PART ? (size_t)split * p.M + m : (size_t)m;
#pragma unroll
          for (int j = 0; j < NF; ++j) p.out[row * p.ldo + n0 + 16 * j + r16] = acc[i][j][v];
        }
      }
  }
}

// LDS stages of the row-tiled GEMM: with one workgroup per CU (at most 256
// workgroups) as many as fit below 160 KB, up to 4; else 2, so that two
// workgroups share a CU.  Measured with weights streamed from HBM: 7B
// gate/up at M = 160 (172 workgroups) 67.7 -> 54.4 us with 4 stages (2:
// 65.0), QKV 55.3 -> 36.7, LM head 71.9 -> 59.1; 13B gate/up at M = 320
// (432 workgroups) 118 -> 110 us with 2 stages (4: 124.6), LM head 125.5
// -> 111.3 (4: 153.8).
// With at most 256 workgroups (one per CU) the kernel runs 8 waves: two per
// SIMD issue the LDS fills and matrix instructions that one wave per SIMD
// left half idle.  7B paged verify at M = 160 (kernel trace): gate/up 56.4
// -> 54.4 us, O / down with K split 24.3 -> 22.9, LM head 62.8 -> 60.7;
// above 256 workgroups two 4-wave workgroups share a CU instead.
constexpr int rows_stage_kb(int mf, int nf, int waves) {
  const int fa = 4 * mf, fw = 4 * nf, la = (fa + waves - 1) / waves, lw = (fw + waves - 1) / waves;
  return fa + fw + ((waves * la > fa || waves * lw > fw) ? 1 : 0);
}
constexpr int rows_stages_max(int mf, int nf, int waves) {
  return 159 / rows_stage_kb(mf, nf, waves) >= 4 ? 4 : 3;
}
constexpr bool rows_waves8(int epi, int mf) { return epi != EPI_RESID && epi != EPI_QKV && mf != 8; }
int gemm_rows_stages(int mf, int nf, int grid, int epi) {
  return grid <= 256 ? rows_stages_max(mf, nf, rows_waves8(epi, mf) ? 8 : 4) : 2;
}
size_t gemm_rows_lds(int mf, int nf, int nb, int waves) {
  const size_t stages = (size_t)nb * rows_stage_kb(mf, nf, waves) * 1024;
  const size_t red = waves == 8 ? (size_t)4 * mf * nf * 4 * 64 * sizeof(float) : 0;
  return std::max(stages, red);
}

template <int EPI, int MF, int NF, int NB, int WAVES>
static hipError_t launch_rows_t(int gz, const GemmParams& p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const size_t lds = gemm_rows_lds(MF, NF, NB, WAVES);
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute((const void*)gemm_rows_kernel<MF, NF, EPI, NB, WAVES>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  launch_k(gemm_rows_kernel<MF, NF, EPI, NB, WAVES>, dim3(p.N / (32 * NF) * gz * std::max(p.ksplit, 1)),
           dim3(64 * WAVES), (uint32_t)lds, s, e0, e1, p);
  return hipGetLastError();
}

template <int EPI>
static hipError_t launch_rows_e(int mf, int nf, int gz, const GemmParams& p, hipStream_t s, hipEvent_t e0,
                                hipEvent_t e1) {
  const int grid = p.N / (32 * nf) * gz * std::max(p.ksplit, 1);
  const int nb = gemm_rows_stages(mf, nf, grid, EPI);
  // the residual-add epilogue (a tile of residual values held), the QKV
  // epilogue (the row positions, KV blocks and rotary inputs of all of a
  // lane's rows prefetched) and 256-row tiles stay on 4 waves: 8 would leave
  // them short of registers (QKV on 8 waves with a row-at-a-time epilogue:
  // 7B at M = 160 50.2 us against 45.5)
#define SD_ROWS_CASE(MFv, NFv)                                                            \
  if (mf == MFv && nf == NFv) {                                                           \
    constexpr int w1 = rows_waves8(EPI, MFv) ? 8 : 4;                                     \
    constexpr int hi = rows_stages_max(MFv, NFv, w1);                                     \
    return nb == 2 ? launch_rows_t<EPI, MFv, NFv, 2, 4>(gz, p, s, e0, e1)                 \
                   : launch_rows_t<EPI, MFv, NFv, hi, w1>(gz, p, s, e0, e1);              \
  }
  SD_ROWS_CASE(4, 2) SD_ROWS_CASE(5, 2) SD_ROWS_CASE(6, 2) SD_ROWS_CASE(8, 2)
  SD_ROWS_CASE(4, 4) SD_ROWS_CASE(5, 4) SD_ROWS_CASE(6, 4) SD_ROWS_CASE(8, 4)
#undef SD_ROWS_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_rows(int epi, int mf, int nf, const GemmParams& p, hipStream_t s, hipEvent_t e0,
                            hipEvent_t e1) {
  const int bn = 32 * nf, bm = 32 * mf;
  if (p.N % bn || p.M < 1 || ((size_t)p.K * 2) % GEMM_CHUNK) return hipErrorInvalidValue;
  // a K split writes partial sums (PART) and needs at least one stage per range
  if (p.ksplit > 1 && (epi != EPI_PART || p.ksplit > (int)((size_t)p.K * 2 / GEMM_CHUNK))) return hipErrorInvalidValue;
  if (epi == EPI_PART && p.ksplit < 1) return hipErrorInvalidValue;
  const int gz = (p.M + bm - 1) / bm;
  switch (epi) {
    case EPI_STORE: return launch_rows_e<EPI_STORE>(mf, nf, gz, p, s, e0, e1);
    case EPI_RESID: return launch_rows_e<EPI_RESID>(mf, nf, gz, p, s, e0, e1);
    case EPI_SWIGLU: return launch_rows_e<EPI_SWIGLU>(mf, nf, gz, p, s, e0, e1);
    case EPI_PART: return launch_rows_e<EPI_PART>(mf, nf, gz, p, s, e0, e1);
    case EPI_QKV:
      if (p.rope.hd % 16 || p.N != (p.rope.H + 2 * p.rope.KV) * p.rope.hd) return hipErrorInvalidValue;
      return launch_rows_e<EPI_QKV>(mf, nf, gz, p, s, e0, e1);
    default: return hipErrorInvalidValue;
  }
}

// row-major [N, K] -> MFMA-tile layout, one 16-byte unit per thread; bf16
// sources (S = bf16_t) are converted to fp16 (T = f16_t) on the way: exact
// from 2^-14 up, smaller magnitudes round to the fp16 subnormal grid
template <typename S, typename T>
__global__ void pack_linear_kernel(const S* src, T* dst, int N, int K) {
  static_assert(sizeof(S) == sizeof(T), "same element size");
  constexpr int EPL = Tile<T>::EPL, EPK = Tile<T>::EPK;
  const int ks = K / EPK;
  const size_t units = (size_t)N * K / EPL;
  for (size_t u = blockIdx.x * (size_t)blockDim.x + threadIdx.x; u < units; u += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(u % 64);
    const size_t ts = u / 64;
    const int s = (int)(ts % ks), t = (int)(ts / ks);
    const int r = 16 * t + (lane & 15);
    const int k = s * EPK + (lane >> 4) * EPL;
    uint4 v = *(const uint4*)(src + (size_t)r * K + k);
    if constexpr (!std::is_same_v<S, T>) {
      uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
        w[i] = (uint32_t)f2h(bf2f((bf16_t)(w[i] & 0xffffu))) | ((uint32_t)f2h(bf2f((bf16_t)(w[i] >> 16))) << 16);
      v = make_uint4(w[0], w[1], w[2], w[3]);
    }
    *(uint4*)(dst + u * EPL) = v;
  }
}

hipError_t launch_pack_linear(int dtype, const void* src, void* dst, int N, int K, hipStream_t s) {
  const size_t esz = dtype == 0 ? 2 : 4;
  if (N <= 0 || K <= 0 || N % 16 || ((size_t)K * esz) % 64) return hipErrorInvalidValue;
  const size_t units = (size_t)N * K * esz / 16;
  const int blocks = (int)std::min<size_t>((units + 255) / 256, 65536);
  if (dtype == 0)
    hipLaunchKernelGGL((pack_linear_kernel<bf16_t, f16_t>), dim3(blocks), dim3(256), 0, s, (const bf16_t*)src,
                       (f16_t*)dst, N, K);
  else
    hipLaunchKernelGGL((pack_linear_kernel<float, float>), dim3(blocks), dim3(256), 0, s, (const float*)src,
                       (float*)dst, N, K);
  return hipGetLastError();
}

template <typename T, int EPI, int NT, int U>
static hipError_t launch_mt(int mt, dim3 grid, int threads, const GemmParams& p, hipStream_t s, hipEvent_t e0,
                            hipEvent_t e1) {
  switch (mt) {
    case 1:
    case 2:
      // 96-column tiles (balanced mode) only for 3-tile row blocks
      if constexpr (NT <= 4) {
        if (mt == 1) launch_k(gemm_kernel<T, 1, NT, U, EPI>, grid, dim3(threads), 0, s, e0, e1, p);
        else launch_k(gemm_kernel<T, 2, NT, U, EPI>, grid, dim3(threads), 0, s, e0, e1, p);
        break;
      }
      return hipErrorInvalidValue;
    case 3:
      if constexpr (NT <= 4 || NT == 6) {
        launch_k(gemm_kernel<T, 3, NT, U, EPI>, grid, dim3(threads), 0, s, e0, e1, p);
        break;
      }
      return hipErrorInvalidValue;
    case 4:
      // 64-row blocks (prefill) only with tiles of up to 32 columns
      if constexpr (NT <= 2) {
        launch_k(gemm_kernel<T, 4, NT, U, EPI>, grid, dim3(threads), 0, s, e0, e1, p);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int EPI>
static hipError_t launch_nt(int nt, int mt, dim3 grid, int threads, const GemmParams& p, hipStream_t s, hipEvent_t e0,
                            hipEvent_t e1) {
  switch (nt) {
    case 1:
      if constexpr (EPI != EPI_SWIGLU) return launch_mt<T, EPI, 1, GEMM_U>(mt, grid, threads, p, s, e0, e1);
      return hipErrorInvalidValue;
    case 2: return launch_mt<T, EPI, 2, GEMM_U>(mt, grid, threads, p, s, e0, e1);
    case 3:
      // 48-column tiles: only the QKV projection uses them (one tile per CU at 7B)
      if constexpr (EPI == EPI_QKV) return launch_mt<T, EPI, 3, GEMM_U>(mt, grid, threads, p, s, e0, e1);
      return hipErrorInvalidValue;
    case 4: return launch_mt<T, EPI, 4, GEMM_U>(mt, grid, threads, p, s, e0, e1);
    // balanced mode at 33-48 rows: SwiGLU up to 3 gate/up pairs
    case 6:
      if constexpr (EPI == EPI_SWIGLU && sizeof(T) == 2) return launch_mt<T, EPI, 6, GEMM_U>(mt, grid, threads, p, s, e0, e1);
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

bool gemm_config_ok(int dtype, int epi, int nt, int mt, int kw, int grid_x, int ksplit, int grid_z,
                    const GemmParams& p) {
  const size_t kbytes = (size_t)p.K * (dtype == 0 ? 2 : 4);
  if (mt < 1 || mt > 4 || kw < 1 || kw > 4) return false;
  // instantiated tiles: 48 columns for QKV only, 96 columns (16-bit SwiGLU,
  // 3 row tiles) for balanced mode only
  switch (nt) {
    case 1: if (epi == EPI_SWIGLU) return false; break;
    case 2: break;
    case 3: if (epi != EPI_QKV || mt > 3) return false; break;
    case 4: if (mt > 3) return false; break;
    case 6: if (epi != EPI_SWIGLU || dtype != 0 || mt != 3 || p.tile_unit <= 0) return false; break;
    default: return false;
  }
  if (mt == 4 && nt > 2) return false;
  if (p.tile_unit > 0) {
    // balanced mode: one M block, no K split, every workgroup within nt tiles
    if (p.tile_unit > 2 || p.N % (16 * p.tile_unit) || grid_x < 1 || grid_z != 1 || ksplit != 1 ||
        epi == EPI_QKV || epi == EPI_PART || (epi == EPI_SWIGLU && p.tile_unit != 2))
      return false;
    const int units = p.N / (16 * p.tile_unit);
    if (units < grid_x || (units + grid_x - 1) / grid_x * p.tile_unit > nt) return false;
  } else if (p.N % (16 * nt) || grid_x * 16 * nt != p.N) {
    return false;
  }
  if (grid_z * 16 * mt < p.M || kbytes % GEMM_CHUNK) return false;
  if (ksplit < 1 || (ksplit > 1 && epi != EPI_PART) || ksplit > (int)(kbytes / GEMM_CHUNK)) return false;
  if (epi == EPI_QKV && (kw != 4 || p.rope.hd % 16 || p.N != (p.rope.H + 2 * p.rope.KV) * p.rope.hd)) return false;
  return true;
}

hipError_t launch_gemm(int dtype, int epi, int nt, int mt, int kw, int grid_x, int ksplit, int grid_z,
                       const GemmParams& p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (!gemm_config_ok(dtype, epi, nt, mt, kw, grid_x, ksplit, grid_z, p)) return hipErrorInvalidValue;
  // several M blocks over column tiles in groups of 8: the XCD-aware 1-D grid
  GemmParams q = p;
  q.mblocks = 1;
  dim3 grid(grid_x, ksplit, grid_z);
  if (grid_z > 1 && ksplit == 1 && grid_x % 8 == 0) {
    q.mblocks = grid_z;
    grid = dim3(grid_x * grid_z, 1, 1);
  }
  const int threads = 64 * kw;
  if (dtype == 0) {
    if (epi == EPI_STORE) return launch_nt<f16_t, EPI_STORE>(nt, mt, grid, threads, q, s, e0, e1);
    if (epi == EPI_RESID) return launch_nt<f16_t, EPI_RESID>(nt, mt, grid, threads, q, s, e0, e1);
    if (epi == EPI_QKV) return launch_nt<f16_t, EPI_QKV>(nt, mt, grid, threads, q, s, e0, e1);
    if (epi == EPI_PART) return launch_nt<f16_t, EPI_PART>(nt, mt, grid, threads, q, s, e0, e1);
    return launch_nt<f16_t, EPI_SWIGLU>(nt, mt, grid, threads, q, s, e0, e1);
  }
  if (epi == EPI_STORE) return launch_nt<float, EPI_STORE>(nt, mt, grid, threads, q, s, e0, e1);
  if (epi == EPI_RESID) return launch_nt<float, EPI_RESID>(nt, mt, grid, threads, q, s, e0, e1);
  if (epi == EPI_QKV) return launch_nt<float, EPI_QKV>(nt, mt, grid, threads, q, s, e0, e1);
  if (epi == EPI_PART) return launch_nt<float, EPI_PART>(nt, mt, grid, threads, q, s, e0, e1);
  return launch_nt<float, EPI_SWIGLU>(nt, mt, grid, threads, q, s, e0, e1);
}

}  // namespace sd
