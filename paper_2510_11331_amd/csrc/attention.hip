// Causal multi-query attention over the paged KV cache (Section II-A: eq.
// d_kv grows the cache by concatenation, done by the QKV projection's
// epilogue; eq. d_atte / f21 attend with softmax(q K^T / sqrt(d0)) V), and
// the rotary (cos, sin) table that epilogue reads.
//
// Paged layout of one layer's pool: head-major tiles [kv head][block][K|V]
// (kv_tile_off), so that the blocks of one task and head, allocated in
// order, are one contiguous run; K in the layout of the S = K Q^T matrix
// instruction for 16-bit caches (kv_key_off: every wave load of a key k-step
// is a contiguous 1 KB) or as [16 tokens][hd] for fp32; V transposed so that
// the P*V operand of a matrix instruction is 4 consecutive tokens of one
// dimension (kv_val_off: for 16-bit caches two such quads per 16-byte unit,
// 1 KB per wave load; [hd][16 tokens] for fp32); a slot's block table maps
// position / 16 to a block.
//
// Attention work item = (row block, kv head, key split).  A row block is a
// run of consecutive rows of one task (the gamma+1 verify rows of a task, its
// 1-2 draft rows, or a run of prefill rows); all G query heads of the kv
// head and all rows of the block are one set of query vectors that shares
// every K/V tile.  Query i only sees keys at positions <= its own.  Each work
// item keeps an online softmax (running max, running sum, rescaled output);
// when the keys are split (evenly over the item's context), partial (max,
// sum, output) triples go to a workspace with device-scope stores, and the
// last split of the item to finish merges them in split order (the fp32
// kernel leaves the merge to a second kernel).
//
// bf16 models (fp16 KV cache, see f16_t): S^T = K Q^T and O^T += V^T P^T on
// v_mfma_f32_16x16x32_f16, 16 query vectors per wave, keys streamed from the
// cache straight into registers 32 at a time (two blocks), one step ahead,
// with non-temporal loads (each cache byte is read once per pass); q and p
// enter the matrix instruction as fp16 hi + lo pairs, which keeps them at
// ~2^-22 relative precision.  fp32 models: a vector kernel with K/V staged
// in LDS.
#include "sd_internal.h"

#include <algorithm>

namespace sd {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// rotary (cos, sin) table: angle pos * theta^(-2i/hd) in float64, rounded to
// float32 once (the rotation itself is done in float32 by the QKV epilogue)
__global__ void rope_table_kernel(float2* tab, int n_pos, int half, double theta) {
  const size_t n = (size_t)n_pos * half;
  for (size_t idx = blockIdx.x * (size_t)blockDim.x + threadIdx.x; idx < n; idx += (size_t)gridDim.x * blockDim.x) {
    const int pos = (int)(idx / half), i = (int)(idx % half);
    const double ang = (double)pos * pow(theta, -2.0 * (double)i / (double)(2 * half));
    double s, c;
    sincos(ang, &s, &c);
    tab[idx] = make_float2((float)c, (float)s);
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// the vector kernel serves fp32 caches only (16-bit caches run on the matrix kernel)
template <typename T> struct KvT;
template <> struct KvT<float> {
  static constexpr int KST_PAD = 1;
  static constexpr int EPU = 4;
};

// dynamic LDS layout, in bytes
__host__ __device__ inline size_t attn_lds_bytes(int hd, int esz, int qmax) {
  const int kst = hd + (esz == 2 ? 2 : 1);
  size_t b = (size_t)64 * kst * esz + (size_t)64 * hd * esz;
  b = (b + 15) & ~(size_t)15;
  b += (size_t)qmax * hd * 4 + (size_t)qmax * 65 * 4 + (size_t)qmax * 4 * 4;
  return b;
}

template <typename T, int HD>
__global__ __launch_bounds__(256) void attention_kernel(AttnParams p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  constexpr int KST = HD + KvT<T>::KST_PAD;
  constexpr int EPU = KvT<T>::EPU;
  constexpr int NQG = 256 / HD;            // query groups in the P*V phase
  constexpr int QPT = ATTN_QMAX / NQG;     // query vectors per thread in P*V

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rbk = blockIdx.x;
  const int rb = rbk / p.KV, kvh = rbk % p.KV;
  const int split = blockIdx.y;
  int row0, nr;
  if (p.rowblocks) {
    row0 = p.rowblocks[2 * rb];
    nr = p.rowblocks[2 * rb + 1];
  } else {
    row0 = rb * p.R;
    nr = p.R;
  }
  const int G = p.H / p.KV;
  const int Qn = nr * G;
  const int qmax = p.qmax;

  T* Ks = (T*)smem;
  T* Vs = Ks + 64 * KST;
  size_t off = ((size_t)64 * KST + (size_t)64 * HD) * sizeof(T);
  off = (off + 15) & ~(size_t)15;
  float* Qs = (float*)(smem + off);
  float* Ss = Qs + qmax * HD;
  float* Ms = Ss + qmax * 65;
  float* Ls = Ms + qmax;
  float* As = Ls + qmax;
  int* Ps = (int*)(As + qmax);

  int maxpos = -1;
  for (int r = 0; r < nr; ++r) maxpos = max(maxpos, p.row_pos[row0 + r]);
  const int slot = p.row_bt ? 0 : p.row_slot[row0];   // decode passes: the row block's own table row
  const int k_begin = split * p.keys_per_split;
  // keys never extend past the slot's block-table row
  const int k_end = min(min(k_begin + p.keys_per_split, maxpos + 1), p.mbps * 16);
  const int Hq = p.H * HD;

  for (int idx = tid; idx < Qn * HD; idx += 256) {
    const int qi = idx / HD, d = idx % HD;
    const int row = row0 + qi / G, h = kvh * G + qi % G;
    Qs[qi * HD + d] = p.q[(size_t)row * Hq + h * HD + d] * p.scale;
  }
  for (int qi = tid; qi < Qn; qi += 256) {
    Ps[qi] = p.row_pos[row0 + qi / G];
    Ms[qi] = -INFINITY;
    Ls[qi] = 0.f;
  }

  const int dd = tid % HD, qg = tid / HD;
  float o[QPT];
#pragma unroll
  for (int k = 0; k < QPT; ++k) o[k] = 0.f;

  const T* kv = (const T*)p.kv;
  const int32_t* bt = (p.row_bt ? p.row_bt + (size_t)rb * p.mbps : p.block_table + (size_t)slot * p.mbps);

  for (int c = k_begin; c < k_end; c += 64) {
    __syncthreads();
    // stage 64 keys of K and V
    constexpr int UPR = HD / EPU;      // 16-byte units per key row
    for (int idx = tid; idx < 64 * UPR; idx += 256) {
      const int j = idx / UPR, e = (idx % UPR) * EPU;
      const int kp = c + j;
      uint4 kk = make_uint4(0, 0, 0, 0);
      T vv[EPU];
#pragma unroll
      for (int t = 0; t < EPU; ++t) vv[t] = T(0);
      if (kp < k_end) {
        const int blk = bt[kp / 16];
        const size_t base = kv_tile_off(kvh, blk, 0, p.nblk, HD) + (size_t)(kp % 16) * HD + e;
        const size_t vtb = kv_tile_off(kvh, blk, 1, p.nblk, HD);
        kk = *(const uint4*)(kv + base);
#pragma unroll
        for (int t = 0; t < EPU; ++t) vv[t] = kv[vtb + kv_val_off<T>(kp % 16, e + t, HD)];
      }
      uint32_t* kd = (uint32_t*)(Ks + j * KST + e);   // KST*esz is a multiple of 4
      kd[0] = kk.x; kd[1] = kk.y; kd[2] = kk.z; kd[3] = kk.w;
#pragma unroll
      for (int t = 0; t < EPU; ++t) Vs[j * HD + e + t] = vv[t];
    }
    __syncthreads();
    // scores and online softmax: wave w takes query vectors w, w+4, ...; lane = key
    const int kp = c + lane;
    for (int qi = wave; qi < Qn; qi += 4) {
      const float* qv = Qs + qi * HD;
      const T* kr = Ks + lane * KST;
      float s = 0.f;
#pragma unroll 8
      for (int d = 0; d < HD; ++d) s += qv[d] * Store<T>::load(kr, d);
      const bool ok = kp < k_end && kp <= Ps[qi];
      s = ok ? s : -INFINITY;
      const float mold = Ms[qi];
      const float mnew = fmaxf(mold, wave_max(s));
      const float pj = ok ? expf(s - mnew) : 0.f;
      const float psum = wave_sum(pj);
      const float alpha = mold == -INFINITY ? 0.f : expf(mold - mnew);
      Ss[qi * 65 + lane] = pj;
      if (lane == 0) {
        Ms[qi] = mnew;
        Ls[qi] = Ls[qi] * alpha + psum;
        As[qi] = alpha;
      }
    }
    __syncthreads();
    // P*V: thread (dd, qg) accumulates dimension dd of query vectors qg, qg+NQG, ...
#pragma unroll
    for (int k = 0; k < QPT; ++k) {
      const int qi = qg + NQG * k;
      if (qi < Qn) {
        float a = o[k] * As[qi];
        const float* pr = Ss + qi * 65;
#pragma unroll 8
        for (int j = 0; j < 64; ++j) a += pr[j] * Store<T>::load(Vs, j * HD + dd);
        o[k] = a;
      }
    }
  }
  __syncthreads();

  auto emit = [&](int qi, float val) {
    const int row = row0 + qi / G, h = kvh * G + qi % G;
    Store<T>::store((T*)p.out, Tile<T>::off(row, h * HD + dd, Hq), val);
  };

  if (p.splits == 1) {
#pragma unroll
    for (int k = 0; k < QPT; ++k) {
      const int qi = qg + NQG * k;
      if (qi < Qn) {
        const float L = Ls[qi];
        emit(qi, L > 0.f ? o[k] / L : 0.f);
      }
    }
    return;
  }

  // key split: partial (output, max, sum) for attn_merge_kernel
  const size_t item = (size_t)rbk * p.splits;
#pragma unroll
  for (int k = 0; k < QPT; ++k) {
    const int qi = qg + NQG * k;
    if (qi < Qn) p.part_o[((item + split) * qmax + qi) * HD + dd] = o[k];
  }
  for (int qi = tid; qi < Qn; qi += 256) {
    p.part_ml[((item + split) * qmax + qi) * 2 + 0] = Ms[qi];
    p.part_ml[((item + split) * qmax + qi) * 2 + 1] = Ls[qi];
  }
}

// fp16 hi + lo pair of 8 floats (hi = x rounded, lo = the rest rounded),
// packed as two f16x8 operands
__device__ __forceinline__ void split8(const float (&x)[8], u32x4& hi, u32x4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint16_t a0 = f2h(x[2 * k]), a1 = f2h(x[2 * k + 1]);
    const uint16_t b0 = f2h(x[2 * k] - h2f(a0)), b1 = f2h(x[2 * k + 1] - h2f(a1));
    h[k] = (uint32_t)a0 | ((uint32_t)a1 << 16);
    l[k] = (uint32_t)b0 | ((uint32_t)b1 << 16);
  }
  hi = u32x4{h[0], h[1], h[2], h[3]};
  lo = u32x4{l[0], l[1], l[2], l[3]};
}

__device__ __forceinline__ f32x4 mfma_f16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                0, 0);
}

// Wave w of a workgroup (WAVES = 8) takes query tile w % QTe (16 query
// vectors) and key group w / QTe: 32-key steps kb = k_begin + 32 (kg + KG j).
// Lane (r16, g): query r16 of the tile; in S^T it holds keys 4g..4g+3 of
// both blocks of the step, in O^T dimensions 16 dt + 4g .. +3.
template <int HD, int WAVES>
__global__ __launch_bounds__(64 * WAVES, 8 / WAVES) void attention_mfma_kernel(AttnParams p) {
  constexpr int UPG = HD / 32;             // 16-byte K units per lane group (HD/4 dims)
  constexpr int DT = HD / 16;              // 16-dimension output tiles
  constexpr int NSLOT = WAVES / 2;         // merge slots: half the waves hand over in the first round
  __shared__ float s_o[NSLOT][16][HD + 4];
  __shared__ float s_m[NSLOT][16], s_l[NSLOT][16];

  __shared__ int s_bt[ATTN_BT_CAP];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const int rbk = blockIdx.x;
  const int rb = rbk / p.KV, kvh = rbk % p.KV;
  const int split = blockIdx.y;
  int row0, nr;
  if (p.rowblocks) {
    row0 = p.rowblocks[2 * rb];
    nr = p.rowblocks[2 * rb + 1];
  } else {
    row0 = rb * p.R;
    nr = p.R;
  }
  const int G = p.H / p.KV;
  const int Qn = nr * G;
  const int QT = (Qn + 15) >> 4;
  const int QTe = QT == 3 ? 4 : QT;
  const int KG = WAVES / QTe;
  const int qt = wave % QTe, kg = wave / QTe;
  const bool wave_on = qt < QT;

  // the block's rows (nr <= 64: Qn is at most 64 query vectors) in parallel
  int maxpos = lane < nr ? p.row_pos[row0 + lane] : -1;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) maxpos = max(maxpos, __shfl_xor(maxpos, o));
  maxpos = __builtin_amdgcn_readfirstlane(maxpos);
  const int slot = p.row_bt ? 0 : p.row_slot[row0];   // decode passes: the row block's own table row
  // the item's keys (positions 0 .. maxpos) are dealt out evenly over the
  // splits in 32-key steps, at most the host's keys_per_split per split
  // (which bounds the staged block ids)
  const int kps = p.splits > 1 ? min(p.keys_per_split, ((maxpos + p.splits) / p.splits + 31) / 32 * 32)
                               : p.keys_per_split;
  const int k_begin = split * kps;
  const int k_end = min(min(k_begin + kps, maxpos + 1), p.mbps * 16);

  // block ids of the split's key range, staged in LDS (the host keeps a
  // split within ATTN_BT_CAP blocks): a key load then never waits on the
  // memory counter behind the keys still in flight
  const int32_t* bt = (p.row_bt ? p.row_bt + (size_t)rb * p.mbps : p.block_table + (size_t)slot * p.mbps);
  const int bfirst = k_begin / 16, nbr = max(0, (k_end + 15) / 16 - bfirst);
  for (int i = tid; i < min(nbr, ATTN_BT_CAP); i += blockDim.x) s_bt[i] = bt[bfirst + i];
  __syncthreads();

  const int qi = qt * 16 + r16;
  const bool qvalid = wave_on && qi < Qn;
  const int qrow = row0 + (qvalid ? qi / G : 0);
  const int qh = kvh * G + (qvalid ? qi % G : 0);
  const int qpos = qvalid ? p.row_pos[qrow] : -1;

  u32x4 qhi[UPG], qlo[UPG];
  {
    // always-valid address (row0, head kvh G for idle lanes), zeroed after the load
    const float4* qs = (const float4*)(p.q + (size_t)qrow * p.H * HD + (size_t)qh * HD + g * (HD / 4));
    float4 xv[2 * UPG];
#pragma unroll
    for (int s = 0; s < 2 * UPG; ++s) xv[s] = qs[s];
#pragma unroll
    for (int s = 0; s < UPG; ++s) {
      // scores in log2 units (q pre-scaled by log2 e): the softmax then
      // uses the hardware base-2 exponential
      const float sc = qvalid ? p.scale * 1.4426950408889634f : 0.f;
      float x[8] = {xv[2 * s].x * sc, xv[2 * s].y * sc, xv[2 * s].z * sc, xv[2 * s].w * sc,
                    xv[2 * s + 1].x * sc, xv[2 * s + 1].y * sc, xv[2 * s + 1].z * sc, xv[2 * s + 1].w * sc};
      split8(x, qhi[s], qlo[s]);
    }
  }

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};

  // this kv head's region of the pool ([blocks][K|V][16 x HD], 2 x 16 HD
  // fp16 per block) as a range-checked buffer: steps past the key range
  // load at an out-of-range offset, which returns zero and reads nothing
  constexpr uint32_t BLK_BYTES = 2u * 16u * HD * 2u;
  const __amdgpu_buffer_rsrc_t kvr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<f16_t*>((const f16_t*)p.kv + kv_tile_off(kvh, 0, 0, p.nblk, HD)), (short)0,
      (int)((uint32_t)p.nblk * BLK_BYTES), 0x00020000);
  // key tile in the matrix-instruction layout: k-step s is the 1 KB run at
  // unit 64 s, this lane's 16 bytes at unit 64 s + lane (token r16, dims
  // g HD/4 + 8 s .. + 8); the V tile follows the K tile of the same block
  const uint32_t koff = (uint32_t)lane * 16u;
  // V tile (kv_val_off): unit 4 r16 + g of 32-dim group dp holds tokens
  // 4g..4g+3 of dims 32 dp + r16 and 32 dp + 16 + r16 (the 64 lanes read the
  // group's 1 KB)
  const uint32_t voff = 16u * HD * 2u + (uint32_t)(4 * r16 + g) * 16u;

  // two register stages of one 32-key step: K rows (two blocks), V^T quads
  // as loaded, and the masks of the V entries past the key range (applied
  // by the step, so a load is not consumed the moment it is issued)
  u32x4 Kf[2][2][UPG], Vr[2][2][DT / 2];
  uint32_t Vm[2][2][2];

  auto load = [&]<int S>(int kb) {
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int kt = kb + 16 * t;
      const bool ok = kt < k_end;
      const uint32_t base = ok ? (uint32_t)s_bt[kt / 16 - bfirst] * BLK_BYTES : 0x80000000u;
#pragma unroll
      for (int s = 0; s < UPG; ++s)
        Kf[S][t][s] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(kvr, base + koff + 1024u * s, 0, 2));
      // keys at or past k_end were never written: their scores are masked, and
      // their V entries are zeroed so that p = 0 never meets a NaN/Inf pattern
      const int nq = min(max(k_end - (kt + 4 * g), 0), 4);
      Vm[S][t][0] = nq >= 2 ? 0xffffffffu : (nq == 1 ? 0xffffu : 0u);
      Vm[S][t][1] = nq >= 4 ? 0xffffffffu : (nq == 3 ? 0xffffu : 0u);
#pragma unroll
      for (int dp = 0; dp < DT / 2; ++dp)
        Vr[S][t][dp] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(kvr, base + voff + 1024u * dp, 0, 2));
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  auto step = [&]<int S>(int kb) {
    // four independent accumulation chains (the hi and lo parts of q for
    // each of the two key blocks), so that consecutive matrix instructions
    // do not wait on each other's results; the parts are added at the end
    f32x4 s0 = f32x4{0.f, 0.f, 0.f, 0.f}, s1 = s0, s0l = s0, s1l = s0;
#pragma unroll
    for (int s = 0; s < UPG; ++s) {
      s0 = mfma_f16(Kf[S][0][s], qhi[s], s0);
      s1 = mfma_f16(Kf[S][1][s], qhi[s], s1);
      s0l = mfma_f16(Kf[S][0][s], qlo[s], s0l);
      s1l = mfma_f16(Kf[S][1][s], qlo[s], s1l);
    }
    s0 += s0l;
    s1 += s1l;
    float sc[8];
    bool ok[8];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int k0 = kb + 4 * g + v, k1 = k0 + 16;
      ok[v] = k0 < k_end && k0 <= qpos;
      ok[4 + v] = k1 < k_end && k1 <= qpos;
      sc[v] = s0[v];
      sc[4 + v] = s1[v];
    }
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 8; ++e) mx = ok[e] ? fmaxf(mx, sc[e]) : mx;
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m_run, mx);
    float pe[8], sum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pe[e] = ok[e] ? exp2f(sc[e] - mnew) : 0.f;
      sum += pe[e];
    }
    sum += __shfl_xor(sum, 16);
    sum += __shfl_xor(sum, 32);
    const float alpha = m_run == -INFINITY ? 0.f : exp2f(m_run - mnew);
    l_run = l_run * alpha + sum;
    m_run = mnew;
    u32x4 phi, plo;
    split8(pe, phi, plo);
#pragma unroll
    for (int d = 0; d < DT; ++d) {
      o[d] *= alpha;
      // dims d (even d: x, y of the unit) of tokens 4g..4g+3 of both blocks
      const u32x4 v0 = Vr[S][0][d / 2], v1 = Vr[S][1][d / 2];
      const u32x4 va = (d & 1) ? u32x4{v0.z & Vm[S][0][0], v0.w & Vm[S][0][1], v1.z & Vm[S][1][0], v1.w & Vm[S][1][1]}
                               : u32x4{v0.x & Vm[S][0][0], v0.y & Vm[S][0][1], v1.x & Vm[S][1][0], v1.y & Vm[S][1][1]};
      o[d] = mfma_f16(va, phi, o[d]);
      o[d] = mfma_f16(va, plo, o[d]);
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  // loads are issued unconditionally (past the key range they read
  // nothing), so the compiler keeps the next step in flight during a step
  const int kstep = 32 * KG;
  int kb = k_begin + 32 * kg;
  if (wave_on && kb < k_end) {
    load.template operator()<0>(kb);
    for (; kb < k_end; kb += 2 * kstep) {
      const int kb1 = kb + kstep;
      load.template operator()<1>(kb1);
      step.template operator()<0>(kb);
      if (kb1 >= k_end) break;
      load.template operator()<0>(kb1 + kstep);
      step.template operator()<1>(kb1);
    }
  }

  // merge the key groups of each query tile into key group 0 as a binary
  // tree (fixed order): in the round of stride h, key group kg with
  // kg % 2h == h hands its state to kg - h through slot qt KG/2 + kg / 2h
  for (int h = 1; h < KG; h *= 2) {
    const int sl = qt * (KG / 2) + kg / (2 * h);
    if (wave_on && kg % (2 * h) == h) {
      if (g == 0) {
        s_m[sl][r16] = m_run;
        s_l[sl][r16] = l_run;
      }
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int v = 0; v < 4; ++v) s_o[sl][r16][16 * d + 4 * g + v] = o[d][v];
    }
    __syncthreads();
    if (wave_on && kg % (2 * h) == 0) {
      const float mb = s_m[sl][r16], lb = s_l[sl][r16];
      const float M = fmaxf(m_run, mb);
      const float a = m_run == -INFINITY ? 0.f : exp2f(m_run - M);
      const float b = mb == -INFINITY ? 0.f : exp2f(mb - M);
      l_run = l_run * a + lb * b;
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int v = 0; v < 4; ++v) o[d][v] = o[d][v] * a + s_o[sl][r16][16 * d + 4 * g + v] * b;
      m_run = M;
    }
    __syncthreads();
  }
  const bool owner = wave_on && kg == 0 && qvalid;
  // four consecutive output dimensions of this lane's query, MFMA-tile layout
  auto emit4 = [&](int d, float a0, float a1, float a2, float a3) {
    const size_t off = Tile<f16_t>::off(qrow, qh * HD + 16 * d + 4 * g, p.H * HD);
    *(uint2*)((f16_t*)p.out + off) = make_uint2((uint32_t)f2h(a0) | ((uint32_t)f2h(a1) << 16),
                                                (uint32_t)f2h(a2) | ((uint32_t)f2h(a3) << 16));
  };

  if (p.splits == 1) {
    if (owner) {
      const float inv = l_run > 0.f ? 1.0f / l_run : 0.f;
#pragma unroll
      for (int d = 0; d < DT; ++d) emit4(d, o[d][0] * inv, o[d][1] * inv, o[d][2] * inv, o[d][3] * inv);
    }
    return;
  }

  // key split: this workgroup's partial (output, max, sum) goes out with
  // device-scope stores; the item's last split to finish merges them.  Every
  // value handed over is written and read with device-scope atomic
  // operations, which the L2 of another XCD does not serve stale, so waiting
  // for the stores before counting is all the ordering needed (a release /
  // acquire fence would also write back and invalidate the whole L2, which
  // only data written with plain stores needs)
  const size_t base = (size_t)rbk * p.splits * p.qmax;
  const size_t item = base + (size_t)split * p.qmax + (owner ? qi : 0);
  if (owner) {
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        __hip_atomic_store(p.part_o + item * HD + 16 * d + 4 * g + v, o[d][v], __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    if (g == 0) {
      // natural units for the merge
      __hip_atomic_store(p.part_ml + item * 2, m_run == -INFINITY ? -INFINITY : m_run * 0.6931471805599453f,
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(p.part_ml + item * 2 + 1, l_run, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __shared__ int s_last;
  __builtin_amdgcn_s_waitcnt(0);      // this wave's partial stores have reached device scope
  __syncthreads();
  if (tid == 0) {
    const int old = __hip_atomic_fetch_add(p.cnt + rbk, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = old == p.splits - 1;
    if (last) __hip_atomic_store(p.cnt + rbk, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = last;
  }
  __syncthreads();
  if (!s_last) return;

  // merge, in split order: O = sum_s o_s e^(m_s - M) / sum_s l_s e^(m_s - M),
  // M = max_s m_s; every load of a query's splits is issued before any is used
  __shared__ float s_w[ATTN_QMAX][ATTN_MAX_SPLITS], s_L[ATTN_QMAX];
  for (int qj = tid; qj < Qn; qj += 64 * WAVES) {
    float ms[ATTN_MAX_SPLITS], ls[ATTN_MAX_SPLITS];
#pragma unroll
    for (int sp = 0; sp < ATTN_MAX_SPLITS; ++sp) {
      const size_t it = (base + (size_t)sp * p.qmax + qj) * 2;
      ms[sp] = sp < p.splits ? __hip_atomic_load(p.part_ml + it, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                             : -INFINITY;
      ls[sp] = sp < p.splits ? __hip_atomic_load(p.part_ml + it + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                             : 0.f;
    }
    float M = -INFINITY;
#pragma unroll
    for (int sp = 0; sp < ATTN_MAX_SPLITS; ++sp) M = fmaxf(M, ms[sp]);
    float L = 0.f;
#pragma unroll
    for (int sp = 0; sp < ATTN_MAX_SPLITS; ++sp) {
      const float w = ms[sp] == -INFINITY ? 0.f : expf(ms[sp] - M);
      L += ls[sp] * w;
      s_w[qj][sp] = w;
    }
    s_L[qj] = L;
  }
  __syncthreads();
  for (int idx = tid; idx < Qn * HD; idx += 64 * WAVES) {
    const int qj = idx / HD, d = idx % HD;
    float os[ATTN_MAX_SPLITS];
#pragma unroll
    for (int sp = 0; sp < ATTN_MAX_SPLITS; ++sp)
      os[sp] = sp < p.splits ? __hip_atomic_load(p.part_o + (base + (size_t)sp * p.qmax + qj) * HD + d,
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                             : 0.f;
    float O = 0.f;
#pragma unroll
    for (int sp = 0; sp < ATTN_MAX_SPLITS; ++sp) O += os[sp] * s_w[qj][sp];
    const float L = s_L[qj];
    const int row = row0 + qj / G, h = kvh * G + qj % G;
    Store<f16_t>::store((f16_t*)p.out, Tile<f16_t>::off(row, h * HD + d, p.H * HD), L > 0.f ? O / L : 0.f);
  }
}

// Merge of the key splits of every (row block, kv head) item of the fp32
// kernel, in split order: O = sum_s o_s e^(m_s - M) / sum_s l_s e^(m_s - M),
// M = max_s m_s.  (The matrix kernel merges its splits itself: the last split
// of an item to finish reads the others' partials, written with device-scope
// stores, and no L2 write-back or second launch is needed.)
template <typename T, int HD>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams p) {
  const int rbk = blockIdx.x, rb = rbk / p.KV, kvh = rbk % p.KV;
  int row0, nr;
  if (p.rowblocks) {
    row0 = p.rowblocks[2 * rb];
    nr = p.rowblocks[2 * rb + 1];
  } else {
    row0 = rb * p.R;
    nr = p.R;
  }
  const int G = p.H / p.KV, Qn = nr * G;
  const size_t base = (size_t)rbk * p.splits * p.qmax;
  for (int idx = threadIdx.x; idx < Qn * HD; idx += blockDim.x) {
    const int qi = idx / HD, d = idx % HD;
    float M = -INFINITY;
    for (int sp = 0; sp < p.splits; ++sp) M = fmaxf(M, p.part_ml[(base + (size_t)sp * p.qmax + qi) * 2]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
      for (int sp = 0; sp < p.splits; ++sp) {
        const size_t it = base + (size_t)sp * p.qmax + qi;
        const float m = p.part_ml[it * 2];
        if (m == -INFINITY) continue;
        const float w = expf(m - M);
        L += p.part_ml[it * 2 + 1] * w;
        O += p.part_o[it * HD + d] * w;
      }
    }
    const int row = row0 + qi / G, h = kvh * G + qi % G;
    Store<T>::store((T*)p.out, Tile<T>::off(row, h * HD + d, p.H * HD), L > 0.f ? O / L : 0.f);
  }
}

hipError_t launch_rope_table(float2* tab, int n_pos, int half, double theta, hipStream_t s) {
  if (n_pos <= 0 || half <= 0) return hipErrorInvalidValue;
  const size_t n = (size_t)n_pos * half;
  const int blocks = (int)std::min<size_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(rope_table_kernel, dim3(blocks), dim3(256), 0, s, tab, n_pos, half, theta);
  return hipGetLastError();
}

template <typename T, int HD>
static hipError_t launch_attn_t(const AttnParams& p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  const size_t lds = attn_lds_bytes(HD, sizeof(T), p.qmax);
  static size_t attr_bytes = 64 * 1024;     // launches above the default limit raise it first
  if (lds > attr_bytes) {
    hipError_t e = hipFuncSetAttribute((const void*)attention_kernel<T, HD>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_bytes = lds;
  }
  const bool split = p.splits > 1;
  launch_k(attention_kernel<T, HD>, dim3(p.nrb * p.KV, p.splits), dim3(256), (uint32_t)lds, s, e0,
           split ? nullptr : e1, p);
  if (split) launch_k(attn_merge_kernel<T, HD>, dim3(p.nrb * p.KV), dim3(256), 0, s, nullptr, e1, p);
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, const AttnParams& p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (p.nrb <= 0) return hipSuccess;
  if (p.qmax > ATTN_QMAX) return hipErrorInvalidValue;
  if (p.keys_per_split % 64 || p.keys_per_split > ATTN_BT_CAP * 16) return hipErrorInvalidValue;
  const dim3 grid(p.nrb * p.KV, p.splits);
  if (dtype == 0) {
    // a split item's last workgroup merges: every split needs the counter, and
    // the merge holds at most ATTN_MAX_SPLITS partials per query
    if (p.splits > 1 && (!p.cnt || p.splits > ATTN_MAX_SPLITS)) return hipErrorInvalidValue;
    // four waves per workgroup for large grids (hd 64: 1024 or more
    // workgroups, hd 128: 2048): two then share a CU, and one's start and
    // merge overlap the other's stream.  13B B = 64 (2560 verify and 1024
    // draft workgroups): step 19.73 -> 18.38 ms; 7B paged B = 32 (1024
    // verify workgroups) is 0.7 % slower with four, so keeps eight.  Split
    // hd 128 items (7B B = 1: a few hundred keys per split) also take four:
    // a two-round key-group merge instead of three, 14.2 -> 13.9 us per
    // layer (with twice the splits on them, 14.8)
    const bool many = grid.x * grid.y >= (p.hd == 64 ? 1024u : 2048u) || (p.hd == 128 && p.splits > 1);
    if (p.hd == 64) {
      if (many) launch_k(attention_mfma_kernel<64, 4>, grid, dim3(64 * 4), 0, s, e0, e1, p);
      else launch_k(attention_mfma_kernel<64, 8>, grid, dim3(64 * 8), 0, s, e0, e1, p);
    } else if (p.hd == 128) {
      if (many) launch_k(attention_mfma_kernel<128, 4>, grid, dim3(64 * 4), 0, s, e0, e1, p);
      else launch_k(attention_mfma_kernel<128, 8>, grid, dim3(64 * 8), 0, s, e0, e1, p);
    } else {
      return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  if (p.hd == 64) return launch_attn_t<float, 64>(p, s, e0, e1);
  if (p.hd == 128) return launch_attn_t<float, 128>(p, s, e0, e1);
  return hipErrorInvalidValue;
}

size_t attention_lds_bytes(int hd, int esz, int qmax) { return attn_lds_bytes(hd, esz, qmax); }

}  // namespace sd
