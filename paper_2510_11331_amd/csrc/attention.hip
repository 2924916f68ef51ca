// Rotary embedding + KV append, and causal multi-query attention over the
// paged KV cache (Section II-A: eq. d_kv grows the cache by concatenation;
// eq. d_atte / f21 attend with softmax(q K^T / sqrt(d0)) V).
//
// Paged layout of one layer's pool: [block][K|V][kv_head][16 tokens][hd] in
// the model dtype; a slot's block table maps position / 16 to a block.
//
// Attention work item = (row block, kv head, key split).  A row block is a
// run of consecutive rows of one task (the gamma+1 verify rows of a task, its
// 1-2 draft rows, or up to 64/G prefill rows); all G query heads of the kv
// head and all rows of the block share every K/V tile, which is staged in
// LDS 64 keys at a time.  Query i only sees keys at positions <= its own.
// Each work item keeps an online softmax (running max, running sum,
// rescaled output); when the keys are split, partial (max, sum, output)
// triples go to a workspace and the last-arriving workgroup of the
// (row block, kv head) merges them in split order.
#include "sd_internal.h"

namespace sd {

template <typename T>
__global__ __launch_bounds__(256) void rope_append_kernel(RopeParams p) {
  const int r = blockIdx.x;
  const int pos = p.row_pos[r];
  if (pos < 0) return;
  const int slot = p.row_slot[r];
  const int hd = p.hd, half = hd / 2;
  const int Nq = p.H * hd, Nk = p.KV * hd;
  const float* src = p.qkv + (size_t)r * (Nq + 2 * Nk);
  const bool ok = pos < p.state[slot * ST_N + ST_CAP];
  const int blk = ok ? p.block_table[(size_t)slot * p.mbps + pos / 16] : 0;
  const int off = pos % 16;
  T* kv = (T*)p.kv;
  const size_t kbase = (((size_t)blk * 2 + 0) * p.KV) * 16 * hd + (size_t)off * hd;
  const size_t vbase = (((size_t)blk * 2 + 1) * p.KV) * 16 * hd + (size_t)off * hd;

  // thread -> frequency index i (fixed), heads strided; angle in float64
  const int nh = p.H + p.KV;
  for (int idx = threadIdx.x; idx < nh * half; idx += blockDim.x) {
    const int i = idx % half, h = idx / half;
    const double ang = (double)pos * pow(p.theta, -2.0 * (double)i / (double)hd);
    double sd_, cd_;
    sincos(ang, &sd_, &cd_);
    const float c = (float)cd_, s = (float)sd_;
    if (h < p.H) {
      const float a = src[h * hd + i], b = src[h * hd + i + half];
      float* q = p.q + (size_t)r * Nq + h * hd;
      q[i] = a * c - b * s;
      q[i + half] = a * s + b * c;
    } else if (ok) {
      const int kh = h - p.H;
      const float a = src[Nq + kh * hd + i], b = src[Nq + kh * hd + i + half];
      Store<T>::store(kv, kbase + (size_t)kh * 16 * hd + i, a * c - b * s);
      Store<T>::store(kv, kbase + (size_t)kh * 16 * hd + i + half, a * s + b * c);
    }
  }
  if (ok) {
    for (int idx = threadIdx.x; idx < Nk; idx += blockDim.x) {
      const int kh = idx / hd, d = idx % hd;
      Store<T>::store(kv, vbase + (size_t)kh * 16 * hd + d, src[Nq + Nk + idx]);
    }
  } else if (threadIdx.x == 0) {
    atomicOr(p.err, ERR_KV_OVERFLOW);
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

template <typename T> struct KvT;
template <> struct KvT<bf16_t> {
  static constexpr int KST_PAD = 2;   // K row stride hd+2 elements: 32-bit reads hit distinct banks
  static constexpr int EPU = 8;       // elements per 16-byte unit
};
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
  __shared__ int s_last;

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
  const int slot = p.row_slot[row0];
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
  const int32_t* bt = p.block_table + (size_t)slot * p.mbps;

  for (int c = k_begin; c < k_end; c += 64) {
    __syncthreads();
    // stage 64 keys of K and V
    constexpr int UPR = HD / EPU;      // 16-byte units per key row
    for (int idx = tid; idx < 64 * UPR; idx += 256) {
      const int j = idx / UPR, e = (idx % UPR) * EPU;
      const int kp = c + j;
      uint4 kk = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
      if (kp < k_end) {
        const int blk = bt[kp / 16];
        const size_t base = (((size_t)blk * 2) * p.KV + kvh) * 16 * HD + (size_t)(kp % 16) * HD + e;
        const size_t vbase = base + (size_t)p.KV * 16 * HD;
        kk = *(const uint4*)(kv + base);
        vv = *(const uint4*)(kv + vbase);
      }
      uint32_t* kd = (uint32_t*)(Ks + j * KST + e);   // KST*esz is a multiple of 4
      kd[0] = kk.x; kd[1] = kk.y; kd[2] = kk.z; kd[3] = kk.w;
      *(uint4*)(Vs + j * HD + e) = vv;
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
    Store<T>::store((T*)p.out, (size_t)row * Hq + h * HD + dd, val);
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
  __threadfence();
  __syncthreads();
  if (tid == 0) s_last = atomicAdd(&p.counters[rbk], 1) == p.splits - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();
#pragma unroll
  for (int k = 0; k < QPT; ++k) {
    const int qi = qg + NQG * k;
    if (qi >= Qn) continue;
    float M = -INFINITY;
    for (int sp = 0; sp < p.splits; ++sp) M = fmaxf(M, p.part_ml[((item + sp) * qmax + qi) * 2]);
    float L = 0.f, O = 0.f;
    if (M != -INFINITY) {
      for (int sp = 0; sp < p.splits; ++sp) {
        const float m = p.part_ml[((item + sp) * qmax + qi) * 2];
        if (m == -INFINITY) continue;
        const float w = expf(m - M);
        L += p.part_ml[((item + sp) * qmax + qi) * 2 + 1] * w;
        O += p.part_o[((item + sp) * qmax + qi) * HD + dd] * w;
      }
    }
    emit(qi, L > 0.f ? O / L : 0.f);
  }
  if (tid == 0) p.counters[rbk] = 0;
}

hipError_t launch_rope_append(int dtype, const RopeParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if (dtype == 0) hipLaunchKernelGGL(rope_append_kernel<bf16_t>, dim3(p.M), dim3(256), 0, s, p);
  else hipLaunchKernelGGL(rope_append_kernel<float>, dim3(p.M), dim3(256), 0, s, p);
  return hipGetLastError();
}

template <typename T, int HD>
static hipError_t launch_attn_t(const AttnParams& p, hipStream_t s) {
  const size_t lds = attn_lds_bytes(HD, sizeof(T), p.qmax);
  static size_t attr_bytes = 64 * 1024;     // launches above the default limit raise it first
  if (lds > attr_bytes) {
    hipError_t e = hipFuncSetAttribute((const void*)attention_kernel<T, HD>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_bytes = lds;
  }
  hipLaunchKernelGGL((attention_kernel<T, HD>), dim3(p.nrb * p.KV, p.splits), dim3(256), lds, s, p);
  return hipGetLastError();
}

hipError_t launch_attention(int dtype, const AttnParams& p, hipStream_t s) {
  if (p.nrb <= 0) return hipSuccess;
  if (p.qmax > ATTN_QMAX) return hipErrorInvalidValue;
  if (dtype == 0) {
    if (p.hd == 64) return launch_attn_t<bf16_t, 64>(p, s);
    if (p.hd == 128) return launch_attn_t<bf16_t, 128>(p, s);
  } else {
    if (p.hd == 64) return launch_attn_t<float, 64>(p, s);
    if (p.hd == 128) return launch_attn_t<float, 128>(p, s);
  }
  return hipErrorInvalidValue;
}

size_t attention_lds_bytes(int hd, int esz, int qmax) { return attn_lds_bytes(hd, esz, qmax); }

}  // namespace sd
