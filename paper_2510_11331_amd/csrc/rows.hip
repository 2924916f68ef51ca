// Row set-up + embedding + RMSNorm, and plain RMSNorm.
//
// The rows of a pass are derived on the device from the slot state, so a
// step needs no host round trip:
//   verify      row b*(gamma+1)+j: x0 (j = 0) or draft token j-1, position P+j
//               (Section II-A: the verify model takes the bonus token and the
//               gamma new drafts);
//   draft first rows 2b, 2b+1: the pending accepted draft (if any) at P-1,
//               then x0 at P;
//   draft next  row b: draft token i-1 at position P+i;
//   prefill     rows written by the host.
// A row with position -1 is inactive: zero activations, no KV write.
#include "sd_internal.h"

namespace sd {

constexpr int RV = 8;   // at most 8 float4 per thread: rows of up to 8192 entries stay in registers

__device__ __forceinline__ float block_sum256(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

template <typename T> struct Vec4;
template <> struct Vec4<bf16_t> {
  __device__ __forceinline__ static float4 load(const bf16_t* p, int i4) {
    const uint2 u = ((const uint2*)p)[i4];
    return make_float4(bf2f((bf16_t)(u.x & 0xffff)), bf2f((bf16_t)(u.x >> 16)), bf2f((bf16_t)(u.y & 0xffff)),
                       bf2f((bf16_t)(u.y >> 16)));
  }
  // four consecutive elements at element offset off (a multiple of 4)
  __device__ __forceinline__ static void store_at(bf16_t* p, size_t off, float4 v) {
    *(uint2*)(p + off) = make_uint2((uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16),
                                    (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16));
  }
};
template <> struct Vec4<f16_t> {
  __device__ __forceinline__ static void store_at(f16_t* p, size_t off, float4 v) {
    *(uint2*)(p + off) = make_uint2((uint32_t)f2h(v.x) | ((uint32_t)f2h(v.y) << 16),
                                    (uint32_t)f2h(v.z) | ((uint32_t)f2h(v.w) << 16));
  }
};
template <> struct Vec4<float> {
  __device__ __forceinline__ static float4 load(const float* p, int i4) { return ((const float4*)p)[i4]; }
  __device__ __forceinline__ static void store_at(float* p, size_t off, float4 v) { *(float4*)(p + off) = v; }
};

// Four gains as stored (bf16: 8 bytes, fp32: 16), loaded with the row at the
// start of a kernel so that the norm does not wait on a load after its
// reduction (RMSNorm 4.2 -> 3.3 us at 40 x 4096)
template <typename TW> struct Gain4;
template <> struct Gain4<bf16_t> {
  uint2 q;
  __device__ __forceinline__ void load(const bf16_t* p, int i4) { q = ((const uint2*)p)[i4]; }
  __device__ __forceinline__ float4 get() const {
    return make_float4(bf2f((bf16_t)(q.x & 0xffff)), bf2f((bf16_t)(q.x >> 16)), bf2f((bf16_t)(q.y & 0xffff)),
                       bf2f((bf16_t)(q.y >> 16)));
  }
};
template <> struct Gain4<float> {
  float4 q;
  __device__ __forceinline__ void load(const float* p, int i4) { q = ((const float4*)p)[i4]; }
  __device__ __forceinline__ float4 get() const { return q; }
};
template <typename TW, int R>
__device__ __forceinline__ void load_gains(Gain4<TW> (&g)[R], const TW* gain, int d4) {
#pragma unroll
  for (int k = 0; k < R; ++k)
    if (threadIdx.x + 256 * k < d4) g[k].load(gain, threadIdx.x + 256 * k);
}

// row r of out (MFMA-tile layout) = x / sqrt(mean(x^2) + eps) * gain for a
// register-resident row x (float4 i of the row is v[k], i = threadIdx.x + 256 k,
// R of them per thread) and its gains g (loaded by load_gains); TW: storage
// type of the gains (the model's weights), TA: of the output (the
// matrix-product operands: fp16 for a bf16 model)
template <typename TW, typename TA, int R>
__device__ void norm_store(const float4 (&v)[R], const Gain4<TW> (&g)[R], int d, TA* out, int r, float eps,
                           float* red) {
  const int d4 = d >> 2;
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < R; ++k)
    if (threadIdx.x + 256 * k < d4) ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
  ss = block_sum256(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + 256 * k;
    if (i < d4) {
      const float4 gk = g[k].get();
      Vec4<TA>::store_at(out, Tile<TA>::off(r, 4 * i, d),
                        make_float4(v[k].x * inv * gk.x, v[k].y * inv * gk.y, v[k].z * inv * gk.z, v[k].w * inv * gk.w));
    }
  }
}

template <typename T, typename TA, int R>
__global__ __launch_bounds__(256) void rows_embed_kernel(RowsParams p) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  Gain4<T> g[R];
  load_gains<T, R>(g, (const T*)p.gain, p.d >> 2);
  int tok = 0, pos = -1, slot = 0;
  if (p.mode == ROWS_PREFILL) {
    tok = p.row_tok[r];
    pos = p.row_pos[r];
    slot = p.row_slot[r];
  } else {
    int b, j = 0;
    if (p.mode == ROWS_VERIFY) { b = r / (p.gamma + 1); j = r % (p.gamma + 1); }
    else if (p.mode == ROWS_DRAFT_FIRST) { b = r >> 1; j = r & 1; }
    else b = r;
    slot = p.slots[b];
    if (slot < 0 || slot >= p.n_slots) {          // bad slot id: inactive row, flagged
      if (threadIdx.x == 0) {
        atomicOr(p.err, ERR_BAD_TOKEN);
        p.row_tok[r] = 0;
        p.row_pos[r] = -1;
        p.row_slot[r] = 0;
        p.row_blk[r] = -1;
      }
      for (int i = threadIdx.x; i < p.d; i += 256) {
        p.x[(size_t)r * p.d + i] = 0.f;
        Store<TA>::store((TA*)p.xn, Tile<TA>::off(r, i, p.d), 0.f);
      }
      return;
    }
    if (p.row_bt && j == 0)   // the task's block-table row, for this pass's attention
      for (int i = threadIdx.x; i < p.mbps; i += 256)
        p.row_bt[(size_t)b * p.mbps + i] = p.block_table[(size_t)slot * p.mbps + i];
    const int32_t* st = p.state + (size_t)slot * ST_N;
    const int P = st[ST_LEN];
    if (p.mode == ROWS_VERIFY) {
      tok = j == 0 ? st[ST_X0] : p.draft_tok[b * p.gamma + j - 1];
      pos = P + j;
    } else if (p.mode == ROWS_DRAFT_FIRST) {
      if (j == 0) {
        tok = st[ST_PEND];
        pos = tok >= 0 ? P - 1 : -1;
      } else {
        tok = st[ST_X0];
        pos = P;
      }
    } else {
      tok = p.draft_tok[b * p.gamma + p.step_i - 1];
      pos = P + p.step_i;
    }
    if (threadIdx.x == 0) {
      p.row_tok[r] = tok;
      p.row_pos[r] = pos;
      p.row_slot[r] = slot;
    }
  }
  if (threadIdx.x == 0) {
    // KV block of this row for every layer of the pass; a write beyond the
    // slot's capacity is skipped and flagged
    int blk = -1;
    if (pos >= 0) {
      if (pos < p.state[(size_t)slot * ST_N + ST_CAP]) blk = p.block_table[(size_t)slot * p.mbps + pos / 16];
      else atomicOr(p.err, ERR_KV_OVERFLOW);
    }
    p.row_blk[r] = blk;
  }
  if (pos >= 0 && (tok < 0 || tok >= p.V)) {
    if (threadIdx.x == 0) atomicOr(p.err, ERR_BAD_TOKEN);
    tok = 0;
  }
  const int d4 = p.d >> 2;
  const T* e = (const T*)p.embed + (size_t)tok * p.d;
  float4* x = (float4*)(p.x + (size_t)r * p.d);
  float4 v[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + 256 * k;
    v[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (i < d4 && pos >= 0) v[k] = Vec4<T>::load(e, i);
  }
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + 256 * k;
    if (i < d4) x[i] = v[k];
  }
  norm_store<T, TA, R>(v, g, p.d, (TA*)p.xn, r, p.eps, red);
}

// NS: number of K-split partial sums to add into the residual row first (all
// loads are issued before the first add; the adds follow split order)
template <typename T, typename TA, int NS, int R>
__global__ __launch_bounds__(256) void rmsnorm_kernel(NormParams p) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const size_t rin = (size_t)r * p.src_stride + p.src_off;
  float4* x = (float4*)(p.x + rin * p.d);
  const int d4 = p.d >> 2;
  Gain4<T> g[R];
  load_gains<T, R>(g, (const T*)p.gain, d4);
  float4 v[R];
  float4 a[NS > 0 ? NS : 1][R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int i = threadIdx.x + 256 * k;
    v[k] = i < d4 ? x[i] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int sp = 0; sp < NS; ++sp)
      a[sp][k] = i < d4 ? ((const float4*)(p.part + ((size_t)sp * p.rows_in + rin) * p.d))[i]
                        : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  if constexpr (NS > 0) {
#pragma unroll
    for (int k = 0; k < R; ++k) {
#pragma unroll
      for (int sp = 0; sp < NS; ++sp) {
        v[k].x += a[sp][k].x;
        v[k].y += a[sp][k].y;
        v[k].z += a[sp][k].z;
        v[k].w += a[sp][k].w;
      }
      const int i = threadIdx.x + 256 * k;
      if (i < d4) x[i] = v[k];
    }
  }
  norm_store<T, TA, R>(v, g, p.d, (TA*)p.xn, r, p.eps, red);
}

// float4 per thread for a row of d entries: the smallest of 1, 2, 4, 5, 8
// that holds it (the registers a kernel holds follow d, not the largest d)
inline int rows_r(int d) {
  const int need = ((d >> 2) + 255) / 256;
  return need <= 1 ? 1 : need <= 2 ? 2 : need <= 4 ? 4 : need <= 5 ? 5 : 8;
}
#define SD_ROWS_R(R_EXPR, CALL)                  \
  switch (R_EXPR) {                              \
    case 1: { constexpr int R = 1; CALL; } break; \
    case 2: { constexpr int R = 2; CALL; } break; \
    case 4: { constexpr int R = 4; CALL; } break; \
    case 5: { constexpr int R = 5; CALL; } break; \
    default: { constexpr int R = 8; CALL; } break; \
  }

hipError_t launch_rows_embed(int dtype, const RowsParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if ((p.d & 3) || p.d > 256 * 4 * RV) return hipErrorInvalidValue;
  if (dtype == 0) SD_ROWS_R(rows_r(p.d), hipLaunchKernelGGL((rows_embed_kernel<bf16_t, f16_t, R>), dim3(p.M), dim3(256), 0, s, p))
  else SD_ROWS_R(rows_r(p.d), hipLaunchKernelGGL((rows_embed_kernel<float, float, R>), dim3(p.M), dim3(256), 0, s, p))
  return hipGetLastError();
}

template <int NS>
static hipError_t launch_norm_ns(int dtype, const NormParams& p, hipStream_t s) {
  if (dtype == 0) SD_ROWS_R(rows_r(p.d), hipLaunchKernelGGL((rmsnorm_kernel<bf16_t, f16_t, NS, R>), dim3(p.M), dim3(256), 0, s, p))
  else SD_ROWS_R(rows_r(p.d), hipLaunchKernelGGL((rmsnorm_kernel<float, float, NS, R>), dim3(p.M), dim3(256), 0, s, p))
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int dtype, const NormParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if ((p.d & 3) || p.d > 256 * 4 * RV) return hipErrorInvalidValue;
  const int ns = p.part ? p.nsplit : 0;
  switch (ns) {
    case 0: return launch_norm_ns<0>(dtype, p, s);
    case 1: return launch_norm_ns<1>(dtype, p, s);
    case 2: return launch_norm_ns<2>(dtype, p, s);
    case 3: return launch_norm_ns<3>(dtype, p, s);
    case 4: return launch_norm_ns<4>(dtype, p, s);
    case 5: return launch_norm_ns<5>(dtype, p, s);
    case 6: return launch_norm_ns<6>(dtype, p, s);
    default: return hipErrorInvalidValue;
  }
}

__global__ void fill_i32_kernel(int32_t* p, int32_t v, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = v;
}

hipError_t launch_fill_i32(int32_t* p, int32_t v, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int blocks = (int)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(blocks), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

}  // namespace sd
