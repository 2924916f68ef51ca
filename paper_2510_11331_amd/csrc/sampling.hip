// Vocabulary-wide row kernels: target softmax, draft sampling, speculative
// acceptance with residual / reward resampling, and the KV commit.
//
// Speculative sampling (Section II-A, after Leviathan et al.): draft t_i is
// accepted with probability min(1, p_i(t_i) / q_i(t_i)); the first rejected
// position is resampled from norm(max(0, p - q)); after gamma acceptances a
// reward token is drawn from p_{gamma+1}.
//
// Decisions are bit-reproducible given the float32 distributions and uint32
// uniforms, whatever the reduction order:
//   accept   iff  fl32(u * q(t)) < p(t),  u = (r >> 8) 2^-24 (exact float32);
//   sample   W_j = floor(w_j 2^40) (exact), S = sum W_j (integer, order-free),
//            T = floor(S r / 2^32) from 32-bit halves, smallest j with
//            prefix_j > T;
//   residual w_j = max(0, p_j - q_j) with a correctly rounded float32 subtract.
//
// A row (up to 32768 entries) is held in registers by one 1024-thread
// workgroup: for sampling each thread owns 32 consecutive entries (so the
// prefix sum in index order is one block scan of per-thread totals); the
// plain softmax uses a strided float4 layout for coalescing.  All loads of a
// row are issued before any is used.
#include "sd_internal.h"

namespace sd {

constexpr int RT = 1024;          // threads of a row kernel
constexpr int NW = RT / 64;       // waves
constexpr int SEG = 32;           // consecutive entries per thread in sampling kernels
constexpr int SV = SEG / 4;       // float4 per thread in the strided layout (V <= RT * 4 * SV)

__device__ __forceinline__ float wmax(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wsum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ float block_max(float v, float* red) {
  v = wmax(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) r = fmaxf(r, red[w]);
  return r;
}
__device__ float block_sum(float v, float* red) {
  v = wsum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) r += red[w];
  return r;
}

// arg-max with the lowest index on ties
__device__ int block_argmax(float v, int i, float* redv, int* redi) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(v, o);
    const int oi = __shfl_xor(i, o);
    if (ov > v || (ov == v && oi < i)) { v = ov; i = oi; }
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) { redv[threadIdx.x >> 6] = v; redi[threadIdx.x >> 6] = i; }
  __syncthreads();
  float bv = redv[0];
  int bi = redi[0];
#pragma unroll
  for (int w = 1; w < NW; ++w)
    if (redv[w] > bv || (redv[w] == bv && redi[w] < bi)) { bv = redv[w]; bi = redi[w]; }
  return bi;
}

// exclusive prefix of per-thread uint64 values in thread order; *total = sum
__device__ uint64_t block_excl_scan(uint64_t v, uint64_t* red, uint64_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned long long x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned long long y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  __syncthreads();
  if (lane == 63) red[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t a = 0;
    for (int w = 0; w < NW; ++w) { const uint64_t t = red[w]; red[w] = a; a += t; }
    red[NW] = a;
  }
  __syncthreads();
  *total = red[NW];
  return red[wave] + x - v;
}

__device__ __forceinline__ uint64_t fixed40(float w) {
  // w >= 0; w * 2^40 is exact in float32, truncation is the floor
  return w > 0.f ? (uint64_t)(w * 1099511627776.0f) : 0ull;
}

// thread-contiguous segment of a row: entries [SEG*t, SEG*t + SEG) (0 beyond V)
__device__ __forceinline__ void load_seg(const float* row, int V, float (&v)[SEG]) {
  const int j0 = threadIdx.x * SEG;
  if (j0 + SEG <= V && (V & 3) == 0) {
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      const float4 x = *(const float4*)(row + j0 + 4 * k);
      v[4 * k] = x.x; v[4 * k + 1] = x.y; v[4 * k + 2] = x.z; v[4 * k + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < SEG; ++k) v[k] = j0 + k < V ? row[j0 + k] : 0.f;
  }
}

// Integer inverse-CDF draw over the weights w (this thread's segment);
// returns -1 if S == 0.
__device__ int seg_sample(const float (&w)[SEG], uint32_t r, uint64_t* red, int* result) {
  uint64_t local = 0;
#pragma unroll
  for (int k = 0; k < SEG; ++k) local += fixed40(w[k]);
  if (threadIdx.x == 0) *result = -1;
  uint64_t S;
  const uint64_t lo = block_excl_scan(local, red, &S);
  if (S == 0) return -1;
  const uint64_t T = (S >> 32) * (uint64_t)r + (((S & 0xffffffffull) * (uint64_t)r) >> 32);
  if (T >= lo && T < lo + local) {                // this thread's segment holds the draw
    int hit = SEG - 1;
    uint64_t pre = lo;
#pragma unroll
    for (int k = 0; k < SEG; ++k) {                // smallest k with lo + prefix_k > T
      pre += fixed40(w[k]);
      if (pre > T) { hit = k; break; }
    }
    *result = threadIdx.x * SEG + hit;
  }
  __syncthreads();
  return *result;
}

__global__ __launch_bounds__(RT) void softmax_kernel(SoftmaxParams p) {
  __shared__ float red[NW];
  const float* z = p.z + (size_t)blockIdx.x * p.V;
  float* out = p.p + (size_t)blockIdx.x * p.V;
  const int V4 = p.V >> 2;
  float4 x[SV];
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    const int i = threadIdx.x + RT * k;
    x[k] = i < V4 ? ((const float4*)z)[i] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
  }
  if (p.greedy) {
    if (out != z)
#pragma unroll
      for (int k = 0; k < SV; ++k) {
        const int i = threadIdx.x + RT * k;
        if (i < V4) ((float4*)out)[i] = x[k];
      }
    return;
  }
  float m = -INFINITY;
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    x[k].x *= p.inv_tau; x[k].y *= p.inv_tau; x[k].z *= p.inv_tau; x[k].w *= p.inv_tau;
    m = fmaxf(m, fmaxf(fmaxf(x[k].x, x[k].y), fmaxf(x[k].z, x[k].w)));
  }
  m = block_max(m, red);
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    x[k].x = expf(x[k].x - m); x[k].y = expf(x[k].y - m); x[k].z = expf(x[k].z - m); x[k].w = expf(x[k].w - m);
    s += (x[k].x + x[k].y) + (x[k].z + x[k].w);
  }
  s = block_sum(s, red);
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    const int i = threadIdx.x + RT * k;
    if (i < V4) ((float4*)out)[i] = make_float4(x[k].x / s, x[k].y / s, x[k].z / s, x[k].w / s);
  }
}

__global__ __launch_bounds__(RT) void draft_sample_kernel(DraftSampleParams p) {
  __shared__ float red[NW];
  __shared__ int redi[NW];
  __shared__ uint64_t redu[NW + 1];
  __shared__ int result;
  const int b = blockIdx.x;
  const float* z = p.z + (size_t)b * p.V;
  float* q = p.q + ((size_t)b * p.gamma + p.i) * p.V;
  const int j0 = threadIdx.x * SEG;
  float v[SEG];
  load_seg(z, p.V, v);
  int tok;
  if (p.greedy) {
    float bv = -INFINITY;
    int bi = 0x7fffffff;
#pragma unroll
    for (int k = 0; k < SEG; ++k)
      if (j0 + k < p.V && v[k] > bv) { bv = v[k]; bi = j0 + k; }
    tok = block_argmax(bv, bi, red, redi);
    if (tok == 0x7fffffff) tok = 0;
#pragma unroll
    for (int k = 0; k < SEG; ++k)
      if (j0 + k < p.V) q[j0 + k] = v[k];
  } else {
    float m = -INFINITY;
#pragma unroll
    for (int k = 0; k < SEG; ++k) {
      v[k] *= p.inv_tau;
      if (j0 + k < p.V) m = fmaxf(m, v[k]);
    }
    m = block_max(m, red);
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < SEG; ++k) {
      v[k] = j0 + k < p.V ? expf(v[k] - m) : 0.f;
      s += v[k];
    }
    s = block_sum(s, red);
#pragma unroll
    for (int k = 0; k < SEG; ++k) {
      v[k] = v[k] / s;
      if (j0 + k < p.V) q[j0 + k] = v[k];
    }
    const uint32_t r = p.u[(size_t)b * (2 * p.gamma + 1) + p.i];
    tok = seg_sample(v, r, redu, &result);
    if (tok < 0) tok = 0;                       // no integer mass: impossible for a softmax row
  }
  if (threadIdx.x == 0) p.draft_tok[b * p.gamma + p.i] = tok;
}

__device__ int row_argmax(const float* row, int V, float* red, int* redi) {
  float v[SEG];
  load_seg(row, V, v);
  const int j0 = threadIdx.x * SEG;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
#pragma unroll
  for (int k = 0; k < SEG; ++k)
    if (j0 + k < V && v[k] > bv) { bv = v[k]; bi = j0 + k; }
  const int r = block_argmax(bv, bi, red, redi);
  return r == 0x7fffffff ? 0 : r;
}

__global__ __launch_bounds__(RT) void accept_kernel(AcceptParams p) {
  __shared__ float red[NW];
  __shared__ int redi[NW];
  __shared__ uint64_t redu[NW + 1];
  __shared__ int result, s_a;
  const int b = blockIdx.x, g = p.gamma, V = p.V;
  const int32_t* dt = p.draft_tok + (size_t)b * g;
  const float* q = p.q + (size_t)b * g * V;
  const float* pp = p.p + (size_t)b * (g + 1) * V;
  const uint32_t* u = p.u + (size_t)b * (2 * g + 1);
  int a = g, y = 0;
  if (p.greedy) {
    for (int i = 0; i < g; ++i) {
      const int am = row_argmax(pp + (size_t)i * V, V, red, redi);
      if (dt[i] != am) { a = i; y = am; break; }
    }
    if (a == g) y = row_argmax(pp + (size_t)g * V, V, red, redi);
  } else {
    if (threadIdx.x == 0) {
      int aa = g;
      for (int i = 0; i < g; ++i) {
        const int t = dt[i];
        bool ok = false;
        if (t >= 0 && t < V) {
          const float ui = (float)(u[g + i] >> 8) * 5.9604644775390625e-08f;   // * 2^-24, exact
          ok = __fmul_rn(ui, q[(size_t)i * V + t]) < pp[(size_t)i * V + t];
        } else if (p.err) {
          atomicOr(p.err, ERR_BAD_TOKEN);
        }
        if (!ok) { aa = i; break; }
      }
      s_a = aa;
    }
    __syncthreads();
    a = s_a;
    const uint32_t r = u[2 * g];
    float w[SEG];
    load_seg(pp + (size_t)a * V, V, w);
    if (a < g) {
      float res[SEG];
      load_seg(q + (size_t)a * V, V, res);
#pragma unroll
      for (int k = 0; k < SEG; ++k) {
        const float d = __fsub_rn(w[k], res[k]);
        res[k] = d > 0.f ? d : 0.f;
      }
      y = seg_sample(res, r, redu, &result);
      if (y < 0) y = seg_sample(w, r, redu, &result);      // residual without integer mass
    } else {
      y = seg_sample(w, r, redu, &result);
    }
    if (y < 0) y = 0;
  }
  for (int i = threadIdx.x; i <= g; i += RT)
    p.out_tok[(size_t)b * (g + 1) + i] = i < a ? dt[i] : (i == a ? y : -1);
  if (threadIdx.x == 0) p.n_acc[b] = a;
}

__global__ void commit_kernel(CommitParams p) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= p.B) return;
  const int g = p.gamma;
  int a = p.n_acc[b];
  if (a < 0 || a > g) {
    atomicOr(p.err, ERR_BAD_ACCEPT);
    a = a < 0 ? 0 : g;
  }
  const int slot = p.slots[b];
  if (slot < 0 || slot >= p.n_slots) {
    atomicOr(p.err, ERR_BAD_TOKEN);
    return;
  }
  int32_t* st = p.state + (size_t)slot * ST_N;
  const int32_t* ot = p.out_tok + (size_t)b * (g + 1);
  st[ST_LEN] = st[ST_LEN] + a + 1;
  st[ST_X0] = ot[a];
  st[ST_PEND] = a == g ? ot[g - 1] : -1;
}

hipError_t launch_softmax(const SoftmaxParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if (p.V > RT * SEG || (p.V & 3)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(softmax_kernel, dim3(p.M), dim3(RT), 0, s, p);
  return hipGetLastError();
}
hipError_t launch_draft_sample(const DraftSampleParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  if (p.V > RT * SEG) return hipErrorInvalidValue;
  hipLaunchKernelGGL(draft_sample_kernel, dim3(p.B), dim3(RT), 0, s, p);
  return hipGetLastError();
}
hipError_t launch_accept(const AcceptParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  if (p.V > RT * SEG) return hipErrorInvalidValue;
  hipLaunchKernelGGL(accept_kernel, dim3(p.B), dim3(RT), 0, s, p);
  return hipGetLastError();
}
hipError_t launch_commit(const CommitParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  hipLaunchKernelGGL(commit_kernel, dim3((p.B + 255) / 256), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace sd
