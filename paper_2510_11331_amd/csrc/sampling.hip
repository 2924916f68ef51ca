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
#include "sd_internal.h"

namespace sd {

constexpr int RB = 256;   // threads per row kernel

__device__ __forceinline__ float bmax(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}
__device__ __forceinline__ float bsum(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// arg-max over a row, lowest index on ties
__device__ int bargmax(const float* z, int V, float* redv, int* redi) {
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int j = threadIdx.x; j < V; j += RB) {
    const float v = z[j];
    if (v > bv) { bv = v; bi = j; }       // strided ascending: first hit is the lowest index
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o);
    const int oi = __shfl_xor(bi, o);
    if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) { redv[threadIdx.x >> 6] = bv; redi[threadIdx.x >> 6] = bi; }
  __syncthreads();
  float v = redv[0];
  int i = redi[0];
  for (int w = 1; w < 4; ++w)
    if (redv[w] > v || (redv[w] == v && redi[w] < i)) { v = redv[w]; i = redi[w]; }
  return i == 0x7fffffff ? 0 : i;
}

__device__ __forceinline__ uint64_t fixed40(float w) {
  // w >= 0; w * 2^40 is exact in float32, truncation is the floor
  return w > 0.f ? (uint64_t)(w * 1099511627776.0f) : 0ull;
}

// Integer inverse-CDF draw with weights wf(j), j < V; returns -1 if S == 0.
// Thread t owns the contiguous index range [t*seg, (t+1)*seg).
template <typename WF>
__device__ int block_sample(WF wf, int V, uint32_t r, uint64_t* part, int* result) {
  const int seg = (V + RB - 1) / RB;
  const int j0 = min(V, (int)threadIdx.x * seg), j1 = min(V, j0 + seg);
  uint64_t local = 0;
  for (int j = j0; j < j1; ++j) local += fixed40(wf(j));
  __syncthreads();
  part[threadIdx.x] = local;
  if (threadIdx.x == 0) *result = -1;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t acc = 0;
    for (int t = 0; t < RB; ++t) { const uint64_t v = part[t]; part[t] = acc; acc += v; }
    part[RB] = acc;
  }
  __syncthreads();
  const uint64_t S = part[RB];
  if (S == 0) return -1;
  const uint64_t T = (S >> 32) * (uint64_t)r + (((S & 0xffffffffull) * (uint64_t)r) >> 32);
  const uint64_t lo = part[threadIdx.x];
  if (T >= lo && T < lo + local) {
    uint64_t acc = lo;
    for (int j = j0; j < j1; ++j) {
      acc += fixed40(wf(j));
      if (acc > T) { *result = j; break; }
    }
  }
  __syncthreads();
  return *result;
}

// softmax(z / tau) of one row into out (may alias z)
__device__ void row_softmax(const float* z, float* out, int V, float inv_tau, float* red) {
  float m = -INFINITY;
  for (int j = threadIdx.x; j < V; j += RB) m = fmaxf(m, z[j] * inv_tau);
  m = bmax(m, red);
  float s = 0.f;
  for (int j = threadIdx.x; j < V; j += RB) s += expf(z[j] * inv_tau - m);
  s = bsum(s, red);
  __syncthreads();
  for (int j = threadIdx.x; j < V; j += RB) out[j] = expf(z[j] * inv_tau - m) / s;
  __syncthreads();
}

__global__ __launch_bounds__(RB) void softmax_kernel(SoftmaxParams p) {
  __shared__ float red[4];
  const float* z = p.z + (size_t)blockIdx.x * p.V;
  float* out = p.p + (size_t)blockIdx.x * p.V;
  if (p.greedy) {
    if (out != z)
      for (int j = threadIdx.x; j < p.V; j += RB) out[j] = z[j];
    return;
  }
  row_softmax(z, out, p.V, p.inv_tau, red);
}

__global__ __launch_bounds__(RB) void draft_sample_kernel(DraftSampleParams p) {
  __shared__ float red[4];
  __shared__ float redv[4];
  __shared__ int redi[4];
  __shared__ uint64_t part[RB + 1];
  __shared__ int result;
  const int b = blockIdx.x;
  const float* z = p.z + (size_t)b * p.V;
  float* q = p.q + ((size_t)b * p.gamma + p.i) * p.V;
  int tok;
  if (p.greedy) {
    for (int j = threadIdx.x; j < p.V; j += RB) q[j] = z[j];
    tok = bargmax(z, p.V, redv, redi);
  } else {
    row_softmax(z, q, p.V, p.inv_tau, red);
    const uint32_t r = p.u[(size_t)b * (2 * p.gamma + 1) + p.i];
    tok = block_sample([&](int j) { return q[j]; }, p.V, r, part, &result);
    if (tok < 0) tok = bargmax(z, p.V, redv, redi);    // no integer mass: cannot happen for a softmax row
  }
  if (threadIdx.x == 0) p.draft_tok[b * p.gamma + p.i] = tok;
}

__global__ __launch_bounds__(RB) void accept_kernel(AcceptParams p) {
  __shared__ float redv[4];
  __shared__ int redi[4];
  __shared__ uint64_t part[RB + 1];
  __shared__ int result, s_a, s_y;
  const int b = blockIdx.x, g = p.gamma, V = p.V;
  const int32_t* dt = p.draft_tok + (size_t)b * g;
  const float* q = p.q + (size_t)b * g * V;
  const float* pp = p.p + (size_t)b * (g + 1) * V;
  const uint32_t* u = p.u + (size_t)b * (2 * g + 1);
  int a = g, y = 0;
  if (p.greedy) {
    for (int i = 0; i < g; ++i) {
      const int am = bargmax(pp + (size_t)i * V, V, redv, redi);
      if (dt[i] != am) { a = i; y = am; break; }
    }
    if (a == g) y = bargmax(pp + (size_t)g * V, V, redv, redi);
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
    if (a < g) {
      const float* pa = pp + (size_t)a * V;
      const float* qa = q + (size_t)a * V;
      y = block_sample([&](int j) { const float d = __fsub_rn(pa[j], qa[j]); return d > 0.f ? d : 0.f; },
                       V, r, part, &result);
      if (y < 0) y = block_sample([&](int j) { return pa[j]; }, V, r, part, &result);
    } else {
      const float* pg = pp + (size_t)g * V;
      y = block_sample([&](int j) { return pg[j]; }, V, r, part, &result);
    }
    if (y < 0) y = 0;
  }
  if (threadIdx.x == 0) { s_y = y; }
  __syncthreads();
  for (int i = threadIdx.x; i <= g; i += RB)
    p.out_tok[(size_t)b * (g + 1) + i] = i < a ? dt[i] : (i == a ? s_y : -1);
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
  hipLaunchKernelGGL(softmax_kernel, dim3(p.M), dim3(RB), 0, s, p);
  return hipGetLastError();
}
hipError_t launch_draft_sample(const DraftSampleParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  hipLaunchKernelGGL(draft_sample_kernel, dim3(p.B), dim3(RB), 0, s, p);
  return hipGetLastError();
}
hipError_t launch_accept(const AcceptParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  hipLaunchKernelGGL(accept_kernel, dim3(p.B), dim3(RB), 0, s, p);
  return hipGetLastError();
}
hipError_t launch_commit(const CommitParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  hipLaunchKernelGGL(commit_kernel, dim3((p.B + 255) / 256), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace sd
