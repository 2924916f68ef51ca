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
// workgroup in a strided float4 layout (coalesced loads and stores); the
// prefix sums of a draw are taken in index order from wave scans.  All loads
// of a row are issued before any is used.
#include "sd_internal.h"

namespace sd {

constexpr int RT = 1024;          // threads of a row kernel
constexpr int NW = RT / 64;       // waves
constexpr int SV = 8;             // float4 per thread in the strided layout (V <= RT * 4 * SV)
static_assert(SV * NW % 64 == 0, "draft sampling scans SV * NW totals with one wave");

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

// floor(w 2^40) for 0 <= w < 2^23, exactly: x = w 2^40 is exact in float32;
// hi = floor(x / 2^32) and lo = x - hi 2^32 are exact too (when hi > 0,
// x >= 2^32 has an ulp of at least 2^9, so lo is a representable multiple of
// it below 2^32), and the float -> uint32 conversion of lo truncates = floors.
__device__ __forceinline__ uint64_t fixed40(float w) {
  if (!(w > 0.f)) return 0ull;
  const float x = w * 1099511627776.0f;
  const float hi = floorf(x * 2.3283064365386963e-10f);
  const float lo = x - hi * 4294967296.0f;
  return ((uint64_t)(uint32_t)hi << 32) | (uint64_t)(uint32_t)lo;
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

// x moved by a DPP pattern, 0 where the source lane is out of the row or
// the destination row is masked off
template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t x) {
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, CTRL, ROWS, 0xf, true);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), CTRL, ROWS, 0xf, true);
  return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

// inclusive scan of uint64 values over the 64 lanes of a wave (register-file
// moves: shifts by 1, 2, 4, 8 inside each 16-lane row, then the last lane of
// row 0 / 2 broadcast into rows 1 / 3 and of row 1 into rows 2, 3)
__device__ __forceinline__ uint64_t wave_incl_scan(uint64_t x) {
  x += dpp_u64<0x111, 0xf>(x);    // row_shr:1
  x += dpp_u64<0x112, 0xf>(x);    // row_shr:2
  x += dpp_u64<0x114, 0xf>(x);    // row_shr:4
  x += dpp_u64<0x118, 0xf>(x);    // row_shr:8
  x += dpp_u64<0x142, 0xa>(x);    // row_bcast:15 into rows 1, 3
  x += dpp_u64<0x143, 0xc>(x);    // row_bcast:31 into rows 2, 3
  return x;
}

// Strided float4 layout of a row (coalesced): thread t holds entries
// 4 (t + RT k) .. +3 for k < SV; entries past V read as `fill`.  Index order
// is k-major, then thread, then the 4 entries.
__device__ __forceinline__ void load_strided(const float* row, int V, float4 (&x)[SV], float fill) {
  const int V4 = V >> 2;
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    const int i = threadIdx.x + RT * k;
    x[k] = i < V4 ? ((const float4*)row)[i] : make_float4(fill, fill, fill, fill);
  }
}

// Arg-max of a strided row, lowest index on ties (entries are visited in
// increasing index, so a thread's first strict maximum is its lowest).
__device__ int strided_argmax(const float4 (&x)[SV], float* red, int* redi) {
  float bv = -INFINITY;
  int bi = 0x7fffffff;
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    const int j = 4 * (threadIdx.x + RT * k);
    if (x[k].x > bv) { bv = x[k].x; bi = j; }
    if (x[k].y > bv) { bv = x[k].y; bi = j + 1; }
    if (x[k].z > bv) { bv = x[k].z; bi = j + 2; }
    if (x[k].w > bv) { bv = x[k].w; bi = j + 3; }
  }
  const int r = block_argmax(bv, bi, red, redi);
  return r == 0x7fffffff ? 0 : r;
}

// Integer inverse-CDF draw over strided weights w (>= 0, zero past V) with
// uniform r; -1 if S = 0.  The prefix of W_j = floor(w_j 2^40) in index order
// comes from a wave scan of the per-thread sums of each chunk k and one scan
// over the (k, wave) totals.  Called by every thread of the workgroup.
__device__ int strided_sample(const float4 (&w)[SV], uint32_t r, uint64_t* pre, uint64_t* total, int* result) {
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  __syncthreads();                              // a previous draw's result has been read
  uint64_t L[SV], excl[SV];
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    L[k] = fixed40(w[k].x) + fixed40(w[k].y) + fixed40(w[k].z) + fixed40(w[k].w);
    const uint64_t inc = wave_incl_scan(L[k]);
    excl[k] = inc - L[k];
    if (lane == 63) pre[k * NW + wave] = inc;
  }
  if (t == 0) *result = -1;
  __syncthreads();
  if (wave == 0) {
    // exclusive prefix of the SV * NW totals in (k, wave) order
    constexpr int PER = SV * NW / 64;
    uint64_t a[PER], s = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) { a[e] = pre[PER * lane + e]; s += a[e]; }
    const uint64_t inc = wave_incl_scan(s);
    uint64_t run = inc - s;
#pragma unroll
    for (int e = 0; e < PER; ++e) { pre[PER * lane + e] = run; run += a[e]; }
    if (lane == 63) *total = inc;
  }
  __syncthreads();
  const uint64_t S = *total;
  const uint64_t T = (S >> 32) * (uint64_t)r + (((S & 0xffffffffull) * (uint64_t)r) >> 32);
#pragma unroll
  for (int k = 0; k < SV; ++k) {
    const uint64_t lo = pre[k * NW + wave] + excl[k];
    if (S > 0 && T >= lo && T < lo + L[k]) {      // this thread's 4 entries of chunk k hold the draw
      const float v[4] = {w[k].x, w[k].y, w[k].z, w[k].w};
      uint64_t c = lo;
      int hit = 3;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        c += fixed40(v[e]);
        if (c > T) { hit = e; break; }
      }
      *result = 4 * (t + RT * k) + hit;
    }
  }
  __syncthreads();
  return *result;
}

__global__ __launch_bounds__(RT) void draft_sample_kernel(DraftSampleParams p) {
  __shared__ float red[NW];
  __shared__ int redi[NW];
  __shared__ uint64_t pre[SV * NW];
  __shared__ uint64_t total;
  __shared__ int result;
  const int b = blockIdx.x, t = threadIdx.x;
  float4* q = (float4*)(p.q + ((size_t)b * p.gamma + p.i) * p.V);
  const int V4 = p.V >> 2;
  const uint32_t ur = p.u[(size_t)b * (2 * p.gamma + 1) + p.i];   // loaded with the row, used by the draw
  float4 x[SV];
  load_strided(p.z + (size_t)b * p.V, p.V, x, -INFINITY);
  int tok;
  if (p.greedy) {
#pragma unroll
    for (int k = 0; k < SV; ++k)
      if (t + RT * k < V4) q[t + RT * k] = x[k];
    tok = strided_argmax(x, red, redi);
  } else {
    float m = -INFINITY;
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      x[k].x *= p.inv_tau; x[k].y *= p.inv_tau; x[k].z *= p.inv_tau; x[k].w *= p.inv_tau;
      m = fmaxf(m, fmaxf(fmaxf(x[k].x, x[k].y), fmaxf(x[k].z, x[k].w)));
    }
    m = block_max(m, red);
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      x[k].x = expf(x[k].x - m); x[k].y = expf(x[k].y - m); x[k].z = expf(x[k].z - m); x[k].w = expf(x[k].w - m);
      sum += (x[k].x + x[k].y) + (x[k].z + x[k].w);
    }
    const float inv = 1.0f / block_sum(sum, red);
#pragma unroll
    for (int k = 0; k < SV; ++k) {
      x[k].x *= inv; x[k].y *= inv; x[k].z *= inv; x[k].w *= inv;
      if (t + RT * k < V4) q[t + RT * k] = x[k];
    }
    tok = strided_sample(x, ur, pre, &total, &result);
    if (tok < 0) tok = 0;                       // no integer mass: impossible for a softmax row
  }
  if (t == 0) p.draft_tok[b * p.gamma + p.i] = tok;
}

__global__ __launch_bounds__(RT) void accept_kernel(AcceptParams p) {
  __shared__ float red[NW];
  __shared__ int redi[NW];
  __shared__ uint64_t pre[SV * NW];
  __shared__ uint64_t total;
  __shared__ int result, s_a;
  const int b = blockIdx.x, g = p.gamma, V = p.V;
  const int32_t* dt = p.draft_tok + (size_t)b * g;
  const float* q = p.q + (size_t)b * g * V;
  const float* pp = p.p + (size_t)b * (g + 1) * V;
  const uint32_t* u = p.u + (size_t)b * (2 * g + 1);
  int a = g, y = 0;
  float4 w[SV];
  if (p.greedy) {
    for (int i = 0; i < g; ++i) {
      load_strided(pp + (size_t)i * V, V, w, -INFINITY);
      const int am = strided_argmax(w, red, redi);
      if (dt[i] != am) { a = i; y = am; break; }
    }
    if (a == g) {
      load_strided(pp + (size_t)g * V, V, w, -INFINITY);
      y = strided_argmax(w, red, redi);
    }
  } else {
    // the gamma ratio tests in parallel (lane i of wave 0 tests draft i, all
    // loads in one round trip); a is the first failing test, as in the
    // sequential rule, and only a bad token at position a is flagged (the
    // positions before it were accepted, the ones after it never examined)
    const uint32_t r = u[2 * g];
    if (threadIdx.x < 64) {
      const int i = threadIdx.x;
      const int t = i < g ? dt[i] : 0;
      const bool valid = i < g && t >= 0 && t < V;
      bool ok = false;
      if (valid) {
        const float ui = (float)(u[g + i] >> 8) * 5.9604644775390625e-08f;   // * 2^-24, exact
        ok = __fmul_rn(ui, q[(size_t)i * V + t]) < pp[(size_t)i * V + t];
      }
      const uint64_t fail = __ballot(i < g && !ok);
      const int aa = fail ? __ffsll((unsigned long long)fail) - 1 : g;
      if (i == aa && i < g && !valid && p.err) atomicOr(p.err, ERR_BAD_TOKEN);
      if (i == 0) s_a = aa;
    }
    __syncthreads();
    a = s_a;
    load_strided(pp + (size_t)a * V, V, w, 0.f);
    if (a < g) {
      const float* qa = q + (size_t)a * V;
      const int V4 = V >> 2;
#pragma unroll
      for (int k = 0; k < SV; ++k) {
        // max(0, p - q) with a correctly rounded subtraction, in place
        const int i = threadIdx.x + RT * k;
        const float4 qv = i < V4 ? ((const float4*)qa)[i] : make_float4(0.f, 0.f, 0.f, 0.f);
        w[k].x = fmaxf(__fsub_rn(w[k].x, qv.x), 0.f);
        w[k].y = fmaxf(__fsub_rn(w[k].y, qv.y), 0.f);
        w[k].z = fmaxf(__fsub_rn(w[k].z, qv.z), 0.f);
        w[k].w = fmaxf(__fsub_rn(w[k].w, qv.w), 0.f);
      }
      y = strided_sample(w, r, pre, &total, &result);
      if (y < 0) {                               // residual without integer mass: draw from p
        load_strided(pp + (size_t)a * V, V, w, 0.f);
        y = strided_sample(w, r, pre, &total, &result);
      }
    } else {
      y = strided_sample(w, r, pre, &total, &result);
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
  if (p.V > RT * 4 * SV || (p.V & 3)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(softmax_kernel, dim3(p.M), dim3(RT), 0, s, p);
  return hipGetLastError();
}
hipError_t launch_draft_sample(const DraftSampleParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  if (p.V > RT * 4 * SV || (p.V & 3)) return hipErrorInvalidValue;   // rows are read as float4
  hipLaunchKernelGGL(draft_sample_kernel, dim3(p.B), dim3(RT), 0, s, p);
  return hipGetLastError();
}
hipError_t launch_accept(const AcceptParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  if (p.V > RT * 4 * SV || (p.V & 3)) return hipErrorInvalidValue;   // rows are read as float4
  hipLaunchKernelGGL(accept_kernel, dim3(p.B), dim3(RT), 0, s, p);
  return hipGetLastError();
}
// Forced acceptance for workload generation: with probability alpha (the
// slot's draft uniform below alpha 2^32) draft token i of a task becomes the
// token its reference continuation holds at that position (P + i + 1, P the
// committed length).  Used with greedy verification, where the draft
// uniforms are otherwise unused.
__global__ void force_draft_kernel(ForceParams p) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= p.B) return;
  const int slot = p.slots[b];
  if (slot < 0 || slot >= p.n_slots) return;
  const int pos = p.state[(size_t)slot * ST_N + ST_LEN] + p.i + 1;
  const uint32_t u = p.u[(size_t)b * (2 * p.gamma + 1) + p.i];
  if ((uint64_t)u < p.threshold && pos >= 0 && pos < p.cont_len)
    p.draft_tok[(size_t)b * p.gamma + p.i] = p.cont[(size_t)b * p.cont_len + pos];
}

hipError_t launch_force_draft(const ForceParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  hipLaunchKernelGGL(force_draft_kernel, dim3((p.B + 255) / 256), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_commit(const CommitParams& p, hipStream_t s) {
  if (p.B <= 0) return hipSuccess;
  hipLaunchKernelGGL(commit_kernel, dim3((p.B + 255) / 256), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace sd
