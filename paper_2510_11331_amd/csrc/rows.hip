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

__device__ __forceinline__ float block_sum256(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

template <typename T>
__device__ void norm_row(const float* x, const T* gain, T* out, int d, float eps, float* red) {
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) ss += x[i] * x[i];
  ss = block_sum256(ss, red);
  const float inv = 1.0f / sqrtf(ss / (float)d + eps);
  for (int i = threadIdx.x; i < d; i += 256)
    Store<T>::store(out, i, x[i] * inv * Store<T>::load(gain, i));
}

template <typename T>
__global__ __launch_bounds__(256) void rows_embed_kernel(RowsParams p) {
  __shared__ float red[4];
  const int r = blockIdx.x;
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
      }
      for (int i = threadIdx.x; i < p.d; i += 256) {
        p.x[(size_t)r * p.d + i] = 0.f;
        Store<T>::store((T*)p.xn, (size_t)r * p.d + i, 0.f);
      }
      return;
    }
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
  if (pos >= 0 && (tok < 0 || tok >= p.V)) {
    if (threadIdx.x == 0) atomicOr(p.err, ERR_BAD_TOKEN);
    tok = 0;
  }
  float* x = p.x + (size_t)r * p.d;
  const T* e = (const T*)p.embed + (size_t)tok * p.d;
  for (int i = threadIdx.x; i < p.d; i += 256) x[i] = pos >= 0 ? Store<T>::load(e, i) : 0.f;
  __syncthreads();
  norm_row<T>(x, (const T*)p.gain, (T*)p.xn + (size_t)r * p.d, p.d, p.eps, red);
}

template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(NormParams p) {
  __shared__ float red[4];
  const int r = blockIdx.x;
  const float* x = p.x + ((size_t)r * p.src_stride + p.src_off) * p.d;
  norm_row<T>(x, (const T*)p.gain, (T*)p.xn + (size_t)r * p.d, p.d, p.eps, red);
}

hipError_t launch_rows_embed(int dtype, const RowsParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if (dtype == 0) hipLaunchKernelGGL(rows_embed_kernel<bf16_t>, dim3(p.M), dim3(256), 0, s, p);
  else hipLaunchKernelGGL(rows_embed_kernel<float>, dim3(p.M), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(int dtype, const NormParams& p, hipStream_t s) {
  if (p.M <= 0) return hipSuccess;
  if (dtype == 0) hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(p.M), dim3(256), 0, s, p);
  else hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(p.M), dim3(256), 0, s, p);
  return hipGetLastError();
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
