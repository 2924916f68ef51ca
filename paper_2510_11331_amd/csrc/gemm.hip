// Skinny GEMM for the projections of the draft and verify passes:
// out[M, N] = A[M, K] * W[N, K]^T with M = rows of the pass (a few to a few
// dozen in decoding, up to 64 per block in prefill), fp32 accumulation.
//
// The pass is bound by streaming W from HBM, so the kernel is organised
// around that stream:
//   * each wave owns NT 16-row tiles of W (16*NT output columns) and streams
//     them straight from global memory into registers, 256 contiguous bytes
//     of a row per step and lane group (no LDS round trip: every weight byte
//     is used by exactly one wave), one step ahead of the MFMAs;
//   * the activations A[M, K-range] are shared by the 4 waves of a workgroup
//     and staged through LDS in 256-byte column chunks, double buffered;
//   * the K permutation inside a chunk is the same for A and W, so each lane
//     reads 64 contiguous bytes of its weight row per step;
//   * bf16: one v_mfma_f32_16x16x32_bf16 per 16-byte unit; fp32: four
//     v_mfma_f32_16x16x4_f32;
//   * K is split over gridDim.y when the column tiles alone cannot fill the
//     256 CUs; partial tiles go to a workspace and the last-arriving
//     workgroup of a column tile adds them in split order (deterministic)
//     and runs the epilogue.
// Epilogues: store fp32, add into the fp32 residual stream, or SwiGLU over
// interleaved gate/up rows (written in the model dtype).
#include "sd_internal.h"

namespace sd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Mfma;
template <> struct Mfma<bf16_t> {
  __device__ __forceinline__ static f32x4 step(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
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

template <typename T, int MT, int NT, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(GemmParams p) {
  constexpr int ROWB = GEMM_CHUNK + 16;          // LDS row stride (bytes), padded
  constexpr int UNITS = GEMM_CHUNK / 64;         // 16-byte units per lane group per step
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][MT * 16 * ROWB];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, g = lane >> 4;
  const size_t kbytes = (size_t)p.K * sizeof(T);
  const int m0 = blockIdx.z * MT * 16;
  const int split = blockIdx.y;
  const int n_wave = (blockIdx.x * GEMM_WAVES + wave) * 16 * NT;
  const bool active = n_wave < p.N;
  const int total_chunks = (int)(kbytes / GEMM_CHUNK);
  const int c0 = split * p.chunks_per_split;
  const int c1 = min(c0 + p.chunks_per_split, total_chunks);

  const unsigned char* A = (const unsigned char*)p.A;
  const unsigned char* wrow[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j)
    wrow[j] = (const unsigned char*)p.W + (size_t)(active ? n_wave + 16 * j + r16 : 0) * kbytes + g * 64;

  const int arow = tid >> 4, acol = (tid & 15) * 16;

  f32x4 acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 w0[NT][UNITS], w1[NT][UNITS], ab[MT];

  auto load_w = [&](u32x4 (&w)[NT][UNITS], int c) {
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int u = 0; u < UNITS; ++u)
        w[j][u] = *(const u32x4*)(wrow[j] + (size_t)c * GEMM_CHUNK + u * 16);
  };
  auto load_a = [&](int c) {
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int m = m0 + arow + 16 * i;
      ab[i] = m < p.M ? *(const u32x4*)(A + (size_t)m * kbytes + (size_t)c * GEMM_CHUNK + acol)
                      : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store_a = [&](unsigned char* L) {
#pragma unroll
    for (int i = 0; i < MT; ++i) *(u32x4*)(L + (arow + 16 * i) * ROWB + acol) = ab[i];
  };
  auto compute = [&](const unsigned char* L, u32x4 (&w)[NT][UNITS]) {
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const u32x4 af = *(const u32x4*)(L + (i * 16 + r16) * ROWB + g * 64 + u * 16);
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = Mfma<T>::step(af, w[j][u], acc[i][j]);
      }
    }
  };

  if (c0 < c1) {
    if (active) load_w(w0, c0);
    load_a(c0);
    store_a(lds[0]);
    __syncthreads();
    for (int c = c0; c < c1; c += 2) {
      const bool has1 = c + 1 < c1;
      if (has1) {
        if (active) load_w(w1, c + 1);
        load_a(c + 1);
      }
      if (active) compute(lds[0], w0);
      if (has1) store_a(lds[1]);
      __syncthreads();
      if (!has1) break;
      const bool has2 = c + 2 < c1;
      if (has2) {
        if (active) load_w(w0, c + 2);
        load_a(c + 2);
      }
      if (active) compute(lds[1], w1);
      if (has2) store_a(lds[0]);
      __syncthreads();
    }
  }

  // accumulator element (i, j, v) is row m0 + 16 i + 4 g + v, column n_wave + 16 j + r16
  if (p.splits > 1) {
    if (active) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int m = m0 + 16 * i + 4 * g + v;
            if (m < p.M)
              p.partial[((size_t)split * p.M + m) * p.N + n_wave + 16 * j + r16] = acc[i][j][v];
          }
    }
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = atomicAdd(&p.counters[blockIdx.x], 1) == p.splits - 1;
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    if (active) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const int m = m0 + 16 * i + 4 * g + v;
            float s = 0.f;
            if (m < p.M)
              for (int sp = 0; sp < p.splits; ++sp)
                s += p.partial[((size_t)sp * p.M + m) * p.N + n_wave + 16 * j + r16];
            acc[i][j][v] = s;
          }
    }
    if (tid == 0) p.counters[blockIdx.x] = 0;
  }
  if (!active) return;

#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int m = m0 + 16 * i + 4 * g + v;
      if (m >= p.M) continue;
      if constexpr (EPI == EPI_SWIGLU) {
        const int F = p.N / 2;
        const int f = n_wave / 2 + r16;
        const float gate = acc[i][0][v], up = acc[i][1][v];
        Store<T>::store((T*)p.out_t, (size_t)m * F + f, silu(gate) * up);
      } else {
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          float* o = p.out + (size_t)m * p.ldo + n_wave + 16 * j + r16;
          if constexpr (EPI == EPI_RESID) *o += acc[i][j][v];
          else *o = acc[i][j][v];
        }
      }
    }
}

template <typename T, int EPI>
static hipError_t launch_mt(int mt, dim3 grid, const GemmParams& p, hipStream_t s) {
  constexpr int NT = EPI == EPI_SWIGLU ? 2 : 1;
  switch (mt) {
    case 1: hipLaunchKernelGGL((gemm_kernel<T, 1, NT, EPI>), grid, dim3(256), 0, s, p); break;
    case 2: hipLaunchKernelGGL((gemm_kernel<T, 2, NT, EPI>), grid, dim3(256), 0, s, p); break;
    case 3: hipLaunchKernelGGL((gemm_kernel<T, 3, NT, EPI>), grid, dim3(256), 0, s, p); break;
    case 4: hipLaunchKernelGGL((gemm_kernel<T, 4, NT, EPI>), grid, dim3(256), 0, s, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(int dtype, int epi, int mt, int grid_x, int grid_z, const GemmParams& p,
                       hipStream_t s) {
  dim3 grid(grid_x, p.splits, grid_z);
  if (dtype == 0) {
    if (epi == EPI_STORE) return launch_mt<bf16_t, EPI_STORE>(mt, grid, p, s);
    if (epi == EPI_RESID) return launch_mt<bf16_t, EPI_RESID>(mt, grid, p, s);
    return launch_mt<bf16_t, EPI_SWIGLU>(mt, grid, p, s);
  }
  if (epi == EPI_STORE) return launch_mt<float, EPI_STORE>(mt, grid, p, s);
  if (epi == EPI_RESID) return launch_mt<float, EPI_RESID>(mt, grid, p, s);
  return launch_mt<float, EPI_SWIGLU>(mt, grid, p, s);
}

}  // namespace sd
