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
//     often) and splits K over its KW waves (up to 16), interleaved in
//     groups of U k-steps; each wave streams its share of the tile straight
//     into registers, one step group ahead of the MFMAs;
//   * the matching activation fragments are loaded the same way (they are
//     small and stay in L2), so the main loop has no LDS traffic and no
//     barriers; it has no branches either (padding rows and groups past a
//     wave's share are out-of-range buffer loads that return zero), so
//     vmcnt only ever waits for the older step group;
//   * bf16: one v_mfma_f32_16x16x32_bf16 per 16-byte unit; fp32: four
//     v_mfma_f32_16x16x4_f32;
//   * the KW partial tiles are added in wave order through LDS
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

// narrow tiles fit 128 VGPRs and run up to 16 waves; wider ones up to 8
template <int MT, int NT> struct GemmBounds {
  static constexpr int threads = (MT * NT <= 4 && MT < 4 && NT < 4) ? 1024 : 512;
};
int gemm_max_waves(int mt, int nt) { return (mt * nt <= 4 && mt < 4 && nt < 4) ? 16 : 8; }

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
  __shared__ float red[4][MT * NT * 4][64];

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
  const int n0 = bx * 16 * NT;
  const int m0 = bz * MT * 16;
  const uint32_t tile_bytes = (uint32_t)ksteps * 1024u;
  const __amdgpu_buffer_rsrc_t wr = buf_rsrc((const char*)p.W + (size_t)bx * NT * tile_bytes, NT * tile_bytes);
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
  // the block; their positions and KV blocks are loaded before the stream
  // and their rotary (cos, sin) after it, so the epilogue waits on nothing
  int qpos[EPI == EPI_QKV ? MT : 1], qblk[EPI == EPI_QKV ? MT : 1];
  if constexpr (EPI == EPI_QKV) {
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int m = m0 + 16 * i + 4 * g + wave;
      qpos[i] = m < p.M ? p.rope.row_pos[m] : -1;
      qblk[i] = m < p.M ? p.rope.row_blk[m] : -1;
    }
  }

  // groups past nw load zeros (no memory access) and add nothing
  load.template operator()<0>(0);
  for (int i = 0; i < nw; i += 2) {
    load.template operator()<1>(i + 1);
    compute.template operator()<0>();
    load.template operator()<0>(i + 2);
    compute.template operator()<1>();
  }

  float2 qcs[EPI == EPI_QKV ? MT : 1][NT];
  if constexpr (EPI == EPI_QKV) {
    const int half = p.rope.hd / 2;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j) {
        const int c0 = n0 + 16 * j, f = 8 * ((c0 % p.rope.hd) / 16) + (r16 & 7);
        qcs[i][j] = qpos[i] >= 0 ? p.rope.tab[(size_t)qpos[i] * half + f] : float2{1.f, 0.f};
      }
  }

  // Reduction over the KW wave partials, in a fixed order: waves 4.. fold
  // into waves 0..3 four at a time (slot w holds wave w + base), then waves
  // 0..3 publish their sums and every wave finishes the output rows (i, v)
  // with (4 i + v) % KW == wave, adding the four slots in order.
  for (int base = 4; base < KW; base += 4) {
    if (wave >= base && wave < base + 4) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) red[wave - base][(i * NT + j) * 4 + v][lane] = acc[i][j][v];
    }
    __syncthreads();
    if (wave < 4 && wave + base < KW) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) acc[i][j][v] += red[wave][(i * NT + j) * 4 + v][lane];
    }
    __syncthreads();
  }
  const int nslot = min(KW, 4);
  if (wave < nslot) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) red[wave][(i * NT + j) * 4 + v][lane] = acc[i][j][v];
  }
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

  // QKV: what column n0 + 16 j + r16 of this lane is, independent of the
  // row: kind (0 q, 1 k, 2 v), q column, and the K/V element offset of
  // (token 0, block 0) in the cache; a row adds its block and token offsets
  int qkind[EPI == EPI_QKV ? NT : 1], qcol[EPI == EPI_QKV ? NT : 1];
  size_t qkvb[EPI == EPI_QKV ? NT : 1];
  const int Nq = p.rope.H * p.rope.hd;
  if constexpr (EPI == EPI_QKV) {
    const RopeParams& rp = p.rope;
    const int hd = rp.hd, half = hd / 2, Nqk = Nq + rp.KV * hd;
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      const int c0 = n0 + 16 * j;             // first column of the tile
      qkind[j] = c0 < Nq ? 0 : c0 < Nqk ? 1 : 2;
      qcol[j] = 0;
      qkvb[j] = 0;
      if (c0 < Nqk) {
        // rotary pair order: column r16 < 8 of the tile is dim 8b + r16 of
        // head h, column r16 + 8 its partner dim hd/2 + 8b + r16
        const int h = c0 / hd, f = 8 * ((c0 % hd) / 16) + (r16 & 7);
        const int d = r16 < 8 ? f : f + half;
        if (h < rp.H) qcol[j] = h * hd + d;
        else qkvb[j] = kv_tile_off(h - rp.H, 0, 0, rp.nblk, hd) + kv_key_off<T>(0, d, hd);
      } else {
        const int cv = c0 + r16 - Nqk;
        qkvb[j] = kv_tile_off(cv / hd, 0, 1, rp.nblk, hd) + kv_val_off<T>(0, cv % hd, hd);
      }
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
        for (int w = 1; w < nslot; ++w) t += red[w][(i * NT + j) * 4 + v][lane];
        o[j] = t;
      }
      // QKV: the rotary partner of column r16 is column r16 ^ 8 of the same
      // tile (exchanged while the whole wave is still converged)
      float pr[EPI == EPI_QKV ? NT : 1];
      if constexpr (EPI == EPI_QKV) {
#pragma unroll
        for (int j = 0; j < NT; ++j) pr[j] = __shfl_xor(o[j], 8);
      }
      if (m >= p.M) continue;
      if constexpr (EPI == EPI_QKV) {
        const int pos = qpos[i];                // this lane's row m (v == wave)
        if (pos < 0) continue;                  // row without an input (no pending draft token)
        const int blk = qblk[i];                // -1: K/V not written (over capacity, flagged)
        const int off = pos & 15;
        T* kv = (T*)p.rope.kv;
        const size_t brow = (size_t)max(blk, 0) * 32 * p.rope.hd;   // block offset inside a head's run
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          if (qkind[j] == 0) {
            const float2 cs = qcs[i][j];
            const float a = r16 < 8 ? o[j] : pr[j], b = r16 < 8 ? pr[j] : o[j];
            p.rope.q[(size_t)m * Nq + qcol[j]] = r16 < 8 ? a * cs.x - b * cs.y : a * cs.y + b * cs.x;
          } else if (qkind[j] == 1) {
            if (blk < 0) continue;
            const float2 cs = qcs[i][j];
            const float a = r16 < 8 ? o[j] : pr[j], b = r16 < 8 ? pr[j] : o[j];
            Store<T>::store(kv, qkvb[j] + brow + kv_key_off<T>(off, 0, p.rope.hd),
                            r16 < 8 ? a * cs.x - b * cs.y : a * cs.y + b * cs.x);
          } else {
            if (blk < 0) continue;
            Store<T>::store(kv, qkvb[j] + brow + kv_val_off<T>(off, 0, p.rope.hd), o[j]);
          }
        }
      } else if constexpr (EPI == EPI_SWIGLU) {
        // tiles (2k, 2k+1) are the gate and up rows of the same 16 outputs
        const int F = p.N / 2;
#pragma unroll
        for (int j = 0; j < NT; j += 2)
          Store<T>::store((T*)p.out_t, Tile<T>::off(m, n0 / 2 + 8 * j + r16, F), silu(o[j]) * o[j + 1]);
      } else {
        const size_t row = EPI == EPI_PART ? (size_t)blockIdx.y * p.M + m : (size_t)m;
#pragma unroll
        for (int j = 0; j < NT; ++j) {
          float* dst = p.out + row * p.ldo + n0 + 16 * j + r16;
          if constexpr (EPI == EPI_RESID) *dst += o[j];
          else *dst = o[j];
        }
      }
    }
}

// row-major [N, K] -> MFMA-tile layout, one 16-byte unit per thread
template <typename T>
__global__ void pack_linear_kernel(const T* src, T* dst, int N, int K) {
  constexpr int EPL = Tile<T>::EPL, EPK = Tile<T>::EPK;
  const int ks = K / EPK;
  const size_t units = (size_t)N * K / EPL;
  for (size_t u = blockIdx.x * (size_t)blockDim.x + threadIdx.x; u < units; u += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(u % 64);
    const size_t ts = u / 64;
    const int s = (int)(ts % ks), t = (int)(ts / ks);
    const int r = 16 * t + (lane & 15);
    const int k = s * EPK + (lane >> 4) * EPL;
    *(uint4*)(dst + u * EPL) = *(const uint4*)(src + (size_t)r * K + k);
  }
}

hipError_t launch_pack_linear(int dtype, const void* src, void* dst, int N, int K, hipStream_t s) {
  const size_t esz = dtype == 0 ? 2 : 4;
  if (N <= 0 || K <= 0 || N % 16 || ((size_t)K * esz) % 64) return hipErrorInvalidValue;
  const size_t units = (size_t)N * K * esz / 16;
  const int blocks = (int)std::min<size_t>((units + 255) / 256, 65536);
  if (dtype == 0)
    hipLaunchKernelGGL(pack_linear_kernel<bf16_t>, dim3(blocks), dim3(256), 0, s, (const bf16_t*)src, (bf16_t*)dst, N, K);
  else
    hipLaunchKernelGGL(pack_linear_kernel<float>, dim3(blocks), dim3(256), 0, s, (const float*)src, (float*)dst, N, K);
  return hipGetLastError();
}

template <typename T, int EPI, int NT, int U>
static hipError_t launch_mt(int mt, dim3 grid, int threads, const GemmParams& p, hipStream_t s, hipEvent_t e0,
                            hipEvent_t e1) {
  switch (mt) {
    case 1: launch_k(gemm_kernel<T, 1, NT, U, EPI>, grid, dim3(threads), 0, s, e0, e1, p); break;
    case 2: launch_k(gemm_kernel<T, 2, NT, U, EPI>, grid, dim3(threads), 0, s, e0, e1, p); break;
    case 3:
      if constexpr (NT <= 4) {
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
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm(int dtype, int epi, int nt, int mt, int kw, int grid_x, int ksplit, int grid_z,
                       const GemmParams& p, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  if (kw < 1 || kw > gemm_max_waves(mt, nt)) return hipErrorInvalidValue;
  if (p.N % (16 * nt) || grid_x * 16 * nt != p.N || grid_z * 16 * mt < p.M ||
      ((size_t)p.K * (dtype == 0 ? 2 : 4)) % GEMM_CHUNK)
    return hipErrorInvalidValue;
  if (ksplit < 1 || (ksplit > 1 && epi != EPI_PART) || ksplit > (int)((size_t)p.K * (dtype == 0 ? 2 : 4) / GEMM_CHUNK))
    return hipErrorInvalidValue;
  // several M blocks over column tiles in groups of 8: the XCD-aware 1-D grid
  GemmParams q = p;
  q.mblocks = 1;
  dim3 grid(grid_x, ksplit, grid_z);
  if (grid_z > 1 && ksplit == 1 && grid_x % 8 == 0) {
    q.mblocks = grid_z;
    grid = dim3(grid_x * grid_z, 1, 1);
  }
  const int threads = 64 * kw;
  if (epi == EPI_QKV && (kw != 4 || p.rope.hd % 16 || p.N != (p.rope.H + 2 * p.rope.KV) * p.rope.hd))
    return hipErrorInvalidValue;
  if (dtype == 0) {
    if (epi == EPI_STORE) return launch_nt<bf16_t, EPI_STORE>(nt, mt, grid, threads, q, s, e0, e1);
    if (epi == EPI_RESID) return launch_nt<bf16_t, EPI_RESID>(nt, mt, grid, threads, q, s, e0, e1);
    if (epi == EPI_QKV) return launch_nt<bf16_t, EPI_QKV>(nt, mt, grid, threads, q, s, e0, e1);
    if (epi == EPI_PART) return launch_nt<bf16_t, EPI_PART>(nt, mt, grid, threads, q, s, e0, e1);
    return launch_nt<bf16_t, EPI_SWIGLU>(nt, mt, grid, threads, q, s, e0, e1);
  }
  if (epi == EPI_STORE) return launch_nt<float, EPI_STORE>(nt, mt, grid, threads, q, s, e0, e1);
  if (epi == EPI_RESID) return launch_nt<float, EPI_RESID>(nt, mt, grid, threads, q, s, e0, e1);
  if (epi == EPI_QKV) return launch_nt<float, EPI_QKV>(nt, mt, grid, threads, q, s, e0, e1);
  if (epi == EPI_PART) return launch_nt<float, EPI_PART>(nt, mt, grid, threads, q, s, e0, e1);
  return launch_nt<float, EPI_SWIGLU>(nt, mt, grid, threads, q, s, e0, e1);
}

}  // namespace sd
