// Dense projections of the verify and draft forwards: Y[M][N] = X[M][K] . W[N][K]^T.
//
// At batch 1 the tree has M <= 128 rows, so these products stream the weights from HBM
// once and are bandwidth-bound (arithmetic intensity ~ M flop/byte).  The bf16 path packs
// W once into 16x32 MFMA tiles (1 KB contiguous per tile, one 16-byte load per lane) so a
// wave reads whole kilobytes per instruction; X chunks are staged in LDS and shared by the
// four waves of a workgroup.  The K range is split across workgroups so every launch has
// hundreds of workgroups in flight; each split writes fp32 partials [split][M][N] that the
// consuming kernel (residual add + norm, RoPE + cache append, SwiGLU, logits) sums in a
// fixed order, which keeps results deterministic.
#include <hip/hip_ext.h>

#include "../launch.h"

namespace adt {

// ----------------------------------------------------------------------------- packing
// bf16 tile layout: tile (nt, kt) holds rows nt*16..+15, columns kt*32..+31 as 64 lanes x 8
// values; lane l = g*16 + i carries W[nt*16 + i][kt*32 + g*8 + e], e = 0..7.
struct PackSrc {
  const void* p[4];
  int rows[4];
  int n;
  int mode;   // 0 = stacked, 1 = gate/up interleaved in 16-row blocks
};

__device__ __forceinline__ const void* pack_row(const PackSrc& s, int n, int& r) {
  if (s.mode == 1) {
    const int blk = n / 16;
    r = (blk / 2) * 16 + n % 16;
    return s.p[blk % 2];
  }
  int i = 0;
  while (i < s.n - 1 && n >= s.rows[i]) {
    n -= s.rows[i];
    ++i;
  }
  r = n;
  return s.p[i];
}

__global__ void pack_bf16_kernel(PackSrc s, int N, int K, uint16_t* __restrict__ dst) {
  const int64_t chunks = (int64_t)N * K / 8;
  const int KT = K / 32;
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < chunks; c += (int64_t)gridDim.x * blockDim.x) {
    const int lane = (int)(c % 64);
    const int64_t tile = c / 64;
    const int kt = (int)(tile % KT);
    const int nt = (int)(tile / KT);
    const int n = nt * 16 + lane % 16;
    const int k = kt * 32 + (lane / 16) * 8;
    int r;
    const uint16_t* src = (const uint16_t*)pack_row(s, n, r);
    *reinterpret_cast<u16x8*>(dst + c * 8) = *reinterpret_cast<const u16x8*>(src + (int64_t)r * K + k);
  }
}

__global__ void pack_f32_kernel(PackSrc s, int N, int K, float* __restrict__ dst) {
  const int64_t total = (int64_t)N * K;
  for (int64_t c = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; c < total; c += (int64_t)gridDim.x * blockDim.x) {
    const int n = (int)(c / K), k = (int)(c % K);
    int r;
    const float* src = (const float*)pack_row(s, n, r);
    dst[c] = src[(int64_t)r * K + k];
  }
}

// ----------------------------------------------------------------------------- bf16 MFMA
constexpr int GEMM_THREADS = 256;

// lane (lq, g) holds Y[m = mt*16 + lq][n = nt*16 + 4g + r], r = 0..3: one 16-byte store per row.
template <int MT>
__device__ __forceinline__ void store_partials(const f32x4 (&acc)[MT], float* __restrict__ part, int s, int M, int N,
                                               int nt, int lq, int g) {
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int row = m * 16 + lq;
    if (row < M) *reinterpret_cast<f32x4*>(part + ((int64_t)s * M + row) * N + nt * 16 + 4 * g) = acc[m];
  }
}

// MT = 16-row tiles of M; KC = k-tiles (of 32) staged per LDS round (LDS stays < 64 KB).
// X chunks are staged in LDS and shared by the workgroup's four waves (one n-tile each).
template <int MT, int KC = (MT > 6 ? 4 : 8)>
__global__ __launch_bounds__(GEMM_THREADS) void gemm_bf16_kernel(const uint16_t* __restrict__ X, int ldx,
                                                                 const uint16_t* __restrict__ Wp, int M, int N,
                                                                 int K, int splits, float* __restrict__ part) {
  constexpr int MP = 16 * MT;
  constexpr int XW = KC * 32 + 8;   // padded LDS row (bf16)
  __shared__ __attribute__((aligned(16))) uint16_t Xs[MP][XW];

  const int NT = N / 16, KT = K / 32;
  const int tid = threadIdx.x, wave = tid / WAVE, lane = tid % WAVE;
  const int lq = lane & 15, g = lane >> 4;
  const int nt = blockIdx.x * 4 + wave;
  const int s = blockIdx.y;
  const int kt0 = (int)((int64_t)KT * s / splits), kt1 = (int)((int64_t)KT * (s + 1) / splits);
  const bool active = nt < NT;

  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};

  const bf16x8* wp = reinterpret_cast<const bf16x8*>(Wp) + ((int64_t)(active ? nt : 0) * KT) * 64 + lane;

  for (int c = kt0; c < kt1; c += KC) {
    const int nk = min(KC, kt1 - c);
    bf16x8 wf[KC];
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (active && j < nk) wf[j] = wp[(int64_t)(c + j) * 64];
    __syncthreads();
    const int pieces = MP * nk * 4;
    for (int p = tid; p < pieces; p += GEMM_THREADS) {
      const int r = p / (nk * 4), cc = (p % (nk * 4)) * 8;
      u16x8 v = u16x8{0, 0, 0, 0, 0, 0, 0, 0};
      if (r < M) v = *reinterpret_cast<const u16x8*>(X + (int64_t)r * ldx + c * 32 + cc);
      *reinterpret_cast<u16x8*>(&Xs[r][cc]) = v;
    }
    __syncthreads();
    if (active) {
#pragma unroll
      for (int j = 0; j < KC; ++j) {
        if (j < nk) {
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const bf16x8 bx = *reinterpret_cast<const bf16x8*>(&Xs[m * 16 + lq][j * 32 + g * 8]);
            acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j], bx, acc[m], 0, 0, 0);
          }
        }
      }
    }
  }
  if (active) store_partials<MT>(acc, part, s, M, N, nt, lq, g);
}

// Few tree rows (M <= 32): each wave reads its X fragments straight from global memory (the
// rows are a few KB and L2-resident), so weights and inputs of a whole chunk are in flight
// together and no workgroup barrier is needed.
template <int MT, int KC = 8>
__global__ __launch_bounds__(GEMM_THREADS) void gemm_bf16_direct_kernel(const uint16_t* __restrict__ X, int ldx,
                                                                        const uint16_t* __restrict__ Wp, int M,
                                                                        int N, int K, int splits,
                                                                        float* __restrict__ part) {
  const int NT = N / 16, KT = K / 32;
  const int lane = threadIdx.x % WAVE, lq = lane & 15, g = lane >> 4;
  const int nt = blockIdx.x * 4 + threadIdx.x / WAVE;
  const int s = blockIdx.y;
  if (nt >= NT) return;
  const int kt0 = (int)((int64_t)KT * s / splits), kt1 = (int)((int64_t)KT * (s + 1) / splits);
  f32x4 acc[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bf16x8* wp = reinterpret_cast<const bf16x8*>(Wp) + ((int64_t)nt * KT) * 64 + lane;
  for (int c = kt0; c < kt1; c += KC) {
    const int nk = min(KC, kt1 - c);
    bf16x8 wf[KC], xf[KC][MT];
#pragma unroll
    for (int j = 0; j < KC; ++j) {
      wf[j] = bf16x8{};
#pragma unroll
      for (int m = 0; m < MT; ++m) xf[j][m] = bf16x8{};
      if (j < nk) {
        wf[j] = wp[(int64_t)(c + j) * 64];
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          const int row = m * 16 + lq;
          if (row < M) xf[j][m] = *reinterpret_cast<const bf16x8*>(X + (int64_t)row * ldx + (c + j) * 32 + g * 8);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (j < nk)
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j], xf[j][m], acc[m], 0, 0, 0);
  }
  store_partials<MT>(acc, part, s, M, N, nt, lq, g);
}

// ----------------------------------------------------------------------------- fp32 (vector)
// One wave per output column; lanes stride K, rows in groups of 16, wave-reduced.
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ X, int ldx,
                                                       const float* __restrict__ W, int M, int N, int K,
                                                       float* __restrict__ part) {
  const int wave = threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  const int n = blockIdx.x * 4 + wave;
  if (n >= N) return;
  const float* w = W + (int64_t)n * K;
  for (int m0 = 0; m0 < M; m0 += 16) {
    float acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.f;
    for (int k = lane; k < K; k += WAVE) {
      const float wv = w[k];
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (m0 + i < M) acc[i] = fmaf(X[(int64_t)(m0 + i) * ldx + k], wv, acc[i]);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float v = wave_sum(acc[i]);
      if (lane == 0 && m0 + i < M) part[(int64_t)(m0 + i) * N + n] = v;
    }
  }
}

// ----------------------------------------------------------------------------- host
size_t packed_bytes(int total_rows, int K, int dtype) {
  return (size_t)total_rows * K * (dtype == ADT_BF16 ? 2 : 4);
}

adt_status launch_pack(const void* const* srcs, const int32_t* rows, int n_src, int K, int mode, int dtype, void* dst,
                       hipStream_t st) {
  ADT_CHECK_ARG(srcs && rows && dst && n_src >= 1 && n_src <= 4, ADT_E_ARG, "pack: bad arguments");
  ADT_CHECK_ARG(mode == 0 || (mode == 1 && n_src == 2 && rows[0] == rows[1]), ADT_E_ARG, "pack: bad mode");
  PackSrc s{};
  int N = 0;
  for (int i = 0; i < n_src; ++i) {
    ADT_CHECK_ARG(srcs[i] != nullptr && rows[i] > 0, ADT_E_ARG, "pack: source %d empty", i);
    s.p[i] = srcs[i];
    s.rows[i] = rows[i];
    N += rows[i];
    if (dtype == ADT_BF16) ADT_CHECK_ARG(rows[i] % 16 == 0, ADT_E_SHAPE, "pack: rows %d not a multiple of 16", rows[i]);
  }
  s.n = n_src;
  s.mode = mode;
  if (dtype == ADT_BF16) {
    ADT_CHECK_ARG(K % 32 == 0, ADT_E_SHAPE, "pack: K %d not a multiple of 32", K);
    pack_bf16_kernel<<<1024, 256, 0, st>>>(s, N, K, (uint16_t*)dst);
  } else {
    pack_f32_kernel<<<1024, 256, 0, st>>>(s, N, K, (float*)dst);
  }
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

// Split-K factor: enough workgroups to keep HBM busy (about two per CU) but at least
// eight k-tiles (8 KB of weights per wave) per split, since the consumers sum the splits.
int gemm_splits(int M, int N, int K, int dtype) {
  if (dtype == ADT_F32) return 1;
  const int NB = (N / 16 + 3) / 4;
  const int KT = K / 32;
  int s = (512 + NB - 1) / NB;
  if (s > KT / 8) s = KT / 8;
  if (s < 1) s = 1;
  (void)M;
  return s;
}

// With ev0/ev1 set, the dispatch itself records the events at the kernel's start and end
// (kernel duration, not host-side markers).
adt_status launch_gemm(const void* X, int ldx, const void* Wp, int M, int N, int K, int splits, int dtype, float* part,
                       hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  ADT_CHECK_ARG(M >= 1 && M <= 128, ADT_E_CAPACITY, "gemm: M=%d outside [1,128]", M);
  if (dtype == ADT_F32) {
    hipExtLaunchKernelGGL(gemm_f32_kernel, dim3((N + 3) / 4), dim3(256), 0, st, ev0, ev1, 0, (const float*)X, ldx,
                          (const float*)Wp, M, N, K, part);
    ADT_LAUNCH_CHECK();
    return ADT_OK;
  }
  ADT_CHECK_ARG(N % 16 == 0 && K % 32 == 0 && ldx % 8 == 0, ADT_E_SHAPE, "gemm: N=%d K=%d ldx=%d misaligned", N, K, ldx);
  const dim3 grid((N / 16 + 3) / 4, splits), block(GEMM_THREADS);
  const int mt = (M + 15) / 16;
  const uint16_t* x = (const uint16_t*)X;
  const uint16_t* w = (const uint16_t*)Wp;
#define ADT_GEMM(KERNEL) hipExtLaunchKernelGGL(KERNEL, grid, block, 0, st, ev0, ev1, 0, x, ldx, w, M, N, K, splits, part)
  switch (mt) {
    case 1: ADT_GEMM(gemm_bf16_direct_kernel<1>); break;
    case 2: ADT_GEMM(gemm_bf16_direct_kernel<2>); break;
    case 3: ADT_GEMM(gemm_bf16_kernel<3>); break;
    case 4: ADT_GEMM(gemm_bf16_kernel<4>); break;
    case 5:
    case 6: ADT_GEMM(gemm_bf16_kernel<6>); break;
    default: ADT_GEMM(gemm_bf16_kernel<8>); break;
  }
#undef ADT_GEMM
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

}  // namespace adt
