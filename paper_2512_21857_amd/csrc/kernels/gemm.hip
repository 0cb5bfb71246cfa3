// Dense projections of the verify and draft forwards: Y[M][N] = X[M][K] . W[N][K]^T.
//
// At batch 1 the tree has M <= 128 rows, so these products stream the weights from HBM
// once and are bandwidth-bound (arithmetic intensity ~ M flop/byte).  The bf16 path packs
// W once into 16x32 MFMA tiles (1 KB contiguous per tile, one 16-byte load per lane) so a
// wave reads whole kilobytes per instruction.  One workgroup owns one 16-column output
// tile and the whole K range: its eight waves take contiguous K chunks, issue all their
// weight loads at once, and the partial tiles are summed in LDS in wave order (so results
// are deterministic and no workgroup waits on another).  The finished tile goes through a
// fused epilogue: residual add with the row sums of squares the next RMSNorm needs, RoPE
// with the K/V cache append, SwiGLU, or a plain store.  A GEMM whose input is a normalised
// row applies the norm while loading it (fp32 residual times the row's scale, rounded to
// bf16), so no norm, RoPE, SwiGLU or reduction kernel runs between projections.
#include <hip/hip_ext.h>

#include "../launch.h"

namespace adt {

// ----------------------------------------------------------------------------- packing
// bf16 tile layout: tile (nt, kt) holds packed rows nt*16..+15, columns kt*32..+31 as 64
// lanes x 8 values; lane l = g*16 + i carries W[row(nt*16 + i)][kt*32 + g*8 + e], e = 0..7.
// Packed row order (row(n)):
//   ADT_PACK_STACK    sources stacked in order;
//   ADT_PACK_GATE_UP  two equal sources interleaved in blocks of 8 rows (gate block t, up
//                     block t, ...), so every 16-row tile holds 8 gate and the matching 8 up rows;
//   ADT_PACK_QKV      sources stacked, and inside every head of `group` rows each 16-row tile
//                     holds rows 8u..8u+7 of the head's first half and the same rows of its
//                     second half (a RoPE pair shares a tile).
struct PackSrc {
  const void* p[4];
  int rows[4];
  int n;
  int mode;
  int group;
};

__device__ __forceinline__ const void* pack_row(const PackSrc& s, int n, int& r) {
  if (s.mode == ADT_PACK_GATE_UP) {
    const int blk = n / 8;
    r = (blk / 2) * 8 + n % 8;
    return s.p[blk % 2];
  }
  int i = 0;
  while (i < s.n - 1 && n >= s.rows[i]) {
    n -= s.rows[i];
    ++i;
  }
  if (s.mode == ADT_PACK_QKV) {
    const int half = s.group / 2, e = n % s.group, u = e / 16, t = e % 16;
    n = n - e + (t < 8 ? 8 * u + t : half + 8 * u + t - 8);
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
constexpr int TILE_WAVES = 8;
constexpr int TILE_THREADS = TILE_WAVES * WAVE;

// Eight consecutive fp32 residual values times the row's norm scale, rounded to bf16.
__device__ __forceinline__ bf16x8 norm_load8(const float* __restrict__ p, float r) {
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  const u16x8 u{f2bf(a.x * r), f2bf(a.y * r), f2bf(a.z * r), f2bf(a.w * r),
                f2bf(b.x * r), f2bf(b.y * r), f2bf(b.z * r), f2bf(b.w * r)};
  return __builtin_bit_cast(bf16x8, u);
}

__device__ __forceinline__ f32x4 shfl_xor4(f32x4 v, int mask) {
  return f32x4{__shfl_xor(v[0], mask, WAVE), __shfl_xor(v[1], mask, WAVE), __shfl_xor(v[2], mask, WAVE),
               __shfl_xor(v[3], mask, WAVE)};
}

// Epilogue of one finished 16-row block of tile nt, run by a whole wave: lane (lq, g) holds
// Y[row][nt*16 + 4g + r], r = 0..3.  In a QKV or gate/up tile, columns 0..7 (lanes g < 2)
// pair with columns 8..15 (lanes g + 2).
__device__ __forceinline__ void tile_epilogue(const GemmEpi& e, f32x4 y, int row, int g, int nt, int M, int N) {
  const bool live = row < M;
  const int c = nt * 16 + 4 * g;
  if (e.mode == EPI_STORE) {
    if (live) *reinterpret_cast<f32x4*>(e.out + row * e.ldo + c) = y;
  } else if (e.mode == EPI_RESID) {
    float* hp = e.h + (int64_t)row * N + c;
    if (live) {
      if (!e.assign) {
        const f32x4 o = *reinterpret_cast<const f32x4*>(hp);
        y = f32x4{o[0] + y[0], o[1] + y[1], o[2] + y[2], o[3] + y[3]};
      }
      *reinterpret_cast<f32x4*>(hp) = y;
    }
    float ss = live ? y[0] * y[0] + y[1] * y[1] + y[2] * y[2] + y[3] * y[3] : 0.f;
    ss += __shfl_xor(ss, 16, WAVE);
    ss += __shfl_xor(ss, 32, WAVE);
    if (live && g == 0) e.ssp_out[(int64_t)row * (N / 16) + nt] = ss;
  } else if (e.mode == EPI_QKV) {
    const f32x4 y2 = shfl_xor4(y, 32);
    if (live && g < 2) {
      const int d = N / 3, Dh = e.Dh, half = Dh / 2;
      const int n0 = nt * 16, region = n0 / d, within = n0 % d, head = within / Dh, u = (within % Dh) / 16;
      const int j = 8 * u + 4 * g;   // element of the head's first half held in y[0]
      float a[4] = {y[0], y[1], y[2], y[3]}, b[4] = {y2[0], y2[1], y2[2], y2[3]};
      const int node = e.nb == 1 ? row : row >> 1, branch = row - node * e.nb;
      if (region < 2) {
        const float2* cs = e.rope + (int64_t)e.pos[node] * half + j;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float2 t = cs[r];
          const float x1 = a[r], x2 = b[r];
          a[r] = x1 * t.x - x2 * t.y;
          b[r] = x2 * t.x + x1 * t.y;
        }
      }
      uint16_t* dst = region == 0 ? e.q + (int64_t)row * d + head * Dh
                                  : (region == 1 ? e.kc : e.vc) + branch * e.cache_sb + head * e.stride_h +
                                        (*e.slot0 + (int64_t)node) * Dh;
      *reinterpret_cast<u16x4*>(dst + j) = u16x4{f2bf(a[0]), f2bf(a[1]), f2bf(a[2]), f2bf(a[3])};
      *reinterpret_cast<u16x4*>(dst + j + half) = u16x4{f2bf(b[0]), f2bf(b[1]), f2bf(b[2]), f2bf(b[3])};
    }
  } else if (e.mode == EPI_SWIGLU) {
    const f32x4 u = shfl_xor4(y, 32);
    if (live && g < 2) {
      const int f = nt * 8 + 4 * g;
      *reinterpret_cast<u16x4*>(e.act + (int64_t)row * (N / 2) + f) =
          u16x4{f2bf(y[0] / (1.f + expf(-y[0])) * u[0]), f2bf(y[1] / (1.f + expf(-y[1])) * u[1]),
                f2bf(y[2] / (1.f + expf(-y[2])) * u[2]), f2bf(y[3] / (1.f + expf(-y[3])) * u[3])};
    }
  }
}

// k-tiles per wave per load round: as many as fit about 160 VGPRs of loaded operands (a
// workgroup of 8 waves holds 2 waves per SIMD, so 256 VGPRs per lane are available).
template <int MT, int NTW, bool NORM>
constexpr int tile_kc() {
  constexpr int per = MT * (NORM ? 8 : 4) + NTW * 4;
  constexpr int kc = (MT >= 6 ? 120 : 160) / per;   // the widest row blocks keep room for accumulators
  return kc < 1 ? 1 : (kc > 16 ? 16 : kc);
}

// MT = 16-row blocks of M, NTW = 16-column tiles per workgroup.  Every load of a round is
// issued before any is used (indices clamped instead of branched on, so the loads form one
// batch); rounds past the wave's K range and rows past M only feed discarded results.
template <int MT, int NTW, bool NORM>
__global__ __launch_bounds__(TILE_THREADS) void gemm_tile_kernel(const void* __restrict__ Xv, int ldx,
                                                                 const uint16_t* __restrict__ Wp, int M, int N,
                                                                 int K, GemmEpi epi) {
  constexpr int KC = tile_kc<MT, NTW, NORM>();
  constexpr int TT = MT * NTW;               // 16x16 output blocks per workgroup
  constexpr int TR = TT < 4 ? TT : 4;        // blocks summed per LDS round
  __shared__ f32x4 red[TILE_WAVES][TR][WAVE];
  __shared__ float rscale[NORM ? MT * 16 : 1];
  const int KT = K / 32;
  // the wave index is made scalar, so the K range and the round bounds below are uniform
  // branches that do not split the batch of loads
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / WAVE);
  const int lane = threadIdx.x % WAVE, lq = lane & 15, g = lane >> 4;
  const int kt0 = (int)((int64_t)KT * wave / TILE_WAVES), kt1 = (int)((int64_t)KT * (wave + 1) / TILE_WAVES);
  const bf16x8* wp[NTW];
#pragma unroll
  for (int t = 0; t < NTW; ++t)
    wp[t] = reinterpret_cast<const bf16x8*>(Wp) + (int64_t)(blockIdx.x * NTW + t) * KT * 64 + lane;

  bf16x8 wf[KC][NTW];
  auto load_w = [&](int c) {
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (c + j < kt1)
#pragma unroll
        for (int t = 0; t < NTW; ++t) wf[j][t] = wp[t][(int64_t)(c + j) * 64];
  };
  const float* xf32[MT];
  const uint16_t* xb16[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) {
    const int row = min(m * 16 + lq, M - 1);
    xf32[m] = (const float*)Xv + (int64_t)row * ldx + g * 8;
    xb16[m] = (const uint16_t*)Xv + (int64_t)row * ldx + g * 8;
  }
  float4 xa[KC][MT][NORM ? 2 : 1];
  bf16x8 xb[KC][MT];
  auto load_x = [&](int c) {
#pragma unroll
    for (int j = 0; j < KC; ++j) {
      if (c + j >= kt1) continue;
      const int kk = c + j;
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        if constexpr (NORM) {
          xa[j][m][0] = *reinterpret_cast<const float4*>(xf32[m] + kk * 32);
          xa[j][m][NORM ? 1 : 0] = *reinterpret_cast<const float4*>(xf32[m] + kk * 32 + 4);
        } else {
          xb[j][m] = *reinterpret_cast<const bf16x8*>(xb16[m] + kk * 32);
        }
      }
    }
  };
  // the first round's weights and inputs are in flight while the norm scales are formed
  load_w(kt0);
  load_x(kt0);

  float rr[MT];
  if constexpr (NORM) {
    // Row scales from the per-16-column sums of squares: LPR consecutive lanes per row
    // each sum a strided subset in order, then a fixed butterfly across the LPR lanes.
    constexpr int ROWS = MT * 16;
    constexpr int LPR = TILE_THREADS / ROWS >= 32 ? 32 : (TILE_THREADS / ROWS >= 16 ? 16 : (TILE_THREADS / ROWS >= 8 ? 8 : 4));
    const int row = threadIdx.x / LPR, part = threadIdx.x % LPR;
    float t = 0.f;
    if (row < ROWS) {
      const float* sp = epi.ssp_in + (int64_t)min(row, M - 1) * epi.nss_in;
      const int nss = epi.nss_in;
      for (int i0 = part; i0 < nss; i0 += 8 * LPR) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = sp[min(i0 + j * LPR, nss - 1)];   // one batch of loads
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (i0 + j * LPR < nss) t += v[j];
      }
    }
#pragma unroll
    for (int o = LPR / 2; o >= 1; o >>= 1) t += __shfl_xor(t, o, WAVE);
    if (row < ROWS && part == 0) rscale[row] = row < M ? rsqrtf(t / K + epi.eps) : 0.f;
    __syncthreads();
#pragma unroll
    for (int m = 0; m < MT; ++m) rr[m] = rscale[m * 16 + lq];
  }

  f32x4 acc[NTW][MT];
#pragma unroll
  for (int t = 0; t < NTW; ++t)
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[t][m] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int c = kt0; c < kt1; c += KC) {
    const int nk = min(KC, kt1 - c);
#pragma unroll
    for (int j = 0; j < KC; ++j) {
      if (j < nk) {
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          bf16x8 x;
          if constexpr (NORM) {
            const float4 a = xa[j][m][0], b = xa[j][m][NORM ? 1 : 0];
            const float r = rr[m];
            x = __builtin_bit_cast(bf16x8, u16x8{f2bf(a.x * r), f2bf(a.y * r), f2bf(a.z * r), f2bf(a.w * r),
                                                 f2bf(b.x * r), f2bf(b.y * r), f2bf(b.z * r), f2bf(b.w * r)});
          } else {
            x = xb[j][m];
          }
#pragma unroll
          for (int t = 0; t < NTW; ++t) acc[t][m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[j][t], x, acc[t][m], 0, 0, 0);
        }
      }
    }
    if (c + KC < kt1) {
      load_w(c + KC);
      load_x(c + KC);
    }
  }
  // Sum the waves' partial blocks in wave order; wave i then finishes block q0 + i.
#pragma unroll
  for (int q0 = 0; q0 < TT; q0 += TR) {
#pragma unroll
    for (int i = 0; i < TR; ++i)
      if (q0 + i < TT) red[wave][i][lane] = acc[(q0 + i) / MT % NTW][(q0 + i) % MT];
    __syncthreads();
    if (wave < TR && q0 + wave < TT) {
      f32x4 y = red[0][wave][lane];
#pragma unroll
      for (int w = 1; w < TILE_WAVES; ++w) {
        const f32x4 v = red[w][wave][lane];
        y = f32x4{y[0] + v[0], y[1] + v[1], y[2] + v[2], y[3] + v[3]};
      }
      const int q = q0 + wave;
      tile_epilogue(epi, y, (q % MT) * 16 + lq, g, blockIdx.x * NTW + q / MT, M, N);
    }
    __syncthreads();
  }
}

// ----------------------------------------------------------------------------- fp32 (vector)
// Unfused fp32 path (row kernels finish the layer).  One wave per output column; lanes
// stride K, rows in groups of 16, wave-reduced.
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

adt_status launch_pack(const void* const* srcs, const int32_t* rows, int n_src, int K, int mode, int group, int dtype,
                       void* dst, hipStream_t st) {
  ADT_CHECK_ARG(srcs && rows && dst && n_src >= 1 && n_src <= 4, ADT_E_ARG, "pack: bad arguments");
  ADT_CHECK_ARG(mode == ADT_PACK_STACK || (mode == ADT_PACK_GATE_UP && n_src == 2 && rows[0] == rows[1]) ||
                    (mode == ADT_PACK_QKV && group >= 16 && group % 16 == 0),
                ADT_E_ARG, "pack: bad mode %d (group %d)", mode, group);
  PackSrc s{};
  int N = 0;
  for (int i = 0; i < n_src; ++i) {
    ADT_CHECK_ARG(srcs[i] != nullptr && rows[i] > 0, ADT_E_ARG, "pack: source %d empty", i);
    ADT_CHECK_ARG(mode != ADT_PACK_QKV || rows[i] % group == 0, ADT_E_SHAPE, "pack: %d rows not whole heads", rows[i]);
    ADT_CHECK_ARG(mode != ADT_PACK_GATE_UP || rows[i] % 8 == 0, ADT_E_SHAPE, "pack: gate/up rows %d", rows[i]);
    s.p[i] = srcs[i];
    s.rows[i] = rows[i];
    N += rows[i];
  }
  s.n = n_src;
  s.mode = mode;
  s.group = group;
  if (dtype == ADT_BF16) {
    ADT_CHECK_ARG(N % 16 == 0 && K % 32 == 0, ADT_E_SHAPE, "pack: N=%d K=%d not multiples of 16/32", N, K);
    pack_bf16_kernel<<<1024, 256, 0, st>>>(s, N, K, (uint16_t*)dst);
  } else {
    pack_f32_kernel<<<1024, 256, 0, st>>>(s, N, K, (float*)dst);
  }
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_gemm(const void* X, int ldx, const void* Wp, int M, int N, int K, int dtype, float* part,
                       const GemmEpi& epi, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  ADT_CHECK_ARG(M >= 1 && M <= 128, ADT_E_CAPACITY, "gemm: M=%d outside [1,128]", M);
  if (dtype == ADT_F32) {
    hipExtLaunchKernelGGL(gemm_f32_kernel, dim3((N + 3) / 4), dim3(256), 0, st, ev0, ev1, 0, (const float*)X, ldx,
                          (const float*)Wp, M, N, K, part);
    ADT_LAUNCH_CHECK();
    return ADT_OK;
  }
  ADT_CHECK_ARG(N % 16 == 0 && K % 32 == 0 && ldx % 8 == 0, ADT_E_SHAPE, "gemm: N=%d K=%d ldx=%d misaligned", N, K, ldx);
  const bool norm = epi.ssp_in != nullptr;
  ADT_CHECK_ARG(!norm || epi.nss_in == K / 16, ADT_E_SHAPE, "gemm: norm input needs K/16 sums per row");
  switch (epi.mode) {
    case EPI_STORE: ADT_CHECK_ARG(epi.out && epi.ldo % 4 == 0, ADT_E_ARG, "gemm: store target"); break;
    case EPI_RESID: ADT_CHECK_ARG(epi.h && epi.ssp_out, ADT_E_ARG, "gemm: residual epilogue buffers"); break;
    case EPI_QKV:
      ADT_CHECK_ARG(epi.nb == 1 || epi.nb == 2, ADT_E_ARG, "gemm: QKV epilogue branches %d", epi.nb);
      ADT_CHECK_ARG(epi.Dh >= 16 && epi.Dh % 16 == 0 && N % (3 * epi.Dh) == 0 && epi.q && epi.kc && epi.vc &&
                        epi.slot0 && epi.pos && epi.rope,
                    ADT_E_ARG, "gemm: QKV epilogue (Dh=%d, N=%d)", epi.Dh, N);
      break;
    case EPI_SWIGLU: ADT_CHECK_ARG(epi.act != nullptr, ADT_E_ARG, "gemm: SwiGLU output"); break;
    default: ADT_CHECK_ARG(false, ADT_E_ARG, "gemm: epilogue %d", epi.mode);
  }
  const int mt = (M + 15) / 16;
  // 16-column tiles per workgroup: each wave's input fragments feed all of them, so more
  // tiles cut the re-reads of the input rows, but fewer workgroups leave CUs idle.  The
  // largest of 4, 2, 1 that keeps at least 160 workgroups (measured best on the 36-layer
  // d = 1280 cycle among 96, 160, 256 and always 1; at most 2 from 81 rows on, for registers)
  const int tiles = N / 16;
  int ntw = 1;
  if (tiles % 4 == 0 && tiles / 4 >= 160 && mt <= 4) ntw = 4;
  else if (tiles % 2 == 0 && tiles / 2 >= 160) ntw = 2;
  const dim3 grid(tiles / ntw), block(TILE_THREADS);
  const uint16_t* w = (const uint16_t*)Wp;
#define ADT_GEMM(...) hipExtLaunchKernelGGL(__VA_ARGS__, grid, block, 0, st, ev0, ev1, 0, X, ldx, w, M, N, K, epi)
#define ADT_GEMM_MT(MT, NORM)                          \
  if (ntw == 4) {                                      \
    ADT_GEMM(gemm_tile_kernel<MT, 4, NORM>);           \
  } else if (ntw == 2) {                               \
    ADT_GEMM(gemm_tile_kernel<MT, 2, NORM>);           \
  } else {                                             \
    ADT_GEMM(gemm_tile_kernel<MT, 1, NORM>);           \
  }
#define ADT_GEMM_MT2(MT, NORM)                         \
  if (ntw >= 2) {                                      \
    ADT_GEMM(gemm_tile_kernel<MT, 2, NORM>);           \
  } else {                                             \
    ADT_GEMM(gemm_tile_kernel<MT, 1, NORM>);           \
  }
#define ADT_GEMM_ALL(NORM)             \
  switch (mt) {                        \
    case 1: ADT_GEMM_MT(1, NORM) break; \
    case 2: ADT_GEMM_MT(2, NORM) break; \
    case 3: ADT_GEMM_MT(3, NORM) break; \
    case 4: ADT_GEMM_MT(4, NORM) break; \
    case 5:                            \
    case 6: ADT_GEMM_MT2(6, NORM) break; \
    default: ADT_GEMM_MT2(8, NORM) break; \
  }
  if (norm) {
    ADT_GEMM_ALL(true)
  } else {
    ADT_GEMM_ALL(false)
  }
#undef ADT_GEMM_ALL
#undef ADT_GEMM_MT2
#undef ADT_GEMM_MT
#undef ADT_GEMM
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

}  // namespace adt
