// Dense projections of the verify and draft forwards: Y[M][N] = X[M][K] . W[N][K]^T.
//
// At batch 1 the tree has M <= 128 rows, so these products stream the weights from HBM
// once and are bandwidth-bound (arithmetic intensity ~ M flop/byte).  The bf16 path packs
// W once into 16x32 MFMA tiles (1 KB contiguous per tile, one 16-byte load per lane) so a
// wave reads whole kilobytes per instruction.  A workgroup owns T adjacent 16-column tiles
// and one of S contiguous K ranges; its eight waves split that range, keep the next k-tiles'
// weight and input fragments in flight while multiplying the current ones, and sum their
// partial tiles in LDS in wave order (deterministic; no workgroup waits on another).  T and
// S are chosen so that about one workgroup lands on each CU with as many columns as its
// registers allow: every workgroup reads the M input rows of its K range, so more columns
// per workgroup mean fewer re-reads of the input per weight byte.  The input rows are the
// bf16 activations the previous step stored (the residual projections' finish writes the
// next RMSNorm output).  With S = 1 the finished tile runs a fused epilogue (RoPE with the
// K/V cache append, SwiGLU, or a plain store); residual projections store their K-range
// sums, and resid_norm adds them in range order.
#include <hip/hip_ext.h>

#include <algorithm>

#include "../launch.h"

namespace adt {

ADT_DEVICE_ERROR_WORD(gemm)

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

__device__ __forceinline__ f32x4 shfl_xor4(f32x4 v, int mask) {
  return f32x4{__shfl_xor(v[0], mask, WAVE), __shfl_xor(v[1], mask, WAVE), __shfl_xor(v[2], mask, WAVE),
               __shfl_xor(v[3], mask, WAVE)};
}

// Inputs of a block's epilogue that do not depend on the product, requested by the wave that
// will finish the block before the main loop starts: the residual tile (EPI_RESID), or the
// RoPE factors of the lane's four columns and the cache slot of its row (EPI_QKV).
struct EpiPre {
  float v[8];
  int slot;
};
__device__ __forceinline__ EpiPre epi_preload(const GemmEpi& e, int row, int g, int nt, int M, int N) {
  EpiPre p;
#pragma unroll
  for (int i = 0; i < 8; ++i) p.v[i] = 0.f;
  p.slot = 0;
  if (row >= M) return p;
  if (e.mode == EPI_RESID) {
    if (!e.assign) {
      const f32x4 h = *reinterpret_cast<const f32x4*>(e.resid + (int64_t)row * N + nt * 16 + 4 * g);
#pragma unroll
      for (int i = 0; i < 4; ++i) p.v[i] = h[i];
    }
  } else if (e.mode == EPI_QKV && g < 2) {
    const int d = N / 3, half = e.Dh / 2, n0 = nt * 16, within = n0 % d, u = (within % e.Dh) / 16;
    const int node = e.nb == 1 ? row : row >> 1;
    p.slot = *e.slot0 + node;
    if (n0 / d < 2) {
      const float2* cs = e.rope + (int64_t)e.pos[node] * half + 8 * u + 4 * g;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float2 t = cs[r];
        p.v[2 * r] = t.x;
        p.v[2 * r + 1] = t.y;
      }
    }
  }
  return p;
}

// Epilogue of one finished 16-row block of tile nt, run by a whole wave: lane (lq, g) holds
// Y[row][nt*16 + 4g + r], r = 0..3.  In a QKV or gate/up tile, columns 0..7 (lanes g < 2)
// pair with columns 8..15 (lanes g + 2).
__device__ __forceinline__ void tile_epilogue(const GemmEpi& e, f32x4 y, const EpiPre& pre, int row, int g, int nt,
                                              int M, int N) {
  const bool live = row < M;
  const int c = nt * 16 + 4 * g;
  if (e.mode == EPI_STORE) {
    if (live) *reinterpret_cast<f32x4*>(e.out + row * e.ldo + c) = y;
  } else if (e.mode == EPI_QKV) {
    const f32x4 y2 = shfl_xor4(y, 32);
    if (live && g < 2) {
      const int d = N / 3, Dh = e.Dh, half = Dh / 2;
      const int n0 = nt * 16, region = n0 / d, within = n0 % d, head = within / Dh, u = (within % Dh) / 16;
      const int j = 8 * u + 4 * g;   // element of the head's first half held in y[0]
      float a[4] = {y[0], y[1], y[2], y[3]}, b[4] = {y2[0], y2[1], y2[2], y2[3]};
      const int node = e.nb == 1 ? row : row >> 1, branch = row - node * e.nb;
      (void)node;
      if (region < 2) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float cx = pre.v[2 * r], sx = pre.v[2 * r + 1];
          const float x1 = a[r], x2 = b[r];
          a[r] = x1 * cx - x2 * sx;
          b[r] = x2 * cx + x1 * sx;
        }
      }
      if (region > 0 && e.slot_cap > 0 && pre.slot >= e.slot_cap) {   // a row past the cache
        dev_fail(DEVINV_KV_RANGE);
        return;
      }
      uint16_t* dst = region == 0 ? e.q + (int64_t)row * d + head * Dh
                                  : (region == 1 ? e.kc : e.vc) + branch * e.cache_sb + head * e.stride_h +
                                        (int64_t)pre.slot * Dh;
      *reinterpret_cast<u16x4*>(dst + j) = u16x4{f2bf(a[0]), f2bf(a[1]), f2bf(a[2]), f2bf(a[3])};
      *reinterpret_cast<u16x4*>(dst + j + half) = u16x4{f2bf(b[0]), f2bf(b[1]), f2bf(b[2]), f2bf(b[3])};
    }
  } else if (e.mode == EPI_RESID) {
    if (live) {
      float* hp = e.resid + (int64_t)row * N + c;
      f32x4 h = y;
      if (!e.assign) h = f32x4{pre.v[0] + y[0], pre.v[1] + y[1], pre.v[2] + y[2], pre.v[3] + y[3]};
      *reinterpret_cast<f32x4*>(hp) = h;
      store4(e.act + act_index(row, c, N, e.act_pk), h[0], h[1], h[2], h[3]);
    }
  } else if (e.mode == EPI_SWIGLU) {
    const f32x4 u = shfl_xor4(y, 32);
    if (live && g < 2) {
      const int f = nt * 8 + 4 * g;
      *reinterpret_cast<u16x4*>(e.act + act_index(row, f, N / 2, e.act_pk)) =
          u16x4{f2bf(y[0] / (1.f + expf(-y[0])) * u[0]), f2bf(y[1] / (1.f + expf(-y[1])) * u[1]),
                f2bf(y[2] / (1.f + expf(-y[2])) * u[2]), f2bf(y[3] / (1.f + expf(-y[3])) * u[3])};
    }
  }
}

// Sum of squares of eight bf16 values added to s (products exact in fp32).
__device__ __forceinline__ float sumsq8(bf16x8 v, float s) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const bf16x2 p{v[2 * i], v[2 * i + 1]};
    s = __builtin_amdgcn_fdot2_f32_bf16(p, p, s, false);
  }
  return s;
}

// MT = 16-row blocks of M, T = 16-column tiles per workgroup, KC = k-tiles per load round.
// Workgroup b takes column block b / S and K range b % S; wave w takes the w-th eighth of the
// range.  Rounds are double-buffered: round r + 1's fragments are requested before round r's
// MFMAs, so one round stays in flight per wave.  With stagger the wave starts its rounds at an
// offset that depends on the workgroup (wrapping around its chunk), so the waves of different
// CUs do not read the same input lines at the same time; the sum order stays fixed per tile.
// Loads past the wave's range are clamped to its last k-tile and their products discarded.
// NORM: the waves also sum the squares of the input fragments they multiply (lane (lq, g)
// holds row m * 16 + lq), the sums meet in LDS in wave order, and each finished row is scaled
// by its RMSNorm factor before the epilogue.  PRE: the epilogue's own inputs are requested
// before the main loop (EPI_QKV, EPI_RESID).
template <int MT, int T, int KC, bool NORM, bool PRE>
__global__ __launch_bounds__(TILE_THREADS) void gemm_rows_kernel(const uint16_t* __restrict__ X, int ldx,
                                                                 const uint16_t* __restrict__ Wp, int M, int N, int K,
                                                                 int S, int stagger, GemmEpi epi) {
  constexpr int TT = MT * T;                            // 16x16 output blocks per workgroup
  constexpr int TR = TT < TILE_WAVES ? TT : TILE_WAVES; // blocks finished per LDS round
  constexpr int NR = (TT + TR - 1) / TR;                // rounds
  __shared__ f32x4 red[TILE_WAVES][TR][WAVE];
  const int KT = K / 32;
  const int cb = blockIdx.x / S, sp = blockIdx.x % S;
  // column group cb of G takes tiles [t0, t0 + tc), tc <= T; a shorter group repeats its last
  // tile in the remaining slots (the loop stays free of branches; those products are dropped)
  const int G = gridDim.x / S, tiles = N / 16;
  const int t0 = (int)((int64_t)cb * tiles / G), tc = (int)((int64_t)(cb + 1) * tiles / G) - t0;
  // the wave index is made scalar, so the K range and the round bounds are uniform branches
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / WAVE);
  const int lane = threadIdx.x % WAVE, lq = lane & 15, g = lane >> 4;
  const int ks0 = (int)((int64_t)KT * sp / S), ks1 = (int)((int64_t)KT * (sp + 1) / S);
  const int kt0 = ks0 + (int)((int64_t)(ks1 - ks0) * wave / TILE_WAVES);
  const int kt1 = ks0 + (int)((int64_t)(ks1 - ks0) * (wave + 1) / TILE_WAVES);
  const int nk = kt1 - kt0, span = (nk + KC - 1) / KC * KC;
  const int rot = (stagger && nk > 0) ? (int)((blockIdx.x * 37u) % (unsigned)(span / KC)) * KC : 0;
  const bf16x8* wp[T];
#pragma unroll
  for (int t = 0; t < T; ++t) wp[t] = reinterpret_cast<const bf16x8*>(Wp) + (int64_t)(t0 + min(t, tc - 1)) * KT * 64 + lane;
  // input fragment m of k-tile kk at xp[m] + kk * xks: row-major rows (clamped to M - 1), or
  // the fragment layout's 1 KB blocks (row blocks past the last clamped to it)
  const int mt = (M + 15) / 16;
  const uint16_t* xp[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m)
    xp[m] = ldx == X_FRAG ? X + ((int64_t)min(m, mt - 1) * WAVE + lane) * 8
                          : X + (int64_t)min(m * 16 + lq, M - 1) * ldx + g * 8;
  const int64_t xks = ldx == X_FRAG ? (int64_t)mt * WAVE * 8 : 32;
  // round start of the i-th round (c = kt0 + i * KC) after the rotation
  auto kmap = [&](int c) {
    int r = c - kt0 + rot;
    if (r >= span) r -= span;
    return kt0 + r;
  };
  bf16x8 wa[KC][T], xa[KC][MT], wb[KC][T], xb[KC][MT];
  auto load = [&](bf16x8(&w)[KC][T], bf16x8(&x)[KC][MT], int c) {
    const int c0 = kmap(c);
#pragma unroll
    for (int j = 0; j < KC; ++j) {
      const int kk = min(c0 + j, kt1 - 1);
#pragma unroll
      for (int t = 0; t < T; ++t) w[j][t] = __builtin_nontemporal_load(wp[t] + (int64_t)kk * 64);
#pragma unroll
      for (int m = 0; m < MT; ++m) x[j][m] = *reinterpret_cast<const bf16x8*>(xp[m] + kk * xks);
    }
  };
  // wave w finishes block r * TR + w of round r: its epilogue inputs are requested now
  EpiPre pre[PRE ? NR : 1];
#pragma unroll
  for (int r = 0; r < (PRE ? NR : 1); ++r) {
    const int q = r * TR + wave;
    if (PRE && wave < TR && q < TT && q / MT < tc) pre[r] = epi_preload(epi, (q % MT) * 16 + lq, g, t0 + q / MT, M, N);
  }
  f32x4 acc[T][MT];
  float ss[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) ss[m] = 0.f;
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[t][m] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](bf16x8(&w)[KC][T], bf16x8(&x)[KC][MT], int c) {
    const int c0 = kmap(c);
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (c0 + j < kt1) {
#pragma unroll
        for (int m = 0; m < MT; ++m) {
#pragma unroll
          for (int t = 0; t < T; ++t) acc[t][m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[j][t], x[j][m], acc[t][m], 0, 0, 0);
          if (NORM) ss[m] = sumsq8(x[j][m], ss[m]);
        }
      }
  };
  if (nk > 0) {
    load(wa, xa, kt0);
    for (int c = kt0;;) {
      if (c + KC < kt1) load(wb, xb, c + KC);
      mma(wa, xa, c);
      c += KC;
      if (c >= kt1) break;
      if (c + KC < kt1) load(wa, xa, c + KC);
      mma(wb, xb, c);
      c += KC;
      if (c >= kt1) break;
    }
  }
  // NORM: the row sums of squares of each wave (its four lane groups first), read back per
  // row by the finishing waves after the first barrier below
  __shared__ float red_ss[NORM ? TILE_WAVES : 1][NORM ? MT : 1][16];
  if (NORM) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float v = ss[m];
      v += __shfl_xor(v, 16, WAVE);
      v += __shfl_xor(v, 32, WAVE);
      if (g == 0) red_ss[wave][m][lq] = v;
    }
  }
  // Sum the waves' partial blocks in wave order; wave i then finishes block q0 + i.
#pragma unroll
  for (int rr = 0; rr < NR; ++rr) {
    const int q0 = rr * TR;
#pragma unroll
    for (int i = 0; i < TR; ++i)
      if (q0 + i < TT) red[wave][i][lane] = acc[(q0 + i) / MT % T][(q0 + i) % MT];
    __syncthreads();
    if (wave < TR && q0 + wave < TT && (q0 + wave) / MT < tc) {
      f32x4 y = red[0][wave][lane];
#pragma unroll
      for (int w = 1; w < TILE_WAVES; ++w) {
        const f32x4 v = red[w][wave][lane];
        y = f32x4{y[0] + v[0], y[1] + v[1], y[2] + v[2], y[3] + v[3]};
      }
      const int q = q0 + wave;
      const int row = (q % MT) * 16 + lq, nt = t0 + q / MT;
      if (NORM) {
        float t = 0.f;
#pragma unroll
        for (int w = 0; w < TILE_WAVES; ++w) t += red_ss[w][q % MT][lq];
        const float r = rsqrtf(t / K + epi.norm_eps);
        y = f32x4{y[0] * r, y[1] * r, y[2] * r, y[3] * r};
      }
      if (epi.mode == EPI_PART) {
        if (row < M) *reinterpret_cast<f32x4*>(epi.part + ((int64_t)sp * M + row) * N + nt * 16 + 4 * g) = y;
      } else {
        EpiPre p{};
        if (PRE) p = pre[PRE ? rr : 0];
        else if (epi.mode == EPI_QKV || epi.mode == EPI_RESID) p = epi_preload(epi, row, g, nt, M, N);
        tile_epilogue(epi, y, p, row, g, nt, M, N);
      }
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

// Tiles per workgroup T and K ranges S for M rows of an N x K product, measured with inputs in
// the fragment layout on the 7B layer shapes (K 4096 / 8192 / 11008, N 4096 - 65536) at 8,
// 24, 40 and 61 rows (a round of KC k-tiles per wave: 1 for T >= 3, else 2, or 3 at <= 16
// rows; see launch_gemm).  One K range: T as wide as the registers allow while the launch
// keeps >= 256 workgroups; wider than 2 at <= 32 rows only where that is exactly one
// workgroup per CU or the launch still has >= 1024 (61 rows: QKV T = 3 21 us; gate/up T = 4
// 48 against 50 at T = 2; LM head T = 4 113 against 139; 24 rows: gate/up T = 2 39 against
// 44, LM head T = 4 102 against 109).  partial (the caller adds K-range sums): one tile and
// the whole K per workgroup where that already gives >= 192 workgroups (O 9.1 us and the
// draft FC 15.5 at 61 rows), except a long K at > 32 rows, which takes T = 4 with about ten
// k-tiles per wave per range (down at 61 rows: T = 4 S = 4 20.5 us against 28 at S = 1).
RowsPlan gemm_rows_plan(int M, int N, int K, bool partial, bool wide) {
  const int mt = (M + 15) / 16, tiles = N / 16, KT = K / 32;
  const int tmax = mt <= 4 ? 4 : 2;
  auto ok = [&](int t) { return t <= tmax && tiles % t == 0; };
  if (partial && tiles >= 192 && (mt <= 2 || K <= 8192)) return {1, 1, tiles};
  if (!partial || (mt == 1 && tiles >= 192)) {
    // wide (an epilogue without early inputs, whose registers the accumulators can take), up
    // to 64 rows: one round of the CUs with five or six tiles each where that covers the
    // columns (gate/up: 256 groups of 5-6; 61 rows 37.5 us against 45 with 512 groups of
    // 2-3, 24 rows 34.0 against 37.4 with 688 groups of 2, 8 rows 32.4 against 34.3), and
    // at 49-64 rows 512 groups of 8 for the widest products (LM head 107 us against 118 with
    // 1024 groups of 4)
    if (wide && mt <= 4 && (tiles + 255) / 256 >= 5 && (tiles + 255) / 256 <= 6) return {6, 1, 256};
    if (wide && mt == 4 && tiles >= 2048 && (tiles + 511) / 512 == 8) return {8, 1, 512};
    // a short K (five k-tiles a wave) over 257-510 tiles at <= 32 rows: two tiles per
    // workgroup in one round rather than 1.x rounds of one (LlamaGen-XL gate/up, 448 tiles at
    // 11 rows: 6.6 us against 7.3)
    if (wide && mt <= 2 && KT <= 5 * TILE_WAVES && tiles > 256 && tiles < 512 && tiles % 2 == 0) return {2, 1, tiles / 2};
    // > 32 rows: a multiple of 256 workgroups (whole rounds of the CUs) with at most tmax tiles
    // each, spread evenly
    if (mt >= 3)
      for (int g = 256; g <= tiles; g += 256)
        if ((tiles + g - 1) / g <= tmax) return {(tiles + g - 1) / g, 1, g};
    for (int t : {4, 3, 2}) {
      if (!ok(t) || tiles / t < 256) continue;
      if (t <= 2 || tiles / t == 256 || (mt == 2 && tiles / t >= 1024)) return {t, 1, tiles / t};
    }
    return {1, 1, tiles};
  }
  const int smax = std::max(1, std::min(GEMM_MAX_SPLITS, KT / (10 * TILE_WAVES)));
  int T = 1;
  for (int t : {4, 3, 2})
    if (ok(t) && (tiles / t) * smax >= 192) {
      T = t;
      break;
    }
  const int blocks = tiles / T;
  const int S = blocks >= 192 ? 1 : std::max(1, std::min(smax, 256 / blocks));
  return {T, S, blocks};
}

adt_status launch_gemm(const void* X, int ldx, const void* Wp, int M, int N, int K, int dtype, float* part,
                       const GemmEpi& epi, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1, int* splits) {
  ADT_CHECK_ARG(M >= 1 && M <= 128, ADT_E_CAPACITY, "gemm: M=%d outside [1,128]", M);
  if (dtype == ADT_F32) {
    hipExtLaunchKernelGGL(gemm_f32_kernel, dim3((N + 3) / 4), dim3(256), 0, st, ev0, ev1, 0, (const float*)X, ldx,
                          (const float*)Wp, M, N, K, part);
    ADT_LAUNCH_CHECK();
    if (splits) *splits = 1;
    return ADT_OK;
  }
  ADT_CHECK_ARG(N % 16 == 0 && K % 32 == 0 && ldx % 8 == 0 && (ldx == X_FRAG || ldx >= K), ADT_E_SHAPE,
                "gemm: N=%d K=%d ldx=%d misaligned", N, K, ldx);
  switch (epi.mode) {
    case EPI_STORE: ADT_CHECK_ARG(epi.out && epi.ldo % 4 == 0, ADT_E_ARG, "gemm: store target"); break;
    case EPI_PART: ADT_CHECK_ARG(epi.part != nullptr, ADT_E_ARG, "gemm: partial-sum buffer"); break;
    case EPI_QKV:
      ADT_CHECK_ARG(epi.nb == 1 || epi.nb == 2, ADT_E_ARG, "gemm: QKV epilogue branches %d", epi.nb);
      ADT_CHECK_ARG(epi.Dh >= 16 && epi.Dh % 16 == 0 && N % (3 * epi.Dh) == 0 && epi.q && epi.kc && epi.vc &&
                        epi.slot0 && epi.pos && epi.rope,
                    ADT_E_ARG, "gemm: QKV epilogue (Dh=%d, N=%d)", epi.Dh, N);
      break;
    case EPI_SWIGLU:
      ADT_CHECK_ARG(epi.act != nullptr && (epi.act_pk == 0 || (N / 2 % 32 == 0 && epi.act_pk * 16 >= M)), ADT_E_ARG,
                    "gemm: SwiGLU output (layout %d)", epi.act_pk);
      break;
    case EPI_RESID:
      ADT_CHECK_ARG(epi.resid && epi.act && (epi.act_pk == 0 || (N % 32 == 0 && epi.act_pk * 16 >= M)), ADT_E_ARG,
                    "gemm: residual epilogue (layout %d)", epi.act_pk);
      break;
    default: ADT_CHECK_ARG(false, ADT_E_ARG, "gemm: epilogue %d", epi.mode);
  }
  ADT_CHECK_ARG(epi.norm_eps == 0.f || (epi.norm_eps > 0.f && epi.mode != EPI_PART && epi.mode != EPI_RESID),
                ADT_E_ARG, "gemm: the input norm needs one K range");
  // the residual epilogue takes the residual projections' plan, which must keep one K range
  const RowsPlan p = gemm_rows_plan(M, N, K, epi.mode == EPI_PART || epi.mode == EPI_RESID,
                                    epi.mode == EPI_STORE || epi.mode == EPI_SWIGLU);
  ADT_CHECK_ARG(epi.mode != EPI_RESID || p.S == 1, ADT_E_ARG, "gemm: residual epilogue with %d K ranges", p.S);
  ADT_CHECK_ARG(epi.mode != EPI_PART || (size_t)p.S * M * N <= epi.part_elems, ADT_E_CAPACITY,
                "gemm: %d K-range sums of %d x %d exceed the partial buffer", p.S, M, N);
  const int mt = (M + 15) / 16, KT = K / 32;
  const int stagger = 1;
  const dim3 grid(p.G * p.S), block(TILE_THREADS);
  const uint16_t* x = (const uint16_t*)X;
  const uint16_t* w = (const uint16_t*)Wp;
  // epilogue inputs requested early for QKV and the residual epilogue (not at > 4 row blocks,
  // where the registers are taken by the accumulators)
  const bool pre = (epi.mode == EPI_QKV || epi.mode == EPI_RESID) && mt <= 4;
#define ADT_GR_L(MTV, TV, KCV, NV, PV)                                                                            \
  hipExtLaunchKernelGGL(gemm_rows_kernel<MTV, TV, KCV, NV, (PV && MTV <= 4)>, grid, block, 0, st, ev0, ev1, 0, x, \
                        ldx, w, M, N, K, p.S, stagger, epi)
#define ADT_GR(MTV, TV, KCV)                  \
  if (epi.norm_eps > 0.f) {                   \
    if (pre && MTV <= 4) {                    \
      ADT_GR_L(MTV, TV, KCV, true, true);     \
    } else {                                  \
      ADT_GR_L(MTV, TV, KCV, true, false);    \
    }                                         \
  } else if (pre && MTV <= 4) {               \
    ADT_GR_L(MTV, TV, KCV, false, true);      \
  } else {                                    \
    ADT_GR_L(MTV, TV, KCV, false, false);     \
  }
  // k-tiles per round: one with three or four tiles (their fragments already keep enough in
  // flight), else two, or three for one row block
#define ADT_GR_T4(MTV, KCV)              \
  switch (p.T) {                         \
    case 4: ADT_GR(MTV, 4, 1); break;    \
    case 3: ADT_GR(MTV, 3, 1); break;    \
    case 2: ADT_GR(MTV, 2, KCV); break;  \
    default: ADT_GR(MTV, 1, KCV); break; \
  }
#define ADT_GR_T6(MTV, KCV)  \
  if (p.T == 6) {            \
    ADT_GR(MTV, 6, 1);       \
  } else {                   \
    ADT_GR_T4(MTV, KCV)      \
  }
#define ADT_GR_T8(MTV, KCV)  \
  if (p.T == 8) {            \
    ADT_GR(MTV, 8, 1);       \
  } else {                   \
    ADT_GR_T6(MTV, KCV)      \
  }
#define ADT_GR_T2(MTV, KCV)              \
  if (p.T >= 2) {                        \
    ADT_GR(MTV, 2, KCV);                 \
  } else {                               \
    ADT_GR(MTV, 1, KCV);                 \
  }
  // k-tiles per round: at one row block 3, or the wave's whole K range when that is at most
  // five k-tiles (one round trip: LlamaGen-XL O at 11 rows 4.5 against 4.85 us)
  const bool one_round = (KT + p.S * TILE_WAVES - 1) / (p.S * TILE_WAVES) <= 5;
  switch (mt) {
    case 1:
      if (one_round) {
        ADT_GR_T6(1, 5)
      } else {
        ADT_GR_T6(1, 3)
      }
      break;
    case 2: ADT_GR_T6(2, 2) break;
    case 3: ADT_GR_T6(3, 2) break;
    case 4: ADT_GR_T8(4, 2) break;
    case 5:
    case 6: ADT_GR_T2(6, 2) break;
    default: ADT_GR_T2(8, 2) break;
  }
#undef ADT_GR_T2
#undef ADT_GR_T8
#undef ADT_GR_T6
#undef ADT_GR_T4
#undef ADT_GR
#undef ADT_GR_L
  ADT_LAUNCH_CHECK();
  if (splits) *splits = p.S;
  return ADT_OK;
}

}  // namespace adt
