// Verify projections for many tree rows at once (a batch of trees, M = sum of tree sizes,
// Sec. 3.1 verification applied to several sequences): C[M][N] = X[M][K] . W[N][K]^T with
// bf16 operands stored row-major with K contiguous, fp32 results.  At M in the hundreds the
// product is MFMA-bound, so it is tiled for operand reuse: a workgroup of eight waves (two
// per SIMD, so one issues MFMAs while the other waits on LDS) owns a BN x BM block of C^T
// (256 x 256 or 128 x 128), each wave a (BN/2) x (BM/4) part of 32x32 MFMA blocks
// (v_mfma_f32_32x32x16_bf16, the gfx950 instruction with the highest sustained bf16 rate).
// K advances in 64-wide stages, double-buffered in LDS: the next stage's global loads are in
// flight while the current one is multiplied, and one barrier per stage separates writes of
// one buffer from reads of the other.
//   A operand (W rows):  lane l holds W[n0 + l%32][k0 + 8*(l/32) .. +7]
//   B operand (X rows):  lane l holds X[m0 + l%32][k0 + 8*(l/32) .. +7]
//   D (C^T block):       lane l, register v holds C[m0 + l%32][n0 + 8*(v/4) + 4*(l/32) + v%4]
// so each lane stores four consecutive columns of a C row per register group.
// W is either row-major (ldw) or in the library's packed weight layout (16 x 32 tiles of
// 1 KB, tile (n/16, k/32) at ((n/16) K/32 + k/32) * 512 elements, the 8 elements k..k+7 of
// row n at ((k%32)/8 * 16 + n%16) * 8 within it), so the forwards' packed weights serve the
// batched path too.
#include <hip/hip_ext.h>

#include <algorithm>
#include <cstdint>

#include "../launch.h"

namespace adt {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int NT_WAVES_N = 2, NT_WAVES_M = 4;              // wave grid of a workgroup
constexpr int NT_THREADS = NT_WAVES_N * NT_WAVES_M * WAVE;
constexpr int NT_BK = 64;
constexpr int NT_ROW = NT_BK + 8;   // padded LDS row, bf16 (144 B: 16-byte reads of 16 lanes hit distinct banks)

template <int BN, int BM, bool PACKED>
__global__ __launch_bounds__(NT_THREADS) void gemm_nt_kernel(const uint16_t* __restrict__ X, int64_t ldx,
                                                             const uint16_t* __restrict__ W, int64_t ldw, int M,
                                                             int K, float* __restrict__ C, int64_t ldc) {
  constexpr int WN = BN / NT_WAVES_N, WM = BM / NT_WAVES_M;  // wave quarter of the block
  constexpr int NB = WN / 32, MB = WM / 32;                 // 32x32 blocks per wave
  constexpr int STAGE = (BN + BM) * NT_ROW;                 // bf16 per LDS stage
  constexpr int RPP = NT_THREADS / 8;                       // rows moved per pass (8 threads per 128-byte row)
  constexpr int CH = (BN + BM) / RPP;                       // 16-byte chunks per thread per stage
  constexpr int WCH = BN / RPP;                             // of which W chunks
  __shared__ __attribute__((aligned(16))) uint16_t lds[2 * STAGE];

  // row blocks vary fastest, so the workgroups that share a W tile run at the same time
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int tid = threadIdx.x, wave = tid / WAVE, lane = tid % WAVE;
  const int wn = wave / NT_WAVES_M, wm = wave % NT_WAVES_M;
  const int l32 = lane % 32, hi = lane / 32;

  // chunk i of this thread: row tid/8 + RPP i of the stage (W rows first, then X rows), 16 bytes at column 8 (tid%8)
  const int crow = tid / 8, ccol = (tid % 8) * 8;
  const uint16_t* gsrc[CH];
#pragma unroll
  for (int i = 0; i < CH; ++i) {
    const int row = crow + RPP * i;
    const int n = n0 + row;
    const int64_t wofs = PACKED ? ((int64_t)(n / 16) * (K / 32) + ccol / 32) * 512 + (((ccol % 32) / 8) * 16 + n % 16) * 8
                                : (int64_t)n * ldw + ccol;
    gsrc[i] = i < WCH ? W + wofs
                      : X + (int64_t)min(m0 + row - BN, M - 1) * ldx + ccol;   // rows past M feed discarded columns
  }
  // per stage: 64 columns of X; of W 64 columns, or two packed tiles
  constexpr int WSTEP = PACKED ? 1024 : NT_BK;
  u16x8 stg[CH];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < CH; ++i) stg[i] = *reinterpret_cast<const u16x8*>(gsrc[i] + kt * (i < WCH ? WSTEP : NT_BK));
  };
  auto lstore = [&](int buf) {
    uint16_t* base = lds + buf * STAGE;
#pragma unroll
    for (int i = 0; i < CH; ++i) *reinterpret_cast<u16x8*>(base + (crow + RPP * i) * NT_ROW + ccol) = stg[i];
  };

  f32x16 acc[NB][MB];
#pragma unroll
  for (int a = 0; a < NB; ++a)
#pragma unroll
    for (int b = 0; b < MB; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;

  const int KT = K / NT_BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < KT;
    if (more) gload(kt + 1);
    const uint16_t* Ws = lds + buf * STAGE;
    const uint16_t* Xs = Ws + BN * NT_ROW;
#pragma unroll
    for (int s = 0; s < NT_BK / 16; ++s) {
      bf16x8 a[NB], b[MB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        a[nb] = *reinterpret_cast<const bf16x8*>(Ws + (wn * WN + nb * 32 + l32) * NT_ROW + s * 16 + hi * 8);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        b[mb] = *reinterpret_cast<const bf16x8*>(Xs + (wm * WM + mb * 32 + l32) * NT_ROW + s * 16 + hi * 8);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
          acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[nb], b[mb], acc[nb][mb], 0, 0, 0);
    }
    // the other buffer was last read in the previous stage, which every wave finished
    // before the previous barrier; one barrier makes this stage's writes visible
    if (more) {
      lstore(buf ^ 1);
      __syncthreads();
    }
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int m = m0 + wm * WM + mb * 32 + l32;
      if (m >= M) continue;
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int n = n0 + wn * WN + nb * 32 + 8 * grp + 4 * hi;
        *reinterpret_cast<f32x4*>(C + (int64_t)m * ldc + n) =
            f32x4{acc[nb][mb][4 * grp], acc[nb][mb][4 * grp + 1], acc[nb][mb][4 * grp + 2], acc[nb][mb][4 * grp + 3]};
      }
    }
}

// ---------------------------------------------------------------------------------------------
// Packed weights with many tiles: the operands reach LDS by direct global->LDS DMA
// (global_load_lds_dwordx4: a wave instruction moves 1 KB, lane l's 16 bytes landing at byte
// 16 l), so no registers stage them and no wave spends issue slots storing them.  A workgroup
// of eight waves owns a 256 x 256 block of C^T; K advances in 32-wide stages held in a ring of
// NSTAGE slots of 32 KB, each slot 32 tiles of 1 KB in the packed order (16 rows x 32 columns,
// lane l = 16 g + i holding row i, columns 8g..8g+7): tiles 0-15 the block's W rows, 16-31 its
// X rows.  A packed W tile is copied as stored (1 KB contiguous); an X tile is gathered from
// row-major rows (16 rows x 64 bytes).  The MFMA operand reads of a 16-lane group then cover
// 256 contiguous bytes (no bank conflicts, no padding).
// Pipeline, per stage kt: the fragments of the stage's second half are read while the first
// half's eight MFMAs run; each wave waits for its own DMA of stage kt+1 (the NSTAGE-3 newer
// stages stay in flight) and one barrier publishes it; the DMA of stage kt+NSTAGE-1 then
// refills the slot of stage kt-1, whose fragments every wave consumed before that barrier;
// the next stage's first fragments are read while the second half's MFMAs run.  The DMA and
// the waits are inline assembly because the compiler, which cannot tell LDS slots apart,
// would otherwise wait for every DMA in flight before each LDS read.
constexpr int DMA_NSTAGE = 5;

// M0 is written with s_mov only: an SCC-writing instruction here would corrupt a compare the
// compiler keeps live across the statement.
#define ADT_DMA4(g0, g1, g2, g3, d)                                                                         \
  asm volatile("s_mov_b32 m0, %4\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off\n\t"                          \
               "s_mov_b32 m0, %5\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off\n\t"                          \
               "s_mov_b32 m0, %6\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %2, off\n\t"                          \
               "s_mov_b32 m0, %7\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %3, off" ::"v"(g0),                      \
               "v"(g1), "v"(g2), "v"(g3), "s"(d), "s"((d) + 1024), "s"((d) + 2048), "s"((d) + 3072)          \
               : "memory", "m0")

// With ksplit > 1 the K stages of a block are split into ksplit contiguous ranges, one per
// workgroup: range 0 writes C, range s > 0 writes the fp32 partial P[s-1] ([M][N], row stride
// N), and gemm_nt_reduce_kernel adds them to C in range order (deterministic).
// BN x BM block of C^T per workgroup of WN x WM waves (each a (BN/WN) x (BM/WM) part of 32x32
// MFMA blocks); a stage slot holds (BN + BM) / 16 tiles, four per wave: 256 x 256 or
// 384 x 128 with 2 x 4 or 4 x 2 waves, or 128 x 128 with 2 x 2 (two workgroups per CU).
template <int BN, int BM, int WN, int WM, int NSTAGE>
__global__ __launch_bounds__(WN * WM * WAVE) void gemm_nt_dma_kernel(const uint16_t* __restrict__ X, int64_t ldx,
                                                                     const uint16_t* __restrict__ W, int M, int N,
                                                                     int K, float* __restrict__ C, int64_t ldc,
                                                                     int ksplit, float* __restrict__ P) {
  static_assert(NSTAGE == 4 || NSTAGE == 5, "the wait counts below assume four or five slots");
  constexpr int WAVES = WN * WM, TILES = (BN + BM) / 16, SLOT = TILES * 1024;
  constexpr int WTN = BN / WN, WTM = BM / WM, NB = WTN / 32, MB = WTM / 32;
  static_assert(TILES == 4 * WAVES && (BN / 16) % 4 == 0 && NB >= 1 && MB >= 1, "four DMA tiles per wave");
  constexpr int D = NSTAGE - 1;   // stages in flight ahead of the one being multiplied
  __shared__ __attribute__((aligned(1024))) uint16_t lds[NSTAGE * SLOT / 2];
  // XCD-aware order: workgroup b runs on XCD b % 8; each XCD takes a contiguous range of
  // tiles (row blocks fastest), so the row blocks that share a W block meet in one L2
  const int MT = (M + BM - 1) / BM, G = gridDim.x;
  const int b = blockIdx.x, xcd = b % 8, q = G / 8, r = G % 8;
  const int tk = xcd * q + min(xcd, r) + b / 8;
  const int ks = tk % ksplit, t = tk / ksplit;
  const int m0 = (t % MT) * BM, n0 = (t / MT) * BN;
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid / WAVE), lane = tid % WAVE;
  const int wn = wave / WM, wm = wave % WM;
  constexpr int WAVES_W = (BN / 16) / 4;   // waves that load W tiles
  const int KTall = K / 32, kt0 = (int)((int64_t)KTall * ks / ksplit), kt1 = (int)((int64_t)KTall * (ks + 1) / ksplit);

  // DMA sources: wave w fills tiles 4w..4w+3 of every stage (W tiles first, then X tiles)
  const uint16_t* src[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int T = 4 * wave + i;
    if (wave < WAVES_W) {
      src[i] = W + ((int64_t)(n0 / 16 + T) * (K / 32)) * 512 + lane * 8;
    } else {
      const int m = min(m0 + 16 * (T - BN / 16) + lane % 16, M - 1);   // rows past M feed discarded columns
      src[i] = X + (int64_t)m * ldx + 8 * (lane / 16);
    }
  }
  const int64_t step = wave < WAVES_W ? 512 : 32;
#pragma unroll
  for (int i = 0; i < 4; ++i) src[i] += kt0 * step;   // this workgroup's K range
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint16_t*)lds;
  const uint32_t wdst = lds0 + 4 * wave * 1024;
  const int KT = kt1 - kt0;
  auto issue = [&](int kt) {   // past the last stage: the last stage again, into a slot never read
    const int64_t ks = min(kt, KT - 1) * step;
    const uint32_t d = wdst + (kt % NSTAGE) * SLOT;
    ADT_DMA4(src[0] + ks, src[1] + ks, src[2] + ks, src[3] + ks, d);
  };
  // fragment offsets (bytes) inside a slot: A = W rows wn*WTN + 32 nb + lane%32, B = X rows
  // wm*WTM + 32 mb + lane%32, columns 16 s + 8 (lane/32) of the stage
  const int sub = ((lane / 32) * 16 + lane % 16) * 16;
  const int aoff = (wn * (WTN / 16) + (lane % 32) / 16) * 1024 + sub;
  const int boff = (BN / 16 + wm * (WTM / 16) + (lane % 32) / 16) * 1024 + sub;
  const char* lbase = (const char*)lds;
  auto frags = [&](int kt, int s, bf16x8* a, bf16x8* bb) {
    const char* p = lbase + (kt % NSTAGE) * SLOT + s * 512;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) a[nb] = *reinterpret_cast<const bf16x8*>(p + aoff + nb * 2048);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) bb[mb] = *reinterpret_cast<const bf16x8*>(p + boff + mb * 2048);
  };
  f32x16 acc[NB][MB];
#pragma unroll
  for (int a = 0; a < NB; ++a)
#pragma unroll
    for (int c = 0; c < MB; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][c][v] = 0.f;
  auto mma = [&](const bf16x8* a, const bf16x8* bb) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[nb], bb[mb], acc[nb][mb], 0, 0, 0);
  };

#pragma unroll
  for (int s = 0; s < D; ++s) issue(s);
  if constexpr (D == 3) asm volatile("s_waitcnt vmcnt(8)\n\ts_barrier" ::: "memory");
  else asm volatile("s_waitcnt vmcnt(12)\n\ts_barrier" ::: "memory");
  bf16x8 a0[NB], b0[MB], a1[NB], b1[MB];
  frags(0, 0, a0, b0);
  __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): the loop starts with no LDS read pending
  for (int kt = 0; kt < KT; ++kt) {
    frags(kt, 1, a1, b1);
    mma(a0, b0);
    __builtin_amdgcn_sched_group_barrier(0x100, NB + MB, 0);   // the reads first, then the MFMAs
    __builtin_amdgcn_sched_group_barrier(0x008, NB * MB, 0);
    if constexpr (D == 3) asm volatile("s_waitcnt vmcnt(4)\n\ts_barrier" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(8)\n\ts_barrier" ::: "memory");
    issue(kt + D);
    frags(kt + 1, 0, a0, b0);   // past the last stage: a stale slot, never used
    mma(a1, b1);
    __builtin_amdgcn_sched_group_barrier(0x100, NB + MB, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, NB * MB, 0);
  }
  // no DMA may still be writing this workgroup's LDS when it exits
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  float* out = ks == 0 ? C : P + (int64_t)(ks - 1) * M * N;
  const int64_t ldo = ks == 0 ? ldc : N;
  const int l32 = lane % 32, hi = lane / 32;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int m = m0 + wm * WTM + mb * 32 + l32;
      if (m >= M) continue;
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int n = n0 + wn * WTN + nb * 32 + 8 * grp + 4 * hi;
        *reinterpret_cast<f32x4*>(out + (int64_t)m * ldo + n) =
            f32x4{acc[nb][mb][4 * grp], acc[nb][mb][4 * grp + 1], acc[nb][mb][4 * grp + 2], acc[nb][mb][4 * grp + 3]};
      }
    }
}
#undef ADT_DMA4

// C += P[0] + P[1] + ... in that order, four columns per thread.
__global__ void gemm_nt_reduce_kernel(float* __restrict__ C, int64_t ldc, const float* __restrict__ P, int M, int N,
                                      int nparts) {
  const int64_t quads = (int64_t)M * (N / 4);
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < quads; i += (int64_t)gridDim.x * blockDim.x) {
    const int m = (int)(i / (N / 4)), n = (int)(i % (N / 4)) * 4;
    f32x4 c = *reinterpret_cast<const f32x4*>(C + (int64_t)m * ldc + n);
    for (int s = 0; s < nparts; ++s) {
      const f32x4 p = *reinterpret_cast<const f32x4*>(P + (int64_t)s * M * N + (int64_t)m * N + n);
      c = f32x4{c[0] + p[0], c[1] + p[1], c[2] + p[2], c[3] + p[3]};
    }
    *reinterpret_cast<f32x4*>(C + (int64_t)m * ldc + n) = c;
  }
}

// Plan of the packed path on the DMA pipeline.  A 256 x 256 (or 384 x 128) workgroup takes
// a whole CU by LDS, so the blocks run in rounds of DMA_SLOTS.
//  * few 256 x 256 blocks (under 128) with K >= 8192: K split over ksplit = 4 (else 2)
//    workgroups per block, as far as the partials fit (the partials' traffic stays small
//    beside the product; shorter K runs faster in 128 x 128 blocks, measured at
//    976 x 4096 x 4096);
//  * one partial round of 256 x 256 blocks that 384 x 128 blocks fill further (N a multiple
//    of 384): those, at three quarters of the work per block;
//  * more than one round whose last is at most half full: the columns of the full rounds in
//    one launch, the rest in a second launch with K split over as many workgroups per block
//    as one round holds (at most 4), then the fixed-order reduce of their partials.
constexpr int DMA_SLOTS = 256;
struct NtPlan {
  int bn = 256;      // 256 (256 x 256 blocks) or 384 (384 x 128)
  int ksplit = 1;    // K ranges per block of the (first) launch
  int n_tail = 0;    // columns run by the second launch
  int tail_ks = 1;   // K ranges per block of the second launch
  size_t part = 0;   // fp32 partials used
};
static NtPlan gemm_nt_plan(int M, int N, int K, size_t part_elems) {
  NtPlan p;
  const int mt = (M + 255) / 256, nb = N / 256, kt = K / 32;
  const int64_t tiles = (int64_t)mt * nb;
  if (tiles < 128 && K >= 8192) {
    for (int ks = 4; ks >= 2; ks /= 2)
      if ((size_t)(ks - 1) * M * N <= part_elems && kt >= 4 * ks) {
        p.ksplit = ks;
        p.part = (size_t)(ks - 1) * M * N;
        return p;
      }
    return p;
  }
  if (N % 384 == 0 && tiles >= 128 && tiles < DMA_SLOTS) {
    const int64_t t384 = (int64_t)((M + 127) / 128) * (N / 384);
    if (t384 > tiles && t384 <= DMA_SLOTS) p.bn = 384;
    return p;
  }
  if (tiles > DMA_SLOTS && tiles % DMA_SLOTS != 0 && tiles % DMA_SLOTS <= DMA_SLOTS / 2) {
    const int nb_main = (int)(tiles / DMA_SLOTS * DMA_SLOTS / mt);
    const int tail_tiles = mt * (nb - nb_main);
    const int ks = std::min(4, DMA_SLOTS / tail_tiles);
    const size_t need = (size_t)(ks - 1) * M * (nb - nb_main) * 256;
    if (ks >= 2 && kt >= 4 * ks && need <= part_elems) {
      p.n_tail = (nb - nb_main) * 256;
      p.tail_ks = ks;
      p.part = need;
    }
  }
  return p;
}

// 128 x 128 blocks: with at most half as many blocks as CUs and K >= 2048 the K range is
// split in two, so that twice the CUs work (measured slower at a full round of blocks).
static int gemm_nt_ks128(int M, int N, int K, size_t part_elems) {
  const int64_t blocks = (int64_t)((M + 127) / 128) * (N / 128);
  return (blocks <= DMA_SLOTS / 2 && K >= 2048 && (size_t)M * N <= part_elems) ? 2 : 1;
}

size_t gemm_nt_part_elems(int M, int N, int K) {
  const NtPlan p = gemm_nt_plan(M, N, K, SIZE_MAX);
  const bool dma256 = N % 256 == 0 && (p.bn == 384 || p.ksplit > 1 || (int64_t)(N / 256) * ((M + 255) / 256) >= 128);
  if (dma256) return p.part;
  return gemm_nt_ks128(M, N, K, SIZE_MAX) > 1 ? (size_t)M * N : 0;
}

// One launch of 256 x 256 DMA blocks over columns [0, N) of the operands given (W already
// offset to the first column's packed tile), K split ks ways with the partials reduced.
static void launch_dma256(const uint16_t* x, int64_t ldx, const uint16_t* w, int M, int N, int K, float* C,
                          int64_t ldc, int ks, float* part, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  hipExtLaunchKernelGGL((gemm_nt_dma_kernel<256, 256, 2, 4, DMA_NSTAGE>), dim3((M + 255) / 256 * (N / 256) * ks),
                        dim3(8 * WAVE), 0, st, ev0, ks > 1 ? nullptr : ev1, 0, x, ldx, w, M, N, K, C, ldc, ks, part);
  if (ks > 1) {
    const int64_t quads = (int64_t)M * (N / 4);
    const int blocks = (int)std::min<int64_t>((quads + 255) / 256, 4096);
    hipExtLaunchKernelGGL(gemm_nt_reduce_kernel, dim3(blocks), dim3(256), 0, st, nullptr, ev1, 0, C, ldc,
                          (const float*)part, M, N, ks - 1);
  }
}

adt_status launch_gemm_nt(const void* X, int64_t ldx, const void* W, int64_t ldw, int M, int N, int K, float* C,
                          int64_t ldc, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1, bool packed, float* part,
                          size_t part_elems) {
  ADT_CHECK_ARG(X && W && C, ADT_E_ARG, "gemm_nt: null pointer");
  ADT_CHECK_ARG(M >= 1 && N >= 128 && K >= 64 && N % 128 == 0 && K % 64 == 0, ADT_E_SHAPE,
                "gemm_nt: M=%d N=%d K=%d (N a multiple of 128, K of 64)", M, N, K);
  ADT_CHECK_ARG(ldx >= K && (packed || ldw >= K) && ldc >= N && ldx % 8 == 0 && ldw % 8 == 0 && ldc % 4 == 0,
                ADT_E_SHAPE, "gemm_nt: leading dimensions");
  // Tile choice (measured on the M = 976 projections of the 7B layer shapes): 256 x 256
  // when it still gives every CU a workgroup, else 128 x 128 (two workgroups per CU by LDS);
  // 256 x 128 was never the fastest.
  const int best = (N % 256 == 0 && (int64_t)(N / 256) * ((M + 255) / 256) >= 256) ? 0 : 2;
  const uint16_t* x = (const uint16_t*)X;
  const uint16_t* w = (const uint16_t*)W;
  // Packed weights in 256 x 256 (or 384 x 128) blocks when that gives at least 128
  // workgroups (half the CUs; measured faster than the 128 x 128 blocks down to there), or
  // with K split across workgroups: the DMA pipeline, as planned above.
  if (packed && N % 256 == 0) {
    const NtPlan p = gemm_nt_plan(M, N, K, part ? part_elems : 0);
    if (p.bn == 384) {
      hipExtLaunchKernelGGL((gemm_nt_dma_kernel<384, 128, 4, 2, DMA_NSTAGE>),
                            dim3((M + 127) / 128 * (N / 384)), dim3(8 * WAVE), 0, st, ev0, ev1, 0, x, ldx, w, M, N, K,
                            C, ldc, 1, nullptr);
      ADT_LAUNCH_CHECK();
      return ADT_OK;
    }
    if (p.ksplit > 1 || (int64_t)(N / 256) * ((M + 255) / 256) >= 128) {
      const int n_main = N - p.n_tail;
      launch_dma256(x, ldx, w, M, n_main, K, C, ldc, p.ksplit, part, st, ev0, p.n_tail ? nullptr : ev1);
      ADT_LAUNCH_CHECK();
      if (p.n_tail) {
        launch_dma256(x, ldx, w + (int64_t)(n_main / 16) * (K / 32) * 512, M, p.n_tail, K, C + n_main, ldc, p.tail_ks,
                      part, st, nullptr, ev1);
        ADT_LAUNCH_CHECK();
      }
      return ADT_OK;
    }
  }
  // Packed weights with fewer blocks (the narrow projections of a batch of trees): 128 x 128
  // blocks of four waves through the same DMA pipeline, two workgroups per CU.
  if (packed) {
    const int ks = gemm_nt_ks128(M, N, K, part ? part_elems : 0);
    hipExtLaunchKernelGGL((gemm_nt_dma_kernel<128, 128, 2, 2, DMA_NSTAGE>), dim3((M + 127) / 128 * (N / 128) * ks),
                          dim3(4 * WAVE), 0, st, ev0, ks > 1 ? nullptr : ev1, 0, x, ldx, w, M, N, K, C, ldc, ks, part);
    ADT_LAUNCH_CHECK();
    if (ks > 1) {
      const int64_t quads = (int64_t)M * (N / 4);
      const int blocks = (int)std::min<int64_t>((quads + 255) / 256, 4096);
      hipExtLaunchKernelGGL(gemm_nt_reduce_kernel, dim3(blocks), dim3(256), 0, st, nullptr, ev1, 0, C, ldc,
                            (const float*)part, M, N, ks - 1);
      ADT_LAUNCH_CHECK();
    }
    return ADT_OK;
  }
#define ADT_NT(BNV, BMV, PK)                                                                                    \
  hipExtLaunchKernelGGL(gemm_nt_kernel<BNV, BMV, PK>, dim3((M + BMV - 1) / BMV, N / BNV), dim3(NT_THREADS), 0, st, \
                        ev0, ev1, 0, x, ldx, w, ldw, M, K, C, ldc)
  if (best == 0) {
    if (packed) ADT_NT(256, 256, true);
    else ADT_NT(256, 256, false);
  } else {
    if (packed) ADT_NT(128, 128, true);
    else ADT_NT(128, 128, false);
  }
#undef ADT_NT
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

}  // namespace adt
