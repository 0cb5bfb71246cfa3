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

adt_status launch_gemm_nt(const void* X, int64_t ldx, const void* W, int64_t ldw, int M, int N, int K, float* C,
                          int64_t ldc, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1, bool packed) {
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
