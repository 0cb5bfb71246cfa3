// Codebook neighbour table for relaxed acceptance (set-up, not part of a cycle): for every
// code x, itself followed by the k-1 other codes of highest cosine similarity (ties: lower
// id first).  Similarities are an fp32 tiled product of the normalised codebook with
// itself; each row then takes its top k-1 by a 64-bit radix select and a bitonic sort in LDS.
#include "../launch.h"

namespace adt {

constexpr int KNN_T = 64;   // similarity tile

__global__ void knn_norm_kernel(const float* __restrict__ cb, int n, int dim, float* __restrict__ inv) {
  const int i = blockIdx.x * (blockDim.x / WAVE) + threadIdx.x / WAVE, lane = threadIdx.x % WAVE;
  if (i >= n) return;
  float s = 0.f;
  for (int c = lane; c < dim; c += WAVE) s += cb[(int64_t)i * dim + c] * cb[(int64_t)i * dim + c];
  s = wave_sum(s);
  if (lane == 0) inv[i] = 1.f / sqrtf(s);
}

// sim[i][j] = (cb_i . cb_j) * inv_i * inv_j, 64 x 64 tiles, 256 threads (4 x 4 outputs each).
__global__ __launch_bounds__(256) void knn_sim_kernel(const float* __restrict__ cb, const float* __restrict__ inv,
                                                      int n, int dim, float* __restrict__ sim) {
  __shared__ float A[KNN_T][17], Bt[KNN_T][17];
  const int i0 = blockIdx.y * KNN_T, j0 = blockIdx.x * KNN_T;
  const int tx = threadIdx.x % 16, ty = threadIdx.x / 16;
  float acc[4][4] = {};
  for (int c0 = 0; c0 < dim; c0 += 16) {
    for (int p = threadIdx.x; p < KNN_T * 16; p += 256) {
      const int r = p / 16, c = p % 16;
      A[r][c] = (i0 + r < n && c0 + c < dim) ? cb[(int64_t)(i0 + r) * dim + c0 + c] : 0.f;
      Bt[r][c] = (j0 + r < n && c0 + c < dim) ? cb[(int64_t)(j0 + r) * dim + c0 + c] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < 16; ++c)
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = fmaf(A[ty * 4 + a][c], Bt[tx * 4 + b][c], acc[a][b]);
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int i = i0 + ty * 4 + a, j = j0 + tx * 4 + b;
      if (i < n && j < n) sim[(int64_t)i * n + j] = acc[a][b] * inv[i] * inv[j];
    }
}

// Order-preserving key: larger similarity first, then lower id.
__device__ __forceinline__ uint64_t sim_key(float v, int id) {
  uint32_t b = __float_as_uint(v);
  b = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((uint64_t)b << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)id);
}

constexpr int KNN_SEL_THREADS = 256;
constexpr int KNN_KMAX = 256;

__global__ __launch_bounds__(KNN_SEL_THREADS) void knn_select_kernel(const float* __restrict__ sim, int n, int k,
                                                                     int32_t* __restrict__ out) {
  __shared__ uint32_t hist[256];
  __shared__ uint64_t thr_s;
  __shared__ int need_s, cnt_s;
  __shared__ uint64_t keys[KNN_KMAX];
  const int i = blockIdx.x, tid = threadIdx.x;
  const float* row = sim + (int64_t)i * n;
  const int K = k - 1;            // neighbours besides the code itself
  uint64_t prefix = 0, mask = 0;
  int need = K;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int b = tid; b < 256; b += KNN_SEL_THREADS) hist[b] = 0;
    __syncthreads();
    for (int j = tid; j < n; j += KNN_SEL_THREADS) {
      if (j == i) continue;
      const uint64_t key = sim_key(row[j], j);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255], 1u);
    }
    __syncthreads();
    if (tid == 0) {
      int acc = 0, b = 255;
      for (; b > 0; --b) {
        if (acc + (int)hist[b] >= need) break;
        acc += hist[b];
      }
      thr_s = prefix | ((uint64_t)b << shift);
      need_s = need - acc;
    }
    __syncthreads();
    prefix = thr_s;
    need = need_s;
    mask |= (uint64_t)255 << shift;
    __syncthreads();
  }
  // gather the K keys >= threshold, sort descending (bitonic over KNN_KMAX slots)
  if (tid == 0) cnt_s = 0;
  for (int p = tid; p < KNN_KMAX; p += KNN_SEL_THREADS) keys[p] = 0;
  __syncthreads();
  for (int j = tid; j < n; j += KNN_SEL_THREADS) {
    if (j == i) continue;
    const uint64_t key = sim_key(row[j], j);
    if (key >= prefix) keys[atomicAdd(&cnt_s, 1)] = key;
  }
  __syncthreads();
  for (int size = 2; size <= KNN_KMAX; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int p = tid; p < KNN_KMAX; p += KNN_SEL_THREADS) {
        const int q = p ^ stride;
        if (q > p) {
          const bool desc = ((p & size) == 0);
          const uint64_t a = keys[p], b = keys[q];
          if (desc ? (a < b) : (a > b)) {
            keys[p] = b;
            keys[q] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  int32_t* o = out + (int64_t)i * k;
  if (tid == 0) o[0] = i;
  for (int p = tid; p < K; p += KNN_SEL_THREADS) o[p + 1] = (int32_t)(0xFFFFFFFFu - (uint32_t)keys[p]);
}

size_t knn_ws_bytes(int n) { return (size_t)n * n * 4 + (size_t)n * 4 + 256; }

adt_status launch_codebook_knn(const float* cb, int n, int dim, int k, int32_t* out, void* ws, size_t ws_bytes,
                               hipStream_t st) {
  ADT_CHECK_ARG(k >= 1 && k <= KNN_KMAX && k <= n, ADT_E_UNSUPPORTED, "codebook_knn: k=%d (max %d, n=%d)", k,
                KNN_KMAX, n);
  ADT_CHECK_ARG(ws && ws_bytes >= knn_ws_bytes(n), ADT_E_CAPACITY, "codebook_knn: workspace");
  float* sim = (float*)ws;
  float* inv = sim + (size_t)n * n;
  knn_norm_kernel<<<(n + 3) / 4, 256, 0, st>>>(cb, n, dim, inv);
  ADT_LAUNCH_CHECK();
  dim3 g((n + KNN_T - 1) / KNN_T, (n + KNN_T - 1) / KNN_T);
  knn_sim_kernel<<<g, 256, 0, st>>>(cb, inv, n, dim, sim);
  ADT_LAUNCH_CHECK();
  knn_select_kernel<<<n, KNN_SEL_THREADS, 0, st>>>(sim, n, k, out);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

}  // namespace adt
