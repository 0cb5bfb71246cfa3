// Row-wise kernels of the forwards and of the cache bookkeeping: embedding with its norm, the
// finish of a residual projection (K-range sums, residual add, the next norm), the fp32 path's finishing steps after each projection (residual add + RMSNorm, RoPE + KV
// append, SwiGLU, logits), feature gathers, KV compaction and ancestor masks.  Each kernel
// handles whole rows (at most 128 tree rows per launch), so they are latency-bound and kept
// as simple as possible.
#include <algorithm>

#include "../launch.h"

namespace adt {

constexpr int ROW_THREADS = 256;

ADT_DEVICE_ERROR_WORD(rows)

// h[m] = E[tok[m]] (fp32 residual), a[m] = RMSNorm(h[m]) (raw: h[m] itself) in dtype T
// (layout a_pk).
template <typename T>
__global__ __launch_bounds__(ROW_THREADS) void embed_norm_kernel(const T* __restrict__ E, const int32_t* __restrict__ tok,
                                                                 int d, float eps, float* __restrict__ h,
                                                                 T* __restrict__ a, Branches br, int a_pk, int raw) {
  __shared__ float red[16];
  const int m = blockIdx.x;
  const T* e = E + (int64_t)tok[m / br.nb + (m % br.nb) * br.tok_boff] * d;
  float ss = 0.f;
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    const float v = Elem<T>::load(e, i);
    h[(int64_t)m * d + i] = v;
    ss += v * v;
  }
  const float r = raw ? 1.f : rsqrtf(block_sum(ss, red) / d + eps);
  for (int i = threadIdx.x; i < d; i += blockDim.x)
    Elem<T>::store(a, act_index(m, i, d, a_pk), h[(int64_t)m * d + i] * r);
}

// The bf16 form of embed_norm: 8 columns (16 bytes) per thread and step, VPT steps, every
// load issued before the first store.
template <int VPT>
__global__ __launch_bounds__(ROW_THREADS) void embed_norm_bf16_kernel(const uint16_t* __restrict__ E,
                                                                      const int32_t* __restrict__ tok, int d, float eps,
                                                                      float* __restrict__ h, uint16_t* __restrict__ a,
                                                                      Branches br, int a_pk, int raw) {
  __shared__ float red[16];
  const int m = blockIdx.x;
  const uint16_t* e = E + (int64_t)tok[m / br.nb + (m % br.nb) * br.tok_boff] * d;
  u16x8 v[VPT];
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int c = (j * ROW_THREADS + threadIdx.x) * 8;
    if (c < d) v[j] = *reinterpret_cast<const u16x8*>(e + c);
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int c = (j * ROW_THREADS + threadIdx.x) * 8;
    if (c >= d) continue;
    float f[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      f[t] = bf2f(v[j][t]);
      ss += f[t] * f[t];
    }
    float* hp = h + (int64_t)m * d + c;
    *reinterpret_cast<float4*>(hp) = make_float4(f[0], f[1], f[2], f[3]);
    *reinterpret_cast<float4*>(hp + 4) = make_float4(f[4], f[5], f[6], f[7]);
    if (raw) *reinterpret_cast<u16x8*>(a + act_index(m, c, d, a_pk)) = v[j];
  }
  if (raw) return;
  const float r = rsqrtf(block_sum(ss, red) / d + eps);
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int c = (j * ROW_THREADS + threadIdx.x) * 8;
    if (c >= d) continue;
    u16x8 o;
#pragma unroll
    for (int t = 0; t < 8; ++t) o[t] = f2bf(bf2f(v[j][t]) * r);
    *reinterpret_cast<u16x8*>(a + act_index(m, c, d, a_pk)) = o;
  }
}

// Finish of a residual projection, one row per workgroup: the K-range sums of the row are
// added in range order, added to (or, with assign, written as) the residual row, and the
// row's RMSNorm is stored in the model dtype for the next projection (layout out_pk; out2, if
// given, gets a second copy in layout out2_pk).  With at most 128 rows the launch is a few
// dozen workgroups, so its time is load latency: every thread requests all S sums and the
// residual of its columns (VPT groups of 4) before adding any, and keeps them for the norm.
template <typename T, int VPT, int S>
__global__ __launch_bounds__(1024) void resid_norm_kernel(const float* __restrict__ part, int M, int d, int assign,
                                                          float eps, float* __restrict__ h, T* __restrict__ out,
                                                          int out_pk, T* __restrict__ out2, int out2_pk) {
  __shared__ float red[16];
  const int m = blockIdx.x;
  const int64_t split = (int64_t)M * d;
  float* hr = h + (int64_t)m * d;
  const float* pr = part + (int64_t)m * d;
  float4 y[VPT];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int i = (j * blockDim.x + threadIdx.x) * 4;
    if (i >= d) continue;
    float4 w[S];
#pragma unroll
    for (int sp = 0; sp < S; ++sp) w[sp] = *reinterpret_cast<const float4*>(pr + sp * split + i);
    const float4 o = assign ? make_float4(0.f, 0.f, 0.f, 0.f) : *reinterpret_cast<const float4*>(hr + i);
    float4 v = w[0];
#pragma unroll
    for (int sp = 1; sp < S; ++sp) v = make_float4(v.x + w[sp].x, v.y + w[sp].y, v.z + w[sp].z, v.w + w[sp].w);
    if (!assign) v = make_float4(o.x + v.x, o.y + v.y, o.z + v.z, o.w + v.w);
    *reinterpret_cast<float4*>(hr + i) = v;
    y[j] = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  const float r = rsqrtf(block_sum(ss, red) / d + eps);
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int i = (j * blockDim.x + threadIdx.x) * 4;
    if (i >= d) continue;
    // four columns from a multiple of 4: contiguous in either layout
    store4(out + act_index(m, i, d, out_pk), y[j].x * r, y[j].y * r, y[j].z * r, y[j].w * r);
    if (out2) store4(out2 + act_index(m, i, d, out2_pk), y[j].x * r, y[j].y * r, y[j].z * r, y[j].w * r);
  }
}

// The bf16 form of draft_input: 8 columns per thread and step, loads first.
template <int VPT>
__global__ __launch_bounds__(ROW_THREADS) void draft_input_bf16_kernel(const uint16_t* __restrict__ E,
                                                                       const int32_t* __restrict__ tok,
                                                                       const int32_t* __restrict__ fsrc,
                                                                       const uint16_t* __restrict__ fa,
                                                                       const uint16_t* __restrict__ fb, int d,
                                                                       uint16_t* __restrict__ x, Branches br, int x_pk) {
  const int m = blockIdx.x, node = m / br.nb, b = m % br.nb;
  const uint16_t* e = E + (int64_t)tok[node + b * br.tok_boff] * d;
  const int s = fsrc[node];
  const uint16_t* f = s >= 0 ? fa + ((int64_t)s * br.nb + b) * d
                             : (s <= -2 ? fb + ((int64_t)(-s - 2) * br.nb + b) * d : nullptr);
  u16x8 ev[VPT], fv[VPT];
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int c = (j * ROW_THREADS + threadIdx.x) * 8;
    if (c >= d) continue;
    ev[j] = *reinterpret_cast<const u16x8*>(e + c);
    fv[j] = f ? *reinterpret_cast<const u16x8*>(f + c) : u16x8{0, 0, 0, 0, 0, 0, 0, 0};
  }
#pragma unroll
  for (int j = 0; j < VPT; ++j) {
    const int c = (j * ROW_THREADS + threadIdx.x) * 8;
    if (c >= d) continue;
    *reinterpret_cast<u16x8*>(x + act_index(m, c, 2 * d, x_pk)) = ev[j];
    *reinterpret_cast<u16x8*>(x + act_index(m, d + c, 2 * d, x_pk)) = fv[j];
  }
}

// Rows of 16-byte pieces: dst[i] = src[idx[i]], every piece of a thread loaded before any store.
__global__ __launch_bounds__(ROW_THREADS) void gather_rows16_kernel(const u16x8* __restrict__ src,
                                                                    const int32_t* __restrict__ idx, int pieces,
                                                                    u16x8* __restrict__ dst) {
  const int i = blockIdx.x;
  const u16x8* s = src + (int64_t)idx[i] * pieces;
  u16x8* o = dst + (int64_t)i * pieces;
  for (int c0 = 0; c0 < pieces; c0 += 4 * ROW_THREADS) {
    u16x8 v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = c0 + j * ROW_THREADS + threadIdx.x;
      if (c < pieces) v[j] = s[c];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = c0 + j * ROW_THREADS + threadIdx.x;
      if (c < pieces) o[c] = v[j];
    }
  }
}

// The finish without the norm: element-wise over the M x d residual, four columns per thread;
// the S sums are requested before any is added, and added in range order.
template <int S>
__global__ __launch_bounds__(ROW_THREADS) void resid_add_kernel(const float* __restrict__ part, int M, int d, int assign,
                                                                float* __restrict__ h, uint16_t* __restrict__ out,
                                                                int out_pk) {
  const int64_t i4 = (int64_t)blockIdx.x * ROW_THREADS + threadIdx.x, n4 = (int64_t)M * d / 4;
  if (i4 >= n4) return;
  const int64_t i = i4 * 4, split = (int64_t)M * d;
  float4 w[S];
#pragma unroll
  for (int sp = 0; sp < S; ++sp) w[sp] = *reinterpret_cast<const float4*>(part + sp * split + i);
  const float4 o = assign ? make_float4(0.f, 0.f, 0.f, 0.f) : *reinterpret_cast<const float4*>(h + i);
  float4 v = w[0];
#pragma unroll
  for (int sp = 1; sp < S; ++sp) v = make_float4(v.x + w[sp].x, v.y + w[sp].y, v.z + w[sp].z, v.w + w[sp].w);
  if (!assign) v = make_float4(o.x + v.x, o.y + v.y, o.z + v.z, o.w + v.w);
  *reinterpret_cast<float4*>(h + i) = v;
  const int m = (int)(i / d), c = (int)(i % d);
  store4(out + act_index(m, c, d, out_pk), v.x, v.y, v.z, v.w);
}

// Draft-head input row m: [E[tok[m]] ; parent feature].  fsrc[m] >= 0 picks row fsrc of the
// committed-feature buffer fa, fsrc[m] == -1 gives zeros, fsrc[m] <= -2 picks row -fsrc-2 of
// the draft-feature buffer fb.  x is [M][2d] in layout x_pk.
template <typename T>
__global__ __launch_bounds__(ROW_THREADS) void draft_input_kernel(const T* __restrict__ E, const int32_t* __restrict__ tok,
                                                                  const int32_t* __restrict__ fsrc, const T* __restrict__ fa,
                                                                  const T* __restrict__ fb, int d, T* __restrict__ x,
                                                                  Branches br, int x_pk) {
  const int m = blockIdx.x, node = m / br.nb, b = m % br.nb;
  const T* e = E + (int64_t)tok[node + b * br.tok_boff] * d;
  const int s = fsrc[node];
  // feature sources hold the branches of one node in consecutive rows
  const T* f = s >= 0 ? fa + ((int64_t)s * br.nb + b) * d
                      : (s <= -2 ? fb + ((int64_t)(-s - 2) * br.nb + b) * d : nullptr);
  for (int i = threadIdx.x; i < d; i += blockDim.x) {
    x[act_index(m, i, 2 * d, x_pk)] = e[i];
    const int64_t xf = act_index(m, d + i, 2 * d, x_pk);
    if (f) x[xf] = f[i];
    else Elem<T>::store(x, xf, 0.f);
  }
}

// Sum of the split-K partials of four consecutive columns.
// Summed in split order so results do not depend on the launch shape; loads are issued
// eight at a time.
__device__ __forceinline__ float4 sum_parts4(const float* __restrict__ part, int splits, int64_t stride, int64_t off) {
  float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
  int s = 0;
  for (; s + 8 <= splits; s += 8) {
    float4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = *reinterpret_cast<const float4*>(part + (s + j) * stride + off);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      y.x += v[j].x;
      y.y += v[j].y;
      y.z += v[j].z;
      y.w += v[j].w;
    }
  }
  for (; s < splits; ++s) {
    const float4 v = *reinterpret_cast<const float4*>(part + s * stride + off);
    y.x += v.x;
    y.y += v.y;
    y.z += v.z;
    y.w += v.w;
  }
  return y;
}

// y = sum_s part[s][m][:]; h[m] = (assign ? y : h[m] + y); if a: a[m] = RMSNorm(h[m]).
// One block per row, four columns per thread (d % 4 == 0, d <= 4 * blockDim.x * 4).
template <typename T>
__global__ __launch_bounds__(1024) void add_norm_kernel(const float* __restrict__ part, int splits, int M, int d,
                                                        int assign, float eps, float* __restrict__ h,
                                                        T* __restrict__ a) {
  __shared__ float red[16];
  const int m = blockIdx.x;
  const int64_t stride = (int64_t)M * d;
  float4 hv[4];
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int c = (threadIdx.x + it * blockDim.x) * 4;
    if (c < d) {
      const float4 y = sum_parts4(part, splits, stride, (int64_t)m * d + c);
      float4 v = y;
      if (!assign) {
        const float4 o = *reinterpret_cast<const float4*>(h + (int64_t)m * d + c);
        v = make_float4(o.x + y.x, o.y + y.y, o.z + y.z, o.w + y.w);
      }
      *reinterpret_cast<float4*>(h + (int64_t)m * d + c) = v;
      hv[it] = v;
      ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
  }
  if (a == nullptr) return;
  const float r = rsqrtf(block_sum(ss, red) / d + eps);
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int c = (threadIdx.x + it * blockDim.x) * 4;
    if (c < d) {
      T* out = a + (int64_t)m * d + c;
      Elem<T>::store(out, 0, hv[it].x * r);
      Elem<T>::store(out, 1, hv[it].y * r);
      Elem<T>::store(out, 2, hv[it].z * r);
      Elem<T>::store(out, 3, hv[it].w * r);
    }
  }
}

// cos / sin of rotate-half RoPE for every slot position: tab[p][j] = (cos, sin)(p * theta^(-2j/Dh)),
// computed in double precision and stored as fp32.
__global__ void rope_table_kernel(float2* __restrict__ tab, int positions, int half, int Dh, double theta) {
  const int64_t total = (int64_t)positions * half;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int p = (int)(i / half), j = (int)(i % half);
    double sn, cs;
    sincos((double)p * pow(theta, -2.0 * j / Dh), &sn, &cs);
    tab[i] = make_float2((float)cs, (float)sn);
  }
}

// Sum the QKV partials of row m, rotate q and k at position pos[m] (table lookup), write q to
// qout[m][H][Dh] and k, v to cache slot (*slot0 + m) of every head.  Cache element
// (h, slot, :) at kc + h*stride_h + slot*Dh.  Grid (M, pairs / 256), one (head, pair) per thread.
template <typename T>
__global__ __launch_bounds__(ROW_THREADS) void qkv_rope_kernel(const float* __restrict__ part, int splits, int M,
                                                               int H, int Dh, const int32_t* __restrict__ pos,
                                                               const int32_t* __restrict__ slot0,
                                                               const float2* __restrict__ rope, T* __restrict__ qout,
                                                               T* __restrict__ kc, T* __restrict__ vc,
                                                               int64_t stride_h, Branches br) {
  const int m = blockIdx.x, node = m / br.nb;
  const int d = H * Dh, N = 3 * d, half = Dh / 2;
  const int i = blockIdx.y * blockDim.x + threadIdx.x;
  if (i >= H * half) return;
  const int hh = i / half, j = i % half;
  const int64_t stride = (int64_t)M * N, row = (int64_t)m * N;
  const int c1 = hh * Dh + j, c2 = c1 + half;
  float q1 = 0.f, q2 = 0.f, k1 = 0.f, k2 = 0.f, v1 = 0.f, v2 = 0.f;
#pragma unroll 4
  for (int s = 0; s < splits; ++s) {
    const float* p = part + s * stride + row;
    q1 += p[c1];
    q2 += p[c2];
    k1 += p[d + c1];
    k2 += p[d + c2];
    v1 += p[2 * d + c1];
    v2 += p[2 * d + c2];
  }
  const float2 cs = rope[(int64_t)pos[node] * half + j];
  const int64_t slot = *slot0 + node;
  kc += (m % br.nb) * br.cache_sb;
  vc += (m % br.nb) * br.cache_sb;
  Elem<T>::store(qout, (int64_t)m * d + c1, q1 * cs.x - q2 * cs.y);
  Elem<T>::store(qout, (int64_t)m * d + c2, q2 * cs.x + q1 * cs.y);
  T* kr = kc + hh * stride_h + slot * Dh;
  Elem<T>::store(kr, j, k1 * cs.x - k2 * cs.y);
  Elem<T>::store(kr, j + half, k2 * cs.x + k1 * cs.y);
  T* vr = vc + hh * stride_h + slot * Dh;
  Elem<T>::store(vr, j, v1);
  Elem<T>::store(vr, j + half, v2);
}

// Batched verify, after the QKV projection of packed-order weights: C[m][3d] fp32 whose
// columns follow the ADT_PACK_QKV row order (within a head, 16-column tile u holds dims
// 8u..8u+7 of the head's first half, then the same dims of its second half: RoPE pairs
// sit 8 columns apart).  Row m belongs to sequence seq[m], position pos[m], cache slot
// slot[m]; q row m gets the rotated query, the caches of its sequence (base + seq *
// cache_sb) the rotated key and the value, all in the head's natural dim order.
// Grid (M, pairs / 256 rounded up); one RoPE pair per thread.
template <typename T>
__global__ __launch_bounds__(ROW_THREADS) void qkv_rows_kernel(const float* __restrict__ C, int H, int Dh,
                                                               const int32_t* __restrict__ pos,
                                                               const int32_t* __restrict__ slot,
                                                               const int32_t* __restrict__ seq,
                                                               const float2* __restrict__ rope, T* __restrict__ qout,
                                                               T* __restrict__ kc, T* __restrict__ vc, int64_t stride_h,
                                                               int64_t cache_sb) {
  const int m = blockIdx.x;
  const int d = H * Dh, half = Dh / 2;
  const int i = blockIdx.y * blockDim.x + threadIdx.x;
  if (i >= H * half) return;
  const int hh = i / half, j = i % half;
  const int c1 = hh * Dh + (j / 8) * 16 + j % 8, c2 = c1 + 8;     // packed columns of dims j, j + half
  const float* row = C + (int64_t)m * 3 * d;
  const float2 cs = rope[(int64_t)pos[m] * half + j];
  const float q1 = row[c1], q2 = row[c2], k1 = row[d + c1], k2 = row[d + c2];
  Elem<T>::store(qout, (int64_t)m * d + hh * Dh + j, q1 * cs.x - q2 * cs.y);
  Elem<T>::store(qout, (int64_t)m * d + hh * Dh + j + half, q2 * cs.x + q1 * cs.y);
  const int64_t off = (int64_t)seq[m] * cache_sb + hh * stride_h + (int64_t)slot[m] * Dh;
  Elem<T>::store(kc + off, j, k1 * cs.x - k2 * cs.y);
  Elem<T>::store(kc + off, j + half, k2 * cs.x + k1 * cs.y);
  Elem<T>::store(vc + off, j, row[2 * d + c1]);
  Elem<T>::store(vc + off, j + half, row[2 * d + c2]);
}

// SwiGLU over gate/up products packed in interleaved 8-column blocks: out[m][j] = silu(g) u.
// Grid (M, F / (4 * 256)); four consecutive outputs per thread.
template <typename T>
__global__ __launch_bounds__(ROW_THREADS) void swiglu_kernel(const float* __restrict__ part, int splits, int M, int F,
                                                             T* __restrict__ out) {
  const int m = blockIdx.x, N = 2 * F;
  const int j = (blockIdx.y * blockDim.x + threadIdx.x) * 4;
  if (j >= F) return;
  const int cg = (j / 8) * 16 + j % 8;
  const int64_t stride = (int64_t)M * N, row = (int64_t)m * N;
  const float4 g = sum_parts4(part, splits, stride, row + cg);
  const float4 u = sum_parts4(part, splits, stride, row + cg + 8);
  T* o = out + (int64_t)m * F + j;
  Elem<T>::store(o, 0, g.x / (1.f + expf(-g.x)) * u.x);
  Elem<T>::store(o, 1, g.y / (1.f + expf(-g.y)) * u.y);
  Elem<T>::store(o, 2, g.z / (1.f + expf(-g.z)) * u.z);
  Elem<T>::store(o, 3, g.w / (1.f + expf(-g.w)) * u.w);
}

// out[m][n] = sum_s part[s][m][n]  (logits).
__global__ void reduce_store_kernel(const float* __restrict__ part, int splits, int M, int N, float* __restrict__ out,
                                    int64_t ldo) {
  const int m = blockIdx.y;
  for (int n = blockIdx.x * blockDim.x + threadIdx.x; n < N; n += gridDim.x * blockDim.x) {
    float y = 0.f;
    for (int s = 0; s < splits; ++s) y += part[((int64_t)s * M + m) * N + n];
    out[(int64_t)m * ldo + n] = y;
  }
}

// dst[i] = src[idx[i]] for i < cnt (rows of length d, element type T).
template <typename T>
__global__ void gather_rows_kernel(const T* __restrict__ src, const int32_t* __restrict__ idx, int d,
                                   T* __restrict__ dst) {
  const int i = blockIdx.x;
  const T* s = src + (int64_t)idx[i] * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) dst[(int64_t)i * d + c] = s[c];
}

// KV compaction: one block per (group of G slices, sequence); piece p of a block is 16
// bytes of row m of slice p / pps of the group (pps = a_max rows of 16-byte pieces).  Every
// moved row of a slice is read into registers before any is written (one barrier), so
// in-place moves never read a row already overwritten; a slice never spans two blocks.
template <typename T, int ROWS_MAX>
__global__ __launch_bounds__(ROW_THREADS) void kv_compact_kernel(T* __restrict__ kc, T* __restrict__ vc, int Dh,
                                                                 int64_t stride_b, int64_t stride_s,
                                                                 const int32_t* __restrict__ kv_len, int kv_stride,
                                                                 const int32_t* __restrict__ path, int path_stride,
                                                                 const int32_t* __restrict__ n_acc, int acc_stride,
                                                                 int a_max, int slices, int G) {
  const int b = blockIdx.y, s0 = blockIdx.x * G;
  const int a = min(n_acc[b * acc_stride], a_max);
  const int L = kv_len[b * kv_stride];
  const int per_row = Dh * (int)sizeof(T) / 16;        // 16-byte pieces per row
  const int pps = a_max * per_row;                     // pieces per slice
  const int total = G * pps;
  u16x8 kr[ROWS_MAX], vr[ROWS_MAX];
#pragma unroll
  for (int it = 0; it < ROWS_MAX; ++it) {
    const int p = threadIdx.x + it * ROW_THREADS;
    if (p < total) {
      const int sl = s0 + p / pps, w = p % pps, m = w / per_row + 1, c = w % per_row;
      if (sl < slices && m <= a) {
        // the node at depth m of a BFS-ordered tree has an index in [m, ADT_MAX_NODES); an
        // entry outside is recorded (debug builds) and its row left in place
        const int src = path[(int64_t)b * path_stride + m];
        if (src >= m && src < ADT_MAX_NODES) {
          const int64_t off = b * stride_b + sl * stride_s + (int64_t)(L + src) * Dh;
          kr[it] = reinterpret_cast<const u16x8*>(kc + off)[c];
          vr[it] = reinterpret_cast<const u16x8*>(vc + off)[c];
        } else {
          dev_fail(DEVINV_PATH);
        }
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < ROWS_MAX; ++it) {
    const int p = threadIdx.x + it * ROW_THREADS;
    if (p < total) {
      const int sl = s0 + p / pps, w = p % pps, m = w / per_row + 1, c = w % per_row;
      const int src = (sl < slices && m <= a) ? path[(int64_t)b * path_stride + m] : -1;
      if (sl < slices && m <= a && src >= m && src < ADT_MAX_NODES) {
        const int64_t off = b * stride_b + sl * stride_s + (int64_t)(L + m) * Dh;
        reinterpret_cast<u16x8*>(kc + off)[c] = kr[it];
        reinterpret_cast<u16x8*>(vc + off)[c] = vr[it];
      }
    }
  }
}

// Classifier-free guidance on logits: out[i][v] = u + s (c - u) with c = raw[2i][v] (the
// conditional branch) and u = raw[2i + 1][v].  Grid (V / 4 / 256 rounded up, rows).
__global__ void guide_rows_kernel(const float* __restrict__ raw, int V, float scale, float* __restrict__ out,
                                  int64_t ldo) {
  const int i = blockIdx.y;
  const float* c = raw + (int64_t)2 * i * V;
  const float* u = c + V;
  float* o = out + (int64_t)i * ldo;
  const int v = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (v + 4 <= V) {
    const float4 a = *reinterpret_cast<const float4*>(c + v), b = *reinterpret_cast<const float4*>(u + v);
    *reinterpret_cast<float4*>(o + v) =
        make_float4(b.x + scale * (a.x - b.x), b.y + scale * (a.y - b.y), b.z + scale * (a.z - b.z),
                    b.w + scale * (a.w - b.w));
  } else {
    for (int j = v; j < V; ++j) o[j] = u[j] + scale * (c[j] - u[j]);
  }
}

// Ancestor masks and depths of B BFS-ordered trees; one thread per tree.
__global__ void tree_masks_kernel(const int32_t* __restrict__ parent, const int32_t* __restrict__ n_nodes, int B,
                                  int n_max, uint64_t* __restrict__ mask, int32_t* __restrict__ depth) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int n = min(n_nodes[b], n_max);
  const int32_t* par = parent + (int64_t)b * n_max;
  uint64_t* mk = mask + (int64_t)b * n_max * ADT_MASK_WORDS;
  for (int i = 0; i < n_max; ++i) {
    uint64_t w0 = 0, w1 = 0;
    int dp = 0;
    if (i < n) {
      const int p = par[i];
      if (i == 0 ? p != -1 : !(p >= 0 && p < i)) dev_fail(DEVINV_PARENT);
      if (i > 0 && p >= 0 && p < i) {
        w0 = mk[p * ADT_MASK_WORDS];
        w1 = mk[p * ADT_MASK_WORDS + 1];
        if (depth) dp = depth[(int64_t)b * n_max + p] + 1;
      }
      if (i < 64) w0 |= 1ull << i;
      else w1 |= 1ull << (i - 64);
    }
    mk[i * ADT_MASK_WORDS] = w0;
    mk[i * ADT_MASK_WORDS + 1] = w1;
    if (depth) depth[(int64_t)b * n_max + i] = dp;
  }
}

// ----------------------------------------------------------------------------- host
#define ADT_DISPATCH_T(dtype, ...)             \
  if ((dtype) == ADT_BF16) {                   \
    using T = uint16_t;                        \
    __VA_ARGS__;                               \
  } else {                                     \
    using T = float;                           \
    __VA_ARGS__;                               \
  }

// A fragment layout needs bf16, K % 32 == 0 and enough row blocks for M rows.
static bool frag_ok(int pk, int M, int K, int dtype) {
  return pk == 0 || (dtype == ADT_BF16 && K % 32 == 0 && pk * 16 >= M);
}

adt_status launch_embed_norm(const void* E, const int32_t* tok, int M, int d, float eps, float* h, void* a, int dtype,
                             hipStream_t st, const Branches& br, int a_pk, bool raw) {
  ADT_CHECK_ARG(a != nullptr && h != nullptr, ADT_E_ARG, "embed_norm: outputs");
  ADT_CHECK_ARG(frag_ok(a_pk, M, d, dtype), ADT_E_SHAPE, "embed_norm: fragment layout of %d blocks for %d x %d", a_pk,
                M, d);
  if (dtype == ADT_BF16 && d % 8 == 0 && d <= 4 * 8 * ROW_THREADS) {
    const int vpt = (d + 8 * ROW_THREADS - 1) / (8 * ROW_THREADS);
#define ADT_EN(V)                                                                                                 \
  embed_norm_bf16_kernel<V><<<M, ROW_THREADS, 0, st>>>((const uint16_t*)E, tok, d, eps, h, (uint16_t*)a, br, a_pk, \
                                                       raw ? 1 : 0)
    if (vpt <= 1) ADT_EN(1);
    else if (vpt <= 2) ADT_EN(2);
    else ADT_EN(4);
#undef ADT_EN
  } else {
    ADT_DISPATCH_T(dtype, embed_norm_kernel<T><<<M, ROW_THREADS, 0, st>>>((const T*)E, tok, d, eps, h, (T*)a, br, a_pk,
                                                                           raw ? 1 : 0));
  }
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_resid_norm(const float* part, int S, int M, int d, int assign, float eps, float* h, void* out,
                             int out_pk, void* out2, int out2_pk, int dtype, hipStream_t st) {
  ADT_CHECK_ARG(part && h && out && S >= 1 && S <= GEMM_MAX_SPLITS && M >= 1, ADT_E_ARG, "resid_norm: bad arguments");
  ADT_CHECK_ARG(d % 4 == 0 && d <= 2 * 4 * 1024, ADT_E_SHAPE, "resid_norm: d=%d (a multiple of 4, <= 8192)", d);
  ADT_CHECK_ARG(frag_ok(out_pk, M, d, dtype) && frag_ok(out2 ? out2_pk : 0, M, d, dtype), ADT_E_SHAPE,
                "resid_norm: fragment layouts %d / %d for %d x %d", out_pk, out2_pk, M, d);
  // one group of 4 columns per thread up to 4096 columns (1024 threads), two beyond
  const int vpt = d > 4 * 1024 ? 2 : 1;
  const int threads = std::max(WAVE, (d / 4 / vpt + WAVE - 1) / WAVE * WAVE);
#define ADT_RN(V, SV)                                                                                          \
  resid_norm_kernel<T, V, SV><<<M, threads, 0, st>>>(part, M, d, assign, eps, h, (T*)out, out_pk, (T*)out2, \
                                                     out2_pk)
#define ADT_RN_S(V)                  \
  switch (S) {                       \
    case 1: ADT_RN(V, 1); break;     \
    case 2: ADT_RN(V, 2); break;     \
    case 3: ADT_RN(V, 3); break;     \
    case 4: ADT_RN(V, 4); break;     \
    case 5: ADT_RN(V, 5); break;     \
    case 6: ADT_RN(V, 6); break;     \
    case 7: ADT_RN(V, 7); break;     \
    default: ADT_RN(V, 8); break;    \
  }
  ADT_DISPATCH_T(dtype, if (vpt == 1) { ADT_RN_S(1) } else { ADT_RN_S(2) });
#undef ADT_RN_S
#undef ADT_RN
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_resid_add(const float* part, int S, int M, int d, int assign, float* h, void* out, int out_pk,
                            hipStream_t st) {
  ADT_CHECK_ARG(part && h && out && S >= 1 && S <= GEMM_MAX_SPLITS && M >= 1, ADT_E_ARG, "resid_add: bad arguments");
  ADT_CHECK_ARG(d % 4 == 0 && frag_ok(out_pk, M, d, ADT_BF16), ADT_E_SHAPE, "resid_add: %d x %d (layout %d)", M, d,
                out_pk);
  const int blocks = (int)(((int64_t)M * d / 4 + ROW_THREADS - 1) / ROW_THREADS);
#define ADT_RA(SV) \
  resid_add_kernel<SV><<<blocks, ROW_THREADS, 0, st>>>(part, M, d, assign, h, (uint16_t*)out, out_pk)
  switch (S) {
    case 1: ADT_RA(1); break;
    case 2: ADT_RA(2); break;
    case 3: ADT_RA(3); break;
    case 4: ADT_RA(4); break;
    case 5: ADT_RA(5); break;
    case 6: ADT_RA(6); break;
    case 7: ADT_RA(7); break;
    default: ADT_RA(8); break;
  }
#undef ADT_RA
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_draft_input(const void* E, const int32_t* tok, const int32_t* fsrc, const void* fa, const void* fb,
                              int M, int d, void* x, int dtype, hipStream_t st, const Branches& br, int x_pk) {
  ADT_CHECK_ARG(frag_ok(x_pk, M, 2 * d, dtype), ADT_E_SHAPE, "draft_input: fragment layout of %d blocks for %d x %d",
                x_pk, M, 2 * d);
  if (dtype == ADT_BF16 && d % 8 == 0 && d <= 4 * 8 * ROW_THREADS) {
    const int vpt = (d + 8 * ROW_THREADS - 1) / (8 * ROW_THREADS);
#define ADT_DI(V)                                                                                                  \
  draft_input_bf16_kernel<V><<<M, ROW_THREADS, 0, st>>>((const uint16_t*)E, tok, fsrc, (const uint16_t*)fa,       \
                                                        (const uint16_t*)fb, d, (uint16_t*)x, br, x_pk)
    if (vpt <= 1) ADT_DI(1);
    else if (vpt <= 2) ADT_DI(2);
    else ADT_DI(4);
#undef ADT_DI
  } else {
    ADT_DISPATCH_T(dtype, draft_input_kernel<T><<<M, ROW_THREADS, 0, st>>>((const T*)E, tok, fsrc, (const T*)fa,
                                                                            (const T*)fb, d, (T*)x, br, x_pk));
  }
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_add_norm(const float* part, int splits, int M, int d, int assign, float eps, float* h, void* a,
                           int dtype, hipStream_t st) {
  ADT_CHECK_ARG(d % 4 == 0 && d <= 16 * 1024, ADT_E_SHAPE, "add_norm: d=%d", d);
  int threads = (d / 4 + 63) / 64 * 64;   // one float4 column group per thread when d <= 4096
  if (threads > 1024) threads = 1024;
  if (threads < 64) threads = 64;
  ADT_DISPATCH_T(dtype, add_norm_kernel<T><<<M, threads, 0, st>>>(part, splits, M, d, assign, eps, h, (T*)a));
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_rope_table(float2* tab, int positions, int Dh, double theta, hipStream_t st) {
  rope_table_kernel<<<512, 256, 0, st>>>(tab, positions, Dh / 2, Dh, theta);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_qkv_rope(const float* part, int splits, int M, int H, int Dh, const int32_t* pos,
                           const int32_t* slot0, const float2* rope, void* qout, void* kc, void* vc, int64_t stride_h,
                           int dtype, hipStream_t st, const Branches& br) {
  dim3 grid(M, (H * Dh / 2 + ROW_THREADS - 1) / ROW_THREADS);
  ADT_DISPATCH_T(dtype, qkv_rope_kernel<T><<<grid, ROW_THREADS, 0, st>>>(part, splits, M, H, Dh, pos, slot0, rope,
                                                                          (T*)qout, (T*)kc, (T*)vc, stride_h, br));
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_qkv_rows(const float* C, int M, int H, int Dh, const int32_t* pos, const int32_t* slot,
                           const int32_t* seq, const float2* rope, void* qout, void* kc, void* vc, int64_t stride_h,
                           int64_t cache_sb, int dtype, hipStream_t st) {
  ADT_CHECK_ARG(Dh % 16 == 0, ADT_E_SHAPE, "qkv_rows: head_dim %d", Dh);
  if (M <= 0) return ADT_OK;
  dim3 grid(M, (H * Dh / 2 + ROW_THREADS - 1) / ROW_THREADS);
  ADT_DISPATCH_T(dtype, qkv_rows_kernel<T><<<grid, ROW_THREADS, 0, st>>>(C, H, Dh, pos, slot, seq, rope, (T*)qout,
                                                                          (T*)kc, (T*)vc, stride_h, cache_sb));
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_swiglu(const float* part, int splits, int M, int F, void* out, int dtype, hipStream_t st) {
  ADT_CHECK_ARG(F % 16 == 0, ADT_E_SHAPE, "swiglu: F=%d", F);
  dim3 grid(M, (F / 4 + ROW_THREADS - 1) / ROW_THREADS);
  ADT_DISPATCH_T(dtype, swiglu_kernel<T><<<grid, ROW_THREADS, 0, st>>>(part, splits, M, F, (T*)out));
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_reduce_store(const float* part, int splits, int M, int N, float* out, int64_t ldo, hipStream_t st) {
  dim3 grid((N + 1023) / 1024 < 64 ? (N + 1023) / 1024 : 64, M);
  reduce_store_kernel<<<grid, 1024, 0, st>>>(part, splits, M, N, out, ldo);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_gather_rows(const void* src, const int32_t* idx, int cnt, int d, void* dst, int dtype,
                              hipStream_t st) {
  if (cnt <= 0) return ADT_OK;
  const int64_t row_bytes = (int64_t)d * (dtype == ADT_BF16 ? 2 : 4);
  if (row_bytes % 16 == 0 && ((uintptr_t)src | (uintptr_t)dst) % 16 == 0) {
    gather_rows16_kernel<<<cnt, ROW_THREADS, 0, st>>>((const u16x8*)src, idx, (int)(row_bytes / 16), (u16x8*)dst);
  } else {
    ADT_DISPATCH_T(dtype, gather_rows_kernel<T><<<cnt, ROW_THREADS, 0, st>>>((const T*)src, idx, d, (T*)dst));
  }
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_kv_compact(void* k, void* v, int B, int slices, int Dh, int64_t sb, int64_t ss, const int32_t* kv_len,
                             int kv_stride, const int32_t* path, int path_stride, const int32_t* n_acc, int acc_stride,
                             int a_max, int dtype, hipStream_t st) {
  const int bytes_row = Dh * (dtype == ADT_BF16 ? 2 : 4);
  ADT_CHECK_ARG(bytes_row % 16 == 0, ADT_E_SHAPE, "kv_compact: row of %d bytes not a multiple of 16", bytes_row);
  const int pieces = a_max * bytes_row / 16;   // per slice
  ADT_CHECK_ARG(pieces <= 16 * ROW_THREADS, ADT_E_UNSUPPORTED,
                "kv_compact: %d accepted rows of %d bytes exceed one block's %d-byte staging", a_max, bytes_row,
                16 * ROW_THREADS * 16);
  // as many whole slices per block as its registers hold (one slice when a slice fills them)
  const int rm = pieces <= 4 * ROW_THREADS ? 4 : 16;
  const int G = std::max(1, std::min(slices, rm * ROW_THREADS / std::max(pieces, 1)));
  dim3 grid((slices + G - 1) / G, B);
#define ADT_COMPACT(T, RM)                                                                                        \
  kv_compact_kernel<T, RM><<<grid, ROW_THREADS, 0, st>>>((T*)k, (T*)v, Dh, sb, ss, kv_len, kv_stride, path,       \
                                                         path_stride, n_acc, acc_stride, a_max, slices, G)
  if (dtype == ADT_BF16) {
    if (rm == 4) ADT_COMPACT(uint16_t, 4);
    else ADT_COMPACT(uint16_t, 16);
  } else {
    if (rm == 4) ADT_COMPACT(float, 4);
    else ADT_COMPACT(float, 16);
  }
#undef ADT_COMPACT
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_guide_rows(const float* raw, int rows, int V, float scale, float* out, int64_t ldo, hipStream_t st) {
  if (rows <= 0) return ADT_OK;
  dim3 grid((V / 4 + ROW_THREADS) / ROW_THREADS, rows);
  guide_rows_kernel<<<grid, ROW_THREADS, 0, st>>>(raw, V, scale, out, ldo);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_tree_masks(const int32_t* parent, const int32_t* n_nodes, int B, int n_max, uint64_t* mask,
                             int32_t* depth, hipStream_t st) {
  tree_masks_kernel<<<(B + 63) / 64, 64, 0, st>>>(parent, n_nodes, B, n_max, mask, depth);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

}  // namespace adt
