// Tree attention (Sec. 3.1): every tree node attends to the committed prefix and to the
// nodes on its own root-to-node path (the ancestor bitmask).
//
// bf16 path: both products run on MFMA 16x16x32 with the keys on the A side,
//   S^T[key][q] = K[key][:] . Q[q][:]        (A = K rows, B = Q^T)
//   O^T[d][q]  += V^T[d][key] . P^T[key][q]  (A = V^T rows, B = P^T)
// so each lane owns one query column and the online-softmax rescale is a per-lane scalar.
// Probabilities enter the second product rounded to bf16 (relative error 2^-9 per term, below
// the bf16 rounding of the output itself); steps wholly inside the unmasked prefix skip the
// mask test, and the running output is rescaled only when some row's maximum moved.
// Three kernels by shape: tree_attn_blk_kernel (trees of 17-128 rows over many pairs, in a
// work-balanced sequence order, and every tree over few pairs: one workgroup per pair, or
// per pair and key split, sharing each K/V block through LDS; splits write (O, m, l)
// partials that tree_attn_combine_kernel merges with log-sum-exp weights),
// tree_attn_wg_kernel (trees of at most 16 rows over many pairs: one workgroup per pair
// whose waves split the keys and merge in LDS), and tree_attn_f32_kernel.
#include <hip/hip_ext.h>

#include "../launch.h"

namespace adt {

ADT_DEVICE_ERROR_WORD(attn)

constexpr int ATT_KT = 64;      // keys per LDS tile
constexpr int ATT_MAX_SPLITS = 64;
// Floor of the running maximum (log2 domain) of the MFMA kernels: far below any score, so the
// weights of masked keys (-inf) come out 0 without a test, and split partials that saw no key
// carry weight 0 in the merge.
constexpr float ATT_M_FLOOR = -1e30f;

__device__ __forceinline__ bool tail_visible(uint64_t w0, uint64_t w1, int j) {
  const uint64_t w = j < 64 ? w0 : w1;
  return (w >> (j & 63)) & 1ull;
}

// Whether key `key` is visible to a row with ancestor mask (w0, w1): inside [0, k_end) and
// either in the prefix [0, L) or a marked tree row.  Written without short-circuits, so it
// compiles to selects rather than a branch per element.
__device__ __forceinline__ bool key_visible(int key, int k_end, int L, uint64_t w0, uint64_t w1) {
  const int j = key - L;
  const uint64_t w = j < 64 ? w0 : w1;
  return (key < k_end) & ((key < L) | (bool)((w >> (j & 63)) & 1ull));
}

// 2^x on the transcendental unit alone (no denormal fix-up: softmax weights that small
// are zero for every purpose here).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// The work-balanced sequence order (defined with the shared-block kernel below).
__device__ int balanced_seq(int y, int B, const int32_t* kv_len, const int32_t* n_q, const int32_t* n_tail,
                            int nq_max, int kv_cap, int* scratch);

// One workgroup per (sequence, head): its W = QG x KG waves form QG query groups of QTW
// 16-row query tiles, and each group's KG waves take contiguous, balanced slices of the
// keys (computed on the device from kv_len + n_tail, so no wave idles on an empty split).
// Each wave runs the online softmax over its slice for its query tiles, double-buffering
// 32-key K/V steps in registers; V rows go to the wave's own LDS area as they are and come
// back transposed through gfx950's LDS transpose load.  The KG waves of a group are then merged in LDS
// in wave order, so there is no second kernel and no partials in global memory.
constexpr int AWG_KT = 32;
constexpr int AWG_W = 8;

template <int DH, int QTW, int QG, int NW>
__global__ __launch_bounds__(NW * WAVE) void tree_attn_wg_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
    int64_t stride_b, int64_t stride_h, const int32_t* __restrict__ kv_len, const int32_t* __restrict__ n_q,
    const int32_t* __restrict__ n_tail, const uint64_t* __restrict__ mask, AttnRows rl, int H, int nq_max,
    int kv_cap, float scale_log2, uint16_t* __restrict__ out, int balance) {
  constexpr int KG = NW / QG;                           // key slices per query group
  constexpr int DT = DH / 16, KS = DH / 32;
  // V rows of a step, padded by 32 bytes so that the 8 rows a transpose load touches per
  // pair of 16-lane groups fall on distinct banks
  constexpr int VRW = DH + 16;
  constexpr int VG = (AWG_KT / 4) * (DH / 8) / WAVE;       // (4 keys x 8 dims) groups per lane per step
  constexpr int VT_BYTES = NW * AWG_KT * VRW * 2;
  constexpr int MG_BYTES = NW * 16 * (DH + 2) * 4;      // one query tile of (O, m, l) per wave
  __shared__ __attribute__((aligned(16))) unsigned char smem[VT_BYTES > MG_BYTES ? VT_BYTES : MG_BYTES];

  // workgroup p takes head p % H of sequence p / H, or with balance (a launch whose CUs hold
  // two workgroups each) of the sequence of rank p / H in the work-balanced order, which
  // pairs a long prefix with a short one on every CU
  const int h = blockIdx.x % H, nb = gridDim.x / H;
  const int b = balance && nb > 1 ? balanced_seq(blockIdx.x / H, nb, kv_len, n_q, n_tail, nq_max, kv_cap, (int*)smem)
                                  : blockIdx.x / H;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / WAVE);
  const int qg = wave / KG, kg = wave % KG;
  const int lane = threadIdx.x % WAVE, lq = lane & 15, g = lane >> 4;
  const int L = kv_len[b];
  const int nq = min(n_q[b], nq_max);
  const int total = min(L + n_tail[b], kv_cap);
  if (threadIdx.x == 0 && L + n_tail[b] > kv_cap) dev_fail(DEVINV_KV_RANGE);
  int per = (total + KG - 1) / KG;
  per = (per + 15) / 16 * 16;
  const int k0 = min(total, kg * per), k1 = min(total, k0 + per);

  const uint16_t* kbase = kc + b * stride_b + h * stride_h;
  const uint16_t* vbase = vc + b * stride_b + h * stride_h;
  uint16_t(*Vr)[VRW] = reinterpret_cast<uint16_t(*)[VRW]>(smem + (size_t)wave * AWG_KT * VRW * 2);

  bf16x8 qf[QTW][KS];
  uint64_t mw0[QTW], mw1[QTW];
  f32x4 o[QTW][DT];
  float m_run[QTW], l_run[QTW];
#pragma unroll
  for (int t = 0; t < QTW; ++t) {
    m_run[t] = ATT_M_FLOOR;
    l_run[t] = 0.f;
    mw0[t] = mw1[t] = 0;
#pragma unroll
    for (int d = 0; d < DT; ++d) o[t][d] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[t][kk] = bf16x8{};
    const int qr = (qg * QTW + t) * 16 + lq;
    if (qr < nq) {
      const uint16_t* qp = q + (rl.q_row(b, qr) * H + h) * DH;
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) qf[t][kk] = *reinterpret_cast<const bf16x8*>(qp + kk * 32 + g * 8);
      const uint64_t* mp = mask + rl.m_row(b, qr) * ADT_MASK_WORDS;
      mw0[t] = mp[0];
      mw1[t] = mp[1];
    }
  }

  // K fragments (A operand rows = keys) and, per lane, VG groups of 4 consecutive keys x 8
  // dims of V for one 32-key step; keys clamped to the valid range (masked out below).  Each
  // key is read once per workgroup: nontemporal loads (8 and 16 nodes of the many-pair
  // microbenchmark 0.65 -> 0.70 and 0.65 -> 0.69 of 8 TB/s)
  auto load_step = [&](int kb, bf16x8 (&kd)[2][KS], u16x8 (&vd)[VG][4]) {
    const int last = max(total - 1, 0);
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
      const int key = min(kb + sub * 16 + lq, last);
#pragma unroll
      for (int kk = 0; kk < KS; ++kk)
        kd[sub][kk] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(kbase + (int64_t)key * DH + kk * 32 + g * 8));
    }
#pragma unroll
    for (int j = 0; j < VG; ++j) {
      const int gi = lane + j * WAVE;                      // group: dims c..c+7 of keys 4*r4..4*r4+3
      const int c = (gi % (DH / 8)) * 8, r4 = gi / (DH / 8);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int key = min(kb + 4 * r4 + u, last);
        vd[j][u] = __builtin_nontemporal_load(reinterpret_cast<const u16x8*>(vbase + (int64_t)key * DH + c));
      }
    }
  };
  // One 32-key step: this step's V rows into the wave's LDS area (row-major, padded rows),
  // S^T = K Q^T, the next step's loads, the online softmax, then O^T += V^T P^T with the V^T
  // operand read back by the LDS transpose load: lane (i, g) of ds_read_b64_tr_b16 returns,
  // over slots s = 0..3, element i of the row read by lane 4s + i/4 of its 16-lane group, so
  // lane j addressing row k0 + j/4, columns d0 + 4(j%4)..+3 yields V[k0 + s][d0 + i].
  auto step = [&](int kb, const bf16x8 (&kf)[2][KS], const u16x8 (&vf)[VG][4], bool more, bf16x8 (&kn)[2][KS],
                  u16x8 (&vn)[VG][4]) {
#pragma unroll
    for (int j = 0; j < VG; ++j) {
      const int gi = lane + j * WAVE;
      const int c = (gi % (DH / 8)) * 8, r4 = gi / (DH / 8);
#pragma unroll
      for (int u = 0; u < 4; ++u) *reinterpret_cast<u16x8*>(&Vr[4 * r4 + u][c]) = vf[j][u];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    f32x4 st[QTW][2];
#pragma unroll
    for (int t = 0; t < QTW; ++t)
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        st[t][sub] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
          st[t][sub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[sub][kk], qf[t][kk], st[t][sub], 0, 0, 0);
      }
    if (more) load_step(kb + AWG_KT, kn, vn);
    // lane (lq, g) holds S for query tile t, row lq and keys kb + sub*16 + 4g + r
    const bool prefix_only = kb + AWG_KT <= min(L, k1);
#pragma unroll
    for (int t = 0; t < QTW; ++t) {
      // the maximum of the raw products (the scale is positive), then the weights
      // 2^(s * scale - m) in one FMA each; m is floored at ATT_M_FLOOR, so a masked product
      // (-inf) gives weight 0 and every difference stays finite
      float mx = -INFINITY;
      if (prefix_only) {
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
          for (int r = 0; r < 4; ++r) mx = fmaxf(mx, st[t][sub][r]);
      } else {
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = kb + sub * 16 + 4 * g + r;
            const bool vis = key_visible(key, k1, L, mw0[t], mw1[t]);
            const float v = vis ? st[t][sub][r] : -INFINITY;
            st[t][sub][r] = v;
            mx = fmaxf(mx, v);
          }
      }
      mx = xor16_max(mx);
      mx = xor32_max(mx);
      const float m_new = fmaxf(m_run[t], mx * scale_log2);
      const float alpha = fast_exp2(m_run[t] - m_new);
      float rs = 0.f;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = fast_exp2(fmaf(st[t][sub][r], scale_log2, -m_new));
          st[t][sub][r] = p;
          rs += p;
        }
      rs = xor16_add(rs);
      rs = xor32_add(rs);
      l_run[t] = l_run[t] * alpha + rs;
      m_run[t] = m_new;
      if (!__all(alpha == 1.f)) {
#pragma unroll
        for (int d = 0; d < DT; ++d) o[t][d] *= alpha;
      }
      bf16x8 p1;
#pragma unroll
      for (int r = 0; r < 8; ++r) p1[r] = (__bf16)(r < 4 ? st[t][0][r] : st[t][1][r - 4]);
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        const int col = d * 16 + 4 * (lq & 3), row = lq >> 2;
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)&Vr[4 * g + row][col]);
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)&Vr[16 + 4 * g + row][col]);
        const bf16x8 a = __builtin_bit_cast(bf16x8, v8i16{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
        o[t][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, p1, o[t][d], 0, 0, 0);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };
  bf16x8 kf[2][KS], kn[2][KS];
  u16x8 vf[VG][4], vn[VG][4];
  if (k0 < k1) load_step(k0, kf, vf);
  for (int kb = k0; kb < k1; kb += AWG_KT) {
    const bool more = kb + AWG_KT < k1;
    step(kb, kf, vf, more, kn, vn);
    if (more) {
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) kf[sub][kk] = kn[sub][kk];
#pragma unroll
      for (int j = 0; j < VG; ++j)
#pragma unroll
        for (int u = 0; u < 4; ++u) vf[j][u] = vn[j][u];
    }
  }

  // merge the KG waves of each query group, tile by tile, in wave order
  float* mo = reinterpret_cast<float*>(smem);                      // [wave][16][DH]
  float* mml = mo + NW * 16 * DH;                               // [wave][16][2]
  __syncthreads();
#pragma unroll
  for (int t = 0; t < QTW; ++t) {
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int r = 0; r < 4; ++r) mo[((size_t)wave * 16 + lq) * DH + d * 16 + 4 * g + r] = o[t][d][r];
    if (g == 0) {
      mml[((size_t)wave * 16 + lq) * 2] = m_run[t];
      mml[((size_t)wave * 16 + lq) * 2 + 1] = l_run[t];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < QG * 16 * DH; idx += NW * WAVE) {
      const int qgr = idx / (16 * DH), row = (idx / DH) % 16, d = idx % DH;
      const int qr = (qgr * QTW + t) * 16 + row;
      if (qr >= nq) continue;
      const int w0 = qgr * KG;
      float M = -INFINITY;
#pragma unroll
      for (int w = 0; w < KG; ++w) M = fmaxf(M, mml[((w0 + w) * 16 + row) * 2]);
      float ls = 0.f, acc = 0.f;
#pragma unroll
      for (int w = 0; w < KG; ++w) {
        const float mw = mml[((w0 + w) * 16 + row) * 2];
        if (mw == -INFINITY) continue;
        const float wt = exp2f(mw - M);
        ls += wt * mml[((w0 + w) * 16 + row) * 2 + 1];
        acc += wt * mo[((size_t)(w0 + w) * 16 + row) * DH + d];
      }
      out[rl.o_index(b, qr, H, DH, h, d)] = f2bf(ls > 0.f ? acc / ls : 0.f);
    }
    __syncthreads();
  }
}

// Log-sum-exp merge of the key splits: split s holds the unnormalised O and (m, l) of query
// qr (m in the log2 domain) at row base + s * nq_max + qr.  A thread merges four dims of one
// query (DH / 4 threads per query, COMB_THREADS / (DH / 4) queries per block); weights and
// sums run in split order.  Up to eight splits (every few-pair launch) are merged in one pass
// whose loads are all requested at the start, together with the live row count, which only
// decides the store (rows past it read partial rows the split kernel left alone); more splits
// take two passes of eight-at-a-time requests.
constexpr int COMB_THREADS = 256;
__global__ __launch_bounds__(COMB_THREADS) void tree_attn_combine_kernel(
    const float* __restrict__ part_o, const float* __restrict__ part_ml, const int32_t* __restrict__ n_q, AttnRows rl,
    int H, int nq_max, int splits, int DH, uint16_t* __restrict__ out) {
  const int h = blockIdx.y, b = blockIdx.z, per_q = DH / 4;
  const int qr = blockIdx.x * (COMB_THREADS / per_q) + threadIdx.x / per_q, d = (threadIdx.x % per_q) * 4;
  if (qr >= nq_max) return;
  const int nq = min(n_q[b], nq_max);
  const int64_t base = (((int64_t)b * H + h) * splits) * nq_max + qr;
  float M = -INFINITY, ls = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (splits <= 8) {
    float mv[8], lv[8];
    float4 ov[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      mv[j] = -INFINITY;
      if (j < splits) {
        const int64_t r = base + (int64_t)j * nq_max;
        mv[j] = part_ml[r * 2];
        lv[j] = part_ml[r * 2 + 1];
        ov[j] = *reinterpret_cast<const float4*>(part_o + r * DH + d);
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) M = fmaxf(M, mv[j]);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (mv[j] == -INFINITY) continue;
      const float w = exp2f(mv[j] - M);
      ls += w * lv[j];
      acc = make_float4(acc.x + w * ov[j].x, acc.y + w * ov[j].y, acc.z + w * ov[j].z, acc.w + w * ov[j].w);
    }
  } else {
    for (int s0 = 0; s0 < splits; s0 += 8) {
      float mv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) mv[j] = s0 + j < splits ? part_ml[(base + (int64_t)(s0 + j) * nq_max) * 2] : -INFINITY;
#pragma unroll
      for (int j = 0; j < 8; ++j) M = fmaxf(M, mv[j]);
    }
    for (int s0 = 0; s0 < splits; s0 += 8) {
      float mv[8], lv[8];
      float4 ov[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        mv[j] = -INFINITY;
        if (s0 + j < splits) {
          const int64_t r = base + (int64_t)(s0 + j) * nq_max;
          mv[j] = part_ml[r * 2];
          lv[j] = part_ml[r * 2 + 1];
          ov[j] = *reinterpret_cast<const float4*>(part_o + r * DH + d);
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (mv[j] == -INFINITY) continue;
        const float w = exp2f(mv[j] - M);
        ls += w * lv[j];
        acc = make_float4(acc.x + w * ov[j].x, acc.y + w * ov[j].y, acc.z + w * ov[j].z, acc.w + w * ov[j].w);
      }
    }
  }
  if (qr >= nq) return;
  const float inv = ls > 0.f ? 1.f / ls : 0.f;
  store4(out + rl.o_index(b, qr, H, DH, h, d), acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
}

// fp32 path: one block per (query, head, sequence); scores staged in LDS.
__global__ __launch_bounds__(128) void tree_attn_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ kc, const float* __restrict__ vc, int64_t stride_b,
    int64_t stride_h, const int32_t* __restrict__ kv_len, const int32_t* __restrict__ n_q,
    const int32_t* __restrict__ n_tail, const uint64_t* __restrict__ mask, AttnRows rl, int H, int nq_max,
    int kv_cap, int DH, float scale, float* __restrict__ out) {
  extern __shared__ float smem[];      // DH query values, then kv_cap scores
  __shared__ float red[16];
  const int qr = blockIdx.x, h = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  if (qr >= min(n_q[b], nq_max)) return;
  const int L = kv_len[b];
  const int total = min(L + n_tail[b], kv_cap);
  if (threadIdx.x == 0 && L + n_tail[b] > kv_cap) dev_fail(DEVINV_KV_RANGE);
  const uint64_t* mp = mask + rl.m_row(b, qr) * ADT_MASK_WORDS;
  const uint64_t w0 = mp[0], w1 = mp[1];
  float* qs = smem;
  float* sc = smem + DH;
  const float* qp = q + (rl.q_row(b, qr) * H + h) * DH;
  for (int d = tid; d < DH; d += blockDim.x) qs[d] = qp[d];
  __syncthreads();
  const float* kb = kc + b * stride_b + h * stride_h;
  const float* vb = vc + b * stride_b + h * stride_h;
  float mx = -INFINITY;
  for (int k = tid; k < total; k += blockDim.x) {
    float v = -INFINITY;
    if (k < L || tail_visible(w0, w1, k - L)) {
      float acc = 0.f;
      for (int d = 0; d < DH; ++d) acc += qs[d] * kb[(int64_t)k * DH + d];
      v = acc * scale;
    }
    sc[k] = v;
    mx = fmaxf(mx, v);
  }
  mx = wave_max(mx);
  __syncthreads();
  if (tid % WAVE == 0) red[tid / WAVE] = mx;
  __syncthreads();
  mx = -INFINITY;
  for (int i = 0; i < (int)blockDim.x / WAVE; ++i) mx = fmaxf(mx, red[i]);
  float sum = 0.f;
  for (int k = tid; k < total; k += blockDim.x) {
    const float p = sc[k] == -INFINITY ? 0.f : expf(sc[k] - mx);
    sc[k] = p;
    sum += p;
  }
  sum = block_sum(sum, red + 8);
  __syncthreads();
  for (int d = tid; d < DH; d += blockDim.x) {
    float acc = 0.f;
    for (int k = 0; k < total; ++k) acc += sc[k] * vb[(int64_t)k * DH + d];
    out[(rl.q_row(b, qr) * H + h) * DH + d] = acc / sum;
  }
}

// ----------------------------------------------------------------------------- host
// Large trees over many pairs: one workgroup of NW waves per (sequence, head).  64-key
// blocks of K and V come into LDS once per workgroup (each thread fetches its share of the
// next block into registers while the current one is computed, then stores it; double
// buffered, one barrier per block), and every wave reads them: wave w owns query tile
// w % QT and one of the KH parts of every block's keys (w / QT): KH = 1 for 5-8 tiles,
// 2 for 3-4 tiles (64-key blocks) and, with eight waves, 4 for 2 tiles (128-key blocks);
// a workgroup of NW = 4 waves takes 2 tiles with KH = 2; the parts of a tile are merged in
// LDS at the end, in part order.  K and V rows are stored with their
// 16-byte chunks XOR-swizzled by row, so the K operand reads (16 rows of one chunk column)
// and the V^T reads through the transpose load (8 rows of two chunk columns) each touch
// distinct banks.

template <int DH>
__device__ __forceinline__ int blk_swz_k(int row) { return DH == 128 ? (row & 15) : ((row >> 1) & 7); }
template <int DH>
__device__ __forceinline__ int blk_swz_v(int row) { return DH == 128 ? 2 * (row & 7) : 2 * ((row >> 1) & 3); }

// Many pairs in one launch, one key range per pair: the workgroup in grid row y takes the
// sequence of work rank rho(y) (work = live keys x query tiles; larger first, lower index on
// ties), rho = y in the first half of the rows and B - 1 - (y - half) in the second.  With
// the workgroups dealt out in order, rows y and y + half of one head are the two workgroups
// a CU holds at once in a launch that fits the chip twice, so each CU gets a long sequence
// and a short one instead of whatever the sequence order gives (uniform lengths stay as they
// were).  Every workgroup ranks the B sequences itself, in `scratch` (B + 1 ints of LDS);
// above 512 sequences the order is kept.  The rank index is made scalar, so the ranking adds
// no vector registers to the kernel that calls it.
__device__ int balanced_seq(int y, int B, const int32_t* kv_len, const int32_t* n_q, const int32_t* n_tail,
                            int nq_max, int kv_cap, int* scratch) {
  if (B > 512) return y;
  const int half = (B + 1) / 2, rho = y < half ? y : B - 1 - (y - half);
  for (int t = threadIdx.x; t < B; t += blockDim.x)
    scratch[t] = min(kv_len[t] + n_tail[t], kv_cap) * ((min(n_q[t], nq_max) + 15) / 16);
  __syncthreads();
  for (int t = threadIdx.x; t < B; t += blockDim.x) {
    const int wt = scratch[t];
    int r = 0;
    for (int u = 0; u < B; ++u) {
      const int wu = scratch[u];
      r += (wu > wt) | ((wu == wt) & (u < t));
    }
    if (r == rho) scratch[B] = t;
  }
  __syncthreads();
  const int b = __builtin_amdgcn_readfirstlane(scratch[B]);   // uniform: addresses stay scalar
  __syncthreads();
  return b;
}

template <int DH, int KH, int NW, int P>
__global__ __launch_bounds__(NW * WAVE, P > 1 ? 2 : 4) void tree_attn_blk_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc, const uint16_t* __restrict__ vc,
    int64_t stride_b, int64_t stride_h, const int32_t* __restrict__ kv_len, const int32_t* __restrict__ n_q,
    const int32_t* __restrict__ n_tail, const uint64_t* __restrict__ mask, AttnRows rl, int H, int nq_max,
    int kv_cap, float scale_log2, uint16_t* __restrict__ out, int splits, float* __restrict__ part_o,
    float* __restrict__ part_ml) {
  constexpr int BLK_KT = KH == 4 ? 128 : 64;      // keys per block: 32 per wave and half-step
  constexpr int CH = DH / 8;                     // 16-byte chunks per row
  constexpr int DT = DH / 16, KS = DH / 32;
  constexpr int BLK_BYTES = BLK_KT * DH * 2;     // one block of K or of V
  constexpr int LOADS = BLK_BYTES / (NW * WAVE * 16);   // direct loads per thread per block and operand
  constexpr int SUBS = BLK_KT / KH / 16;         // 16-key sub-blocks per wave per block
  static_assert(LOADS >= 1 && SUBS % 2 == 0, "block shape");
  static_assert((KH - 1) * (NW / KH) * (DT * 4 + 2) * WAVE * 4 <= 4 * BLK_BYTES, "merge area");
  __shared__ __attribute__((aligned(16))) unsigned char smem[4 * BLK_BYTES];   // [buffer][K, V]

  const int h = blockIdx.x, sp = blockIdx.z;
  const int b = (splits == 1 && gridDim.y > 1)
                    ? balanced_seq(blockIdx.y, gridDim.y, kv_len, n_q, n_tail, nq_max, kv_cap, (int*)smem)
                    : blockIdx.y;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / WAVE);
  const int lane = threadIdx.x % WAVE, lq = lane & 15, g = lane >> 4;
  const int QT = (nq_max + 15) / 16;
  const int tile = wave % QT, kpart = wave / QT;
  const bool active = kpart < KH;                // the remaining waves only load
  const int L = kv_len[b];
  const int nq = min(n_q[b], nq_max);
  const int total = min(L + n_tail[b], kv_cap);
  if (threadIdx.x == 0 && L + n_tail[b] > kv_cap) dev_fail(DEVINV_KV_RANGE);
  // with splits > 1, split sp takes a contiguous share of the live blocks (balanced on the
  // device, so a replayed launch follows the growing prefix)
  const int nblk_all = (total + BLK_KT - 1) / BLK_KT;
  const int per = (nblk_all + splits - 1) / splits;
  const int blk0 = min(nblk_all, sp * per), nblk = min(nblk_all, blk0 + per);
  const uint16_t* kbase = kc + b * stride_b + h * stride_h;
  const uint16_t* vbase = vc + b * stride_b + h * stride_h;

  const int qr = tile * 16 + lq;
  bf16x8 qf[KS];
  uint64_t mw0 = 0, mw1 = 0;
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) qf[kk] = bf16x8{};
  if (active && qr < nq) {
    const uint16_t* qp = q + (rl.q_row(b, qr) * H + h) * DH;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qp + kk * 32 + g * 8);
    const uint64_t* mp = mask + rl.m_row(b, qr) * ADT_MASK_WORDS;
    mw0 = mp[0];
    mw1 = mp[1];
  }

  // Slot s (16 bytes) of a block holds row s / CH, chunk (s % CH) ^ swizzle(row); thread t
  // fills slots r * 512 + t.  Keys past the live range repeat the last key (masked below).
  // P register stages: block blk + P is requested while block blk is computed.  Requests
  // are never skipped (a block past the range reads the first 16 bytes of the head instead,
  // one cache line per wave), so the count of loads in flight is the same on every path and
  // a stage waits only for its own loads.
  u16x8 kr[P][LOADS], vr[P][LOADS];
  auto fetch_block = [&](int u, int blk) {
    const int last = max(total - 1, 0);
    const bool live = blk < nblk;
#pragma unroll
    for (int r = 0; r < LOADS; ++r) {
      const int slot = r * NW * WAVE + threadIdx.x, row = slot / CH, phys = slot % CH;
      const int64_t key = min(blk * BLK_KT + row, last);
      const int64_t ko = live ? key * DH + (phys ^ blk_swz_k<DH>(row)) * 8 : 0;
      const int64_t vo = live ? key * DH + (phys ^ blk_swz_v<DH>(row)) * 8 : 0;
      // streamed once per workgroup: nontemporal (32 and 64 nodes of the many-pair
      // microbenchmark 0.64 -> 0.73 and 0.61 -> 0.68-0.70 of 8 TB/s)
      kr[u][r] = __builtin_nontemporal_load(reinterpret_cast<const u16x8*>(kbase + ko));
      vr[u][r] = __builtin_nontemporal_load(reinterpret_cast<const u16x8*>(vbase + vo));
    }
  };
  auto store_block = [&](int u, int buf) {
    unsigned char* kb = smem + buf * 2 * BLK_BYTES;
#pragma unroll
    for (int r = 0; r < LOADS; ++r) {
      const int slot = r * NW * WAVE + threadIdx.x;
      *reinterpret_cast<u16x8*>(kb + slot * 16) = kr[u][r];
      *reinterpret_cast<u16x8*>(kb + BLK_BYTES + slot * 16) = vr[u][r];
    }
  };

  f32x4 o[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) o[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = ATT_M_FLOOR, l_run = 0.f;
  // this wave's share of block blk, read from LDS buffer blk & 1
  auto compute = [&](int blk) {
    const unsigned char* kb = smem + (blk & 1) * 2 * BLK_BYTES;
    const unsigned char* vb = kb + BLK_BYTES;
    // this wave's keys of the block, 32 at a time: S^T = K Q^T (lane (lq, g) gets keys
    // key0 + sub*16 + 4g + r for query column lq), the online softmax, O^T += V^T P^T
#pragma unroll
    for (int hf = 0; hf < SUBS / 2; ++hf) {
      const int kw0 = kpart * (BLK_KT / KH) + hf * 32;   // first key within the block
      const int key0 = blk * BLK_KT + kw0;
      f32x4 st[2];
#pragma unroll
      for (int sub = 0; sub < 2; ++sub) {
        st[sub] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int row = kw0 + sub * 16 + lq;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
          const int phys = (kk * 4 + g) ^ blk_swz_k<DH>(row);
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(kb + row * DH * 2 + phys * 16);
          st[sub] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[kk], st[sub], 0, 0, 0);
        }
      }
      // the maximum of the raw products (the scale is positive), then the weights
      // 2^(s * scale - m) in one FMA each; m is floored at ATT_M_FLOOR, so a masked product
      // (-inf) gives weight 0 and every difference stays finite
      float mx = -INFINITY;
      if (key0 + 32 <= min(L, total)) {
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
          for (int r = 0; r < 4; ++r) mx = fmaxf(mx, st[sub][r]);
      } else {
#pragma unroll
        for (int sub = 0; sub < 2; ++sub)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = key0 + sub * 16 + 4 * g + r;
            const float v = key_visible(key, total, L, mw0, mw1) ? st[sub][r] : -INFINITY;
            st[sub][r] = v;
            mx = fmaxf(mx, v);
          }
      }
      mx = xor16_max(mx);
      mx = xor32_max(mx);
      const float m_new = fmaxf(m_run, mx * scale_log2);
      const float alpha = fast_exp2(m_run - m_new);
      float rs = 0.f;
#pragma unroll
      for (int sub = 0; sub < 2; ++sub)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = fast_exp2(fmaf(st[sub][r], scale_log2, -m_new));
          st[sub][r] = p;
          rs += p;
        }
      rs = xor16_add(rs);
      rs = xor32_add(rs);
      l_run = l_run * alpha + rs;
      m_run = m_new;
      if (!__all(alpha == 1.f)) {
#pragma unroll
        for (int d = 0; d < DT; ++d) o[d] *= alpha;
      }
      // the transpose load of lane j of a 16-lane group addresses row j / 4 and dims
      // 4 (j % 4)..+3 of a 4-row, 16-dim window
      bf16x8 pb;
#pragma unroll
      for (int r = 0; r < 8; ++r) pb[r] = (__bf16)(r < 4 ? st[0][r] : st[1][r - 4]);
      const int r_lo = kw0 + 4 * g + (lq >> 2), r_hi = r_lo + 16;
#pragma unroll
      for (int d = 0; d < DT; ++d) {
        const int c = 2 * d + ((lq & 3) >> 1), half = lq & 1;
        const int off_lo = r_lo * DH * 2 + ((c ^ blk_swz_v<DH>(r_lo)) * 16) + half * 8;
        const int off_hi = r_hi * DH * 2 + ((c ^ blk_swz_v<DH>(r_hi)) * 16) + half * 8;
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vb + off_lo));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(vb + off_hi));
        const bf16x8 a = __builtin_bit_cast(bf16x8, v8i16{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
        o[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb, o[d], 0, 0, 0);
      }
    }
  };
  // (the stages are issued in order: the scheduler may not interleave them, or the first
  // stage stored could be the last to arrive)
#pragma unroll
  for (int u = 0; u < P; ++u) {
    fetch_block(u, blk0 + u);
    __builtin_amdgcn_sched_barrier(0);
  }
  for (int base = blk0; base < nblk; base += P) {
#pragma unroll
    for (int u = 0; u < P; ++u) {
      const int blk = base + u;
      // the buffer written here was last read two blocks ago, before the previous barrier
      // (past the range it is written and never read)
      store_block(u, blk & 1);
      __syncthreads();
      fetch_block(u, blk + P);
      if (active && blk < nblk) compute(blk);
    }
  }

  // KH > 1: parts 1.. of a tile pass their state through LDS to part 0, which merges them
  float* mo = reinterpret_cast<float*>(smem);          // [tile][part - 1][DT * 4 + 2][WAVE]
  if (KH > 1) {
    __syncthreads();
    if (active && kpart >= 1) {
      float* t = mo + (size_t)(tile * (KH - 1) + kpart - 1) * (DT * 4 + 2) * WAVE;
#pragma unroll
      for (int d = 0; d < DT; ++d)
#pragma unroll
        for (int r = 0; r < 4; ++r) t[(d * 4 + r) * WAVE + lane] = o[d][r];
      t[(DT * 4) * WAVE + lane] = m_run;
      t[(DT * 4 + 1) * WAVE + lane] = l_run;
    }
    __syncthreads();
    if (active && kpart == 0) {
#pragma unroll
      for (int kp = 1; kp < KH; ++kp) {
        const float* t = mo + (size_t)(tile * (KH - 1) + kp - 1) * (DT * 4 + 2) * WAVE;
        const float m1 = t[(DT * 4) * WAVE + lane], l1 = t[(DT * 4 + 1) * WAVE + lane];
        const float M = fmaxf(m_run, m1);
        const float w0 = M == -INFINITY ? 0.f : fast_exp2(m_run - M);
        const float w1 = M == -INFINITY ? 0.f : fast_exp2(m1 - M);
#pragma unroll
        for (int d = 0; d < DT; ++d)
#pragma unroll
          for (int r = 0; r < 4; ++r) o[d][r] = o[d][r] * w0 + t[(d * 4 + r) * WAVE + lane] * w1;
        l_run = l_run * w0 + l1 * w1;
        m_run = M;
      }
    }
  }
  if (active && kpart == 0 && qr < nq) {
    if (splits == 1) {
      const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
#pragma unroll
      for (int d = 0; d < DT; ++d)
        store4(out + rl.o_index(b, qr, H, DH, h, d * 16 + 4 * g), o[d][0] * inv, o[d][1] * inv, o[d][2] * inv,
               o[d][3] * inv);
    } else {
      // this split's (O, m, l) for the log-sum-exp merge (m in the log2 domain)
      const int64_t pr = (((int64_t)b * H + h) * splits + sp) * nq_max + qr;
#pragma unroll
      for (int d = 0; d < DT; ++d) *reinterpret_cast<f32x4*>(part_o + pr * DH + d * 16 + 4 * g) = o[d];
      if (g == 0) {
        part_ml[pr * 2] = m_run;
        part_ml[pr * 2 + 1] = l_run;
      }
    }
  }
}

// Key splits of the shared-block kernel for few (sequence, head) pairs: about one workgroup
// per CU, and at least four 64-key blocks per split at the cache capacity.  The live blocks
// are divided among the splits on the device.  (Two blocks per split had given the shorter
// caches about one live block per split at mid-image; four: LlamaGen-XL-shaped attention
// 14.0 -> 11.8 us per layer, 7170 -> 7462 nodes/s, the 7B shapes' split counts unchanged or
// slightly lower.)
static int attn_splits(int B, int H, int kv_cap) {
  int want = (256 + B * H - 1) / (B * H);
  const int max_splits = (kv_cap + 4 * ATT_KT - 1) / (4 * ATT_KT);
  want = want > max_splits ? max_splits : want;
  want = want > ATT_MAX_SPLITS ? ATT_MAX_SPLITS : want;
  return want < 1 ? 1 : want;
}

// Many pairs with trees of 17-128 rows: the shared-block kernel (one K/V stream per pair,
// read by every query tile from LDS).
static bool attn_use_blk(int B, int H, int nq_max) { return B * H >= 128 && nq_max > 16 && nq_max <= 128; }

// Many pairs with trees of at most 16 rows: one workgroup per pair.  Few pairs (one image's
// forwards) take the shared-block kernel with the keys split across workgroups instead.
static bool attn_use_wg(int B, int H, int nq_max) { return B * H >= 128 && nq_max <= 16; }

// Upper bound over every kv_cap: the splits never exceed ceil(256 / (B*H)).
size_t tree_attn_ws_bytes(int B, int H, int Dh, int nq_max, int kv_cap, int dtype) {
  (void)kv_cap;
  if (dtype == ADT_F32) return 0;
  int max_splits = (256 + B * H - 1) / (B * H);
  if (max_splits > ATT_MAX_SPLITS) max_splits = ATT_MAX_SPLITS;
  return (size_t)B * H * max_splits * nq_max * (Dh + 2) * sizeof(float);
}

size_t tree_attn_ws_need(int B, int H, int Dh, int nq_max, int kv_cap, int dtype) {
  if (dtype == ADT_F32 || attn_use_blk(B, H, nq_max) || attn_use_wg(B, H, nq_max)) return 0;
  const int S = attn_splits(B, H, kv_cap);
  return S > 1 ? (size_t)B * H * S * nq_max * (Dh + 2) * sizeof(float) : 0;
}

static adt_status attn_bf16(const void* q, const void* k, const void* v, int64_t sb, int64_t sh, const int32_t* kv_len,
                            const int32_t* n_q, const int32_t* n_tail, const uint64_t* mask, AttnRows rl, int B, int H, int Dh,
                            int nq_max, int kv_cap, float scale, void* out, void* ws, size_t ws_bytes, hipStream_t st,
                            hipEvent_t ev0, hipEvent_t ev1) {
  const float sl2 = scale * LOG2E;
  if (attn_use_wg(B, H, nq_max)) {
    const dim3 grid(B * H);
#define ADT_ATTN_WG(DHV, QTWV, QGV, NWV, BAL)                                                                      \
  hipExtLaunchKernelGGL(tree_attn_wg_kernel<DHV, QTWV, QGV, NWV>, grid, dim3(NWV * WAVE), 0, st, ev0, ev1, 0,       \
                        (const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, sb, sh, kv_len, n_q, n_tail,   \
                        mask, rl, H, nq_max, kv_cap, sl2, (uint16_t*)out, BAL)
    // one query tile (at most 16 rows) per workgroup.  Head size 128 (160-190 VGPRs a wave):
    // four waves, so that two workgroups share a CU and every pair of a 512-pair launch is
    // resident at once, with the sequences in the work-balanced order (microbenchmark at 8 /
    // 16 nodes: 66 / 64-65 % of 8 TB/s, against 61 / 61 % for eight waves, one workgroup per
    // CU, in the plain order)
    if (Dh == 128) ADT_ATTN_WG(128, 1, 1, 4, 1);
    else ADT_ATTN_WG(64, 1, 1, AWG_W, 0);
#undef ADT_ATTN_WG
    ADT_LAUNCH_CHECK();
    return ADT_OK;
  }
  // the shared-block kernel: many pairs with 17-128 rows in one launch, few pairs with the
  // keys split across workgroups and a log-sum-exp merge
  const int S = attn_use_blk(B, H, nq_max) ? 1 : attn_splits(B, H, kv_cap);
  float *part_o = nullptr, *part_ml = nullptr;
  if (S > 1) {
    const size_t need = tree_attn_ws_need(B, H, Dh, nq_max, kv_cap, ADT_BF16);
    ADT_CHECK_ARG(ws != nullptr && ws_bytes >= need, ADT_E_CAPACITY, "tree_attn: workspace %zu < %zu bytes", ws_bytes,
                  need);
    part_o = (float*)ws;
    part_ml = part_o + (size_t)B * H * S * nq_max * Dh;
  }
  const dim3 grid(H, B, S);
  const int qt = (nq_max + 15) / 16;
  hipEvent_t e1 = S > 1 ? nullptr : ev1;
#define ADT_ATTN_BLK_P(DHV, KHV, NWV, PV)                                                                       \
  hipExtLaunchKernelGGL(tree_attn_blk_kernel<DHV, KHV, NWV, PV>, grid, dim3(NWV * WAVE), 0, st, ev0, e1, 0,        \
                        (const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, sb, sh, kv_len, n_q, n_tail,   \
                        mask, rl, H, nq_max, kv_cap, sl2, (uint16_t*)out, S, part_o, part_ml)
  // a split workgroup owns the CU and streams a few blocks, so it keeps three in flight; many
  // pairs without splits keep one (two workgroups share a CU)
#define ADT_ATTN_BLK(DHV, KHV, NWV)        \
  if (S > 1) {                             \
    ADT_ATTN_BLK_P(DHV, KHV, NWV, 3);      \
  } else {                                 \
    ADT_ATTN_BLK_P(DHV, KHV, NWV, 1);      \
  }
  // two tiles at head size 128: four waves (two tiles x two key halves, ~190 VGPRs), so two
  // workgroups share a CU and a 512-pair launch is resident at once (32 nodes: 61 % of
  // 8 TB/s against 58 % with eight waves in 128-key blocks, one workgroup per CU)
  if (Dh == 128) {
    if (qt <= 2) { ADT_ATTN_BLK(128, 2, 4) }
    else if (qt <= 4) { ADT_ATTN_BLK(128, 2, AWG_W) }
    else { ADT_ATTN_BLK(128, 1, AWG_W) }
  } else {
    if (qt <= 2) { ADT_ATTN_BLK(64, 4, AWG_W) }
    else if (qt <= 4) { ADT_ATTN_BLK(64, 2, AWG_W) }
    else { ADT_ATTN_BLK(64, 1, AWG_W) }
  }
#undef ADT_ATTN_BLK
#undef ADT_ATTN_BLK_P
  ADT_LAUNCH_CHECK();
  if (S > 1) {
    const int qpb = COMB_THREADS / (Dh / 4);
    const dim3 g2((nq_max + qpb - 1) / qpb, H, B);
    hipExtLaunchKernelGGL(tree_attn_combine_kernel, g2, dim3(COMB_THREADS), 0, st, nullptr, ev1, 0, part_o, part_ml,
                          n_q, rl, H, nq_max, S, Dh, (uint16_t*)out);
    ADT_LAUNCH_CHECK();
  }
  return ADT_OK;
}

adt_status launch_tree_attn(const void* q, const void* k, const void* v, int64_t sb, int64_t sh, const int32_t* kv_len,
                            const int32_t* n_q, const int32_t* n_tail, const uint64_t* mask, AttnRows rl, int B, int H, int Dh,
                            int nq_max, int kv_cap, float scale, int dtype, void* out, void* ws, size_t ws_bytes,
                            hipStream_t st, hipEvent_t ev0, hipEvent_t ev1) {
  ADT_CHECK_ARG(rl.o_pk == 0 || (dtype == ADT_BF16 && (H * Dh) % 32 == 0 && !rl.row_off &&
                                  (int64_t)(B - 1) * rl.rs_b + (int64_t)(nq_max - 1) * rl.rs_i < 16LL * rl.o_pk),
                ADT_E_ARG, "tree_attn: fragment-layout output of %d row blocks (bf16, rows of a multiple of 32 values)",
                rl.o_pk);
  if (dtype == ADT_F32) {
    const size_t sm = (size_t)(Dh + kv_cap) * sizeof(float);
    ADT_CHECK_ARG(sm <= 60 * 1024, ADT_E_CAPACITY, "tree_attn f32: kv_cap %d too large for LDS scores", kv_cap);
    dim3 grid(nq_max, H, B);
    hipExtLaunchKernelGGL(tree_attn_f32_kernel, grid, dim3(128), sm, st, ev0, ev1, 0, (const float*)q, (const float*)k,
                          (const float*)v, sb, sh, kv_len, n_q, n_tail, mask, rl, H, nq_max, kv_cap, Dh, scale,
                          (float*)out);
    ADT_LAUNCH_CHECK();
    return ADT_OK;
  }
  return attn_bf16(q, k, v, sb, sh, kv_len, n_q, n_tail, mask, rl, B, H, Dh, nq_max, kv_cap, scale, out, ws, ws_bytes,
                   st, ev0, ev1);
}

}  // namespace adt
