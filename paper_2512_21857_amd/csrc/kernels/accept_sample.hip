// Exact and relaxed acceptance by sampling along one verified tree (Sec. 3.1, Eq. 1).
//
// The drafted children are deterministic top-k proposals, so the proposal distribution
// of Eq. 1 is a point mass: child x is accepted with probability p(x); on rejection x is
// removed from p and the next sibling is tried; if every child is rejected the bonus
// token is drawn from the residual.  Relaxed mode (the ADT-Tree+LANTERN rows of Tables
// I-II) also credits x with the mass of its nearest codebook neighbours while that mass
// stays within delta of the remaining total, and removes the credited set on rejection.
//
// p at a row is held as integer weights w = rint(exp(z - max z) * 2^32) over the top_k
// allowed ids (z = logit / T and z - max z in fp32, exp(.) by the fixed double sequence of
// quantised_exp_weight, so the integers do not depend on a math library); every later
// operation is exact integer arithmetic, so the walk does not depend on summation order.  One workgroup per tree: the weights of
// a row are built cooperatively (64-bit radix select for the top-k threshold, block
// reductions), the sibling walk runs on one wave (the tree's parent and token arrays in
// LDS; a relaxed child's neighbour credit by a wave prefix sum; ids removed by rejections
// marked in an LDS bitmap over the row's allowed range instead of zeroing their weights),
// and the bonus is found by a block-wide prefix scan over ids in ascending order.
#include "../launch.h"

namespace adt {

constexpr int AS_THREADS = 1024;
constexpr int AS_DELTA_BITS = 16;
constexpr int AS_MAX_RANGE = 65536;   // allowed ids per row of the exact / relaxed walk (one bitmap bit each)

// 64 random bits at key = seed, counter = (step, node, index, tag): words (x1 << 32 | x0).
// tag 0: acceptance draws; tag 2: drafted children (stochastic children).
__device__ __forceinline__ uint64_t philox_u64(uint64_t seed, uint32_t step, uint32_t node, uint32_t index,
                                               uint32_t tag) {
  uint32_t c[4] = {step, node, index, tag};
  philox4x32_10(c, (uint32_t)seed, (uint32_t)(seed >> 32));
  return ((uint64_t)c[1] << 32) | c[0];
}

__device__ __forceinline__ uint64_t draw_below(uint64_t seed, uint32_t step, uint32_t node, uint32_t trial,
                                               uint64_t W) {
  return __umul64hi(philox_u64(seed, step, node, trial, 0u), W);
}

// Order-preserving 64-bit key: larger z first, then lower id first.
__device__ __forceinline__ uint64_t zkey(float z, int id) {
  uint32_t b = __float_as_uint(z);
  b = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((uint64_t)b << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)id);
}

struct SampleShared {
  uint32_t hist[256];
  uint64_t u64[AS_THREADS / WAVE];
  float f32[AS_THREADS / WAVE];
  uint64_t scan[AS_THREADS];
  uint64_t thr;
  uint64_t total;
  float zmax;
  int node, trial, accepted, done, bonus, a, need, exact;
};

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
  const uint32_t lo = __shfl_xor((uint32_t)v, o, WAVE), hi = __shfl_xor((uint32_t)(v >> 32), o, WAVE);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  const uint32_t lo = __shfl((uint32_t)v, src, WAVE), hi = __shfl((uint32_t)(v >> 32), src, WAVE);
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix sum over the lanes of a wave (lane order).
__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v) {
  const int lane = threadIdx.x % WAVE;
#pragma unroll
  for (int o = 1; o < WAVE; o <<= 1) {
    const uint32_t lo = __shfl_up((uint32_t)v, o, WAVE), hi = __shfl_up((uint32_t)(v >> 32), o, WAVE);
    if (lane >= o) v += ((uint64_t)hi << 32) | lo;
  }
  return v;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += shfl_xor_u64(v, o);
  return v;
}

__device__ uint64_t block_sum_u64(uint64_t v, SampleShared& sh) {
  for (int o = 32; o >= 1; o >>= 1) v += shfl_xor_u64(v, o);
  __syncthreads();
  if (threadIdx.x % WAVE == 0) sh.u64[threadIdx.x / WAVE] = v;
  __syncthreads();
  uint64_t s = 0;
  for (int i = 0; i < AS_THREADS / WAVE; ++i) s += sh.u64[i];
  __syncthreads();
  return s;
}

__device__ float block_max_f32(float v, SampleShared& sh) {
  v = wave_max(v);
  __syncthreads();
  if (threadIdx.x % WAVE == 0) sh.f32[threadIdx.x / WAVE] = v;
  __syncthreads();
  float m = -INFINITY;
  for (int i = 0; i < AS_THREADS / WAVE; ++i) m = fmaxf(m, sh.f32[i]);
  __syncthreads();
  return m;
}

__device__ uint64_t block_min_u64(uint64_t v, SampleShared& sh) {
  for (int o = 32; o >= 1; o >>= 1) {
    const uint64_t u = shfl_xor_u64(v, o);
    v = u < v ? u : v;
  }
  __syncthreads();
  if (threadIdx.x % WAVE == 0) sh.u64[threadIdx.x / WAVE] = v;
  __syncthreads();
  uint64_t m = ~0ull;
  for (int i = 0; i < AS_THREADS / WAVE; ++i) m = sh.u64[i] < m ? sh.u64[i] : m;
  __syncthreads();
  return m;
}

// The K-th largest 64-bit key of the row (K < count): exactly K keys are >= it.  Digits of
// 8 bits from the top; once the digit chosen holds exactly the keys still needed, the
// threshold is the smallest key of that digit's bin (one pass of a block minimum instead of
// the remaining digits: with fp32 logits the bin is usually a single key after 16-24 bits).
__device__ uint64_t radix_select(const float* x, int lo, int hi, int K, float T, SampleShared& sh) {
  uint64_t prefix = 0, mask = 0;
  int need = K;   // rank (1-based) of the threshold among keys matching the prefix
  const int lane = threadIdx.x % WAVE;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < 256; i += AS_THREADS) sh.hist[i] = 0;
    __syncthreads();
    if (shift == 56) {
      // the sign-and-exponent digit: most keys of a wave share a few bins, so the keys in the
      // bins of the wave's first two unassigned lanes are counted with one atomic per bin
      // (the same counts as one atomic per key)
      for (int i = lo + threadIdx.x; i < hi; i += AS_THREADS) {
        const uint32_t bin = (uint32_t)(zkey(x[i] / T, i) >> 56);
        bool act = true;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const uint64_t am = __ballot(act);
          if (am) {
            const int leader = __ffsll((long long)am) - 1;
            const uint32_t lb = (uint32_t)__shfl((int)bin, leader, WAVE);
            const uint64_t peers = __ballot(act && bin == lb);
            if (lane == leader) atomicAdd(&sh.hist[lb], (uint32_t)__popcll(peers));
            if (bin == lb) act = false;
          }
        }
        if (act) atomicAdd(&sh.hist[bin], 1u);
      }
    } else {
      for (int i = lo + threadIdx.x; i < hi; i += AS_THREADS) {
        const uint64_t k = zkey(x[i] / T, i);
        if ((k & mask) == prefix) atomicAdd(&sh.hist[(k >> shift) & 255], 1u);
      }
    }
    __syncthreads();
    // the highest bin b at which the count of keys in bins >= b reaches need (bin 0 if
    // none does): lane l scans bins 255 - 4l .. 252 - 4l after the prefix sums of the lanes
    // above it
    if (threadIdx.x < WAVE) {
      const int l = threadIdx.x;
      uint32_t h[4], cnt = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        h[i] = sh.hist[255 - 4 * l - i];
        cnt += h[i];
      }
      const uint64_t inc = wave_incl_scan_u64(cnt);
      uint32_t acc = (uint32_t)(inc - cnt);
      const uint32_t all = (uint32_t)shfl_u64(inc, WAVE - 1);
      int fb = -1;
      uint32_t facc = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int b = 255 - 4 * l - i;
        if (fb < 0 && b > 0 && acc + h[i] >= (uint32_t)need) {
          fb = b;
          facc = acc;
        }
        acc += h[i];
      }
      const uint64_t m = __ballot(fb >= 0);
      const int src = m ? __ffsll((long long)m) - 1 : -1;
      if (src < 0 && l == 0) {
        sh.thr = prefix;
        sh.need = need - (int)(all - sh.hist[0]);
        sh.exact = sh.need == (int)sh.hist[0];
      } else if (l == src) {
        sh.thr = prefix | ((uint64_t)fb << shift);
        sh.need = need - (int)facc;
        sh.exact = sh.need == (int)sh.hist[fb];
      }
    }
    __syncthreads();
    prefix = sh.thr;
    need = sh.need;
    mask |= (uint64_t)255 << shift;
    const bool exact = sh.exact && shift > 0;
    __syncthreads();
    if (exact) {
      // every key of the bin is among the K largest: the threshold is the bin's smallest key
      uint64_t mn = ~0ull;
      for (int i = lo + threadIdx.x; i < hi; i += AS_THREADS) {
        const uint64_t k = zkey(x[i] / T, i);
        if ((k & mask) == prefix && k < mn) mn = k;
      }
      return block_min_u64(mn, sh);
    }
  }
  return prefix;
}

// Integer weights w[i] = quantised_exp_weight(z_i - max z), z = x[i] / T, over the top_k ids of
// [lo, hi) by (z desc, id asc) (all of them when top_k is 0 or covers the range), zero
// elsewhere in [0, V) (written only with full); returns their total.  Every thread must call it.
__device__ uint64_t build_weights(const float* x, int lo, int hi, int V, float T, int top_k, uint64_t* w,
                                  SampleShared& sh, bool full = true) {
  const int tid = threadIdx.x;
  const int cnt = hi - lo;
  uint64_t thr = 0;
  if (top_k > 0 && top_k < cnt) thr = radix_select(x, lo, hi, top_k, T, sh);
  float zm = -INFINITY;
  for (int i = lo + tid; i < hi; i += AS_THREADS) {
    const float z = x[i] / T;
    if (zkey(z, i) >= thr) zm = fmaxf(zm, z);
  }
  zm = block_max_f32(zm, sh);
  uint64_t part = 0;
  // full: every id of [0, V) is written (zero outside the range); otherwise only [lo, hi),
  // and the caller treats ids outside it as weight 0
  for (int i = full ? tid : lo + tid; i < (full ? V : hi); i += AS_THREADS) {
    uint64_t wi = 0;
    if (i >= lo && i < hi) {
      const float z = x[i] / T;
      if (zkey(z, i) >= thr) wi = quantised_exp_weight(z - zm);
    }
    w[i] = wi;
    part += wi;
  }
  const uint64_t total = block_sum_u64(part, sh);
  __threadfence_block();
  __syncthreads();
  return total;
}

// The top-1 id of softmax(x / T) over [lo, hi): largest z, lowest id.  Every thread calls it.
__device__ int block_top1(const float* x, int lo, int hi, float T, SampleShared& sh) {
  const int tid = threadIdx.x;
  float bz = -INFINITY;
  int bi = 0x7FFFFFFF;
  for (int i = lo + tid; i < hi; i += AS_THREADS) {
    const float z = x[i] / T;
    if (z > bz || (z == bz && i < bi)) {
      bz = z;
      bi = i;
    }
  }
  sh.scan[tid] = ((uint64_t)__float_as_uint(bz) << 32) | (uint32_t)bi;
  __syncthreads();
  if (tid == 0) {
    float best = -INFINITY;
    int bid = lo;
    for (int t = 0; t < AS_THREADS; ++t) {
      const float z = __uint_as_float((uint32_t)(sh.scan[t] >> 32));
      const int id = (int)(uint32_t)sh.scan[t];
      if (id == 0x7FFFFFFF) continue;
      if (z > best || (z == best && id < bid)) {
        best = z;
        bid = id;
      }
    }
    sh.bonus = bid;
  }
  __syncthreads();
  const int r = sh.bonus;
  __syncthreads();
  return r;
}

// Weight of id i of a row whose range starts at lo, with the ids removed so far marked in the
// bitmap zb (bit i - lo); zb null: no removals.
__device__ __forceinline__ uint64_t kept_weight(const uint64_t* w, const uint32_t* zb, int lo, int i) {
  return (zb && ((zb[(i - lo) >> 5] >> ((i - lo) & 31)) & 1u)) ? 0ull : w[i];
}

// Per-thread chunks of [lo, hi) for inverse-CDF lookups: thread t owns ids [b0, b1) and
// sh.scan[t] = the total weight of the ids before its chunk.  Every thread calls it.
__device__ void chunk_scan(const uint64_t* w, int lo, int hi, int& b0, int& b1, uint64_t& own, SampleShared& sh,
                           const uint32_t* zb = nullptr) {
  const int tid = threadIdx.x;
  const int per = (hi - lo + AS_THREADS - 1) / AS_THREADS;
  b0 = lo + tid * per;
  b1 = min(hi, b0 + per);
  uint64_t s = 0;
  for (int i = b0; i < b1; ++i) s += kept_weight(w, zb, lo, i);
  own = s;
  // block exclusive scan of the per-thread sums: within each wave, then over the waves
  const uint64_t incl = wave_incl_scan_u64(s);
  __syncthreads();
  if (tid % WAVE == WAVE - 1) sh.u64[tid / WAVE] = incl;
  __syncthreads();
  uint64_t base = 0;
  for (int i = 0; i < tid / WAVE; ++i) base += sh.u64[i];
  sh.scan[tid] = base + incl - s;
  __syncthreads();
}

// Smallest id with prefix weight > r, if it lies in this thread's chunk (else -1).
__device__ __forceinline__ int chunk_find(const uint64_t* w, int lo, int b0, int b1, uint64_t own, uint64_t r,
                                          const SampleShared& sh, const uint32_t* zb = nullptr) {
  uint64_t run = sh.scan[threadIdx.x];
  if (b0 < b1 && run <= r && r < run + own) {
    for (int i = b0; i < b1; ++i) {
      run += kept_weight(w, zb, lo, i);
      if (run > r) return i;
    }
  }
  return -1;
}

__global__ __launch_bounds__(AS_THREADS) void accept_sample_kernel(
    const float* __restrict__ logits, int64_t ld, int V, const int32_t* __restrict__ parent,
    const int32_t* __restrict__ token, const int32_t* __restrict__ allowed, const int32_t* __restrict__ n_nodes,
    int n_max, int mode, float T, int top_k, uint32_t delta_q, int knn_k, int knn_rows, int knn_stride,
    const int32_t* __restrict__ knn, uint64_t seed, uint32_t step, uint64_t* __restrict__ w,
    int32_t* __restrict__ path, int32_t* __restrict__ n_acc, int32_t* __restrict__ bonus) {
  __shared__ SampleShared sh;
  __shared__ uint32_t zb[AS_MAX_RANGE / 32];   // ids of the current row removed by rejections (bit i: id lo + i)
  __shared__ int32_t par_s[ADT_MAX_NODES], tok_s[ADT_MAX_NODES];
  const int tid = threadIdx.x, lane = tid % WAVE;
  const int n = min(*n_nodes, n_max);
  for (int i = tid; i < n; i += AS_THREADS) {
    par_s[i] = parent[i];
    tok_s[i] = token[i];
  }
  if (tid == 0) {
    sh.node = 0;
    sh.a = 0;
    sh.done = 0;
    sh.bonus = 0;
    path[0] = 0;
  }
  __syncthreads();
  for (int guard = 0; guard < ADT_MAX_NODES; ++guard) {
    const int u = sh.node;
    const int lo = max(0, min(allowed[u * 2], V)), hi = max(lo, min(allowed[u * 2 + 1], V));
    const float* x = logits + (int64_t)u * ld;
    for (int i = tid; i < (hi - lo + 31) / 32; i += AS_THREADS) zb[i] = 0;
    const uint64_t total = build_weights(x, lo, hi, V, T, top_k, w, sh, false);
    // --- sibling walk on wave 0: the children of u in node order, one at a time (every lane
    // holds the same W, draw and mass); ids outside [lo, hi) weigh 0
    if (tid < WAVE) {
      const bool relaxed = mode == ADT_ACCEPT_RELAXED;
      auto in_range = [&](int i) { return i >= lo && i < hi; };
      auto removed = [&](int i) { return (zb[(i - lo) >> 5] >> ((i - lo) & 31)) & 1u; };
      // the next child of u at or after node `from` (n if none), by a ballot over par_s
      auto next_child = [&](int from) -> int {
        for (int b = from; b < n; b += WAVE) {
          const int i = b + lane;
          const uint64_t m = __ballot(i < n && par_s[i] == u);
          if (m) return b + __ffsll((long long)m) - 1;
        }
        return n;
      };
      // Relaxed mode: a child's inputs (its token, the token's weight, the ids and weights of
      // its first 128 neighbours) are requested one child ahead.  w does not change during the
      // walk (removals are bits of zb, tested when the values are used), so the early loads
      // read what the walk would read later.
      struct Ahead {
        int xt, y0, y1;
        uint64_t wx, w0, w1;
      };
      auto fetch = [&](int c) {
        Ahead f{0, -1, -1, 0ull, 0ull, 0ull};
        if (c >= n) return f;
        f.xt = min(max(tok_s[c], 0), V - 1);
        if (in_range(f.xt)) f.wx = w[f.xt];
        if (relaxed && f.xt < knn_rows) {
          const int32_t* nb = knn + (int64_t)f.xt * knn_stride;
          if (1 + lane < knn_k) f.y0 = nb[1 + lane];
          if (1 + WAVE + lane < knn_k) f.y1 = nb[1 + WAVE + lane];
          if (in_range(f.y0)) f.w0 = w[f.y0];
          if (in_range(f.y1)) f.w1 = w[f.y1];
        }
        return f;
      };
      uint64_t W = total;
      int trial = 0, acc = -1;
      if (!relaxed) {
        // exact: a child's one weight is requested when its turn comes, behind its draw (a
        // request one child ahead measured slower here)
        for (int c = u + 1; c < n; ++c) {
          if (par_s[c] != u) continue;
          const int xt = min(max(tok_s[c], 0), V - 1);
          const uint64_t r = draw_below(seed, step, (uint32_t)u, (uint32_t)trial, W);
          ++trial;
          const uint64_t mass = in_range(xt) && !removed(xt) ? w[xt] : 0ull;
          if (r < mass) {
            acc = c;
            break;
          }
          uint64_t gone = 0;
          if (lane == 0 && in_range(xt)) {
            const uint32_t bit = 1u << ((xt - lo) & 31);
            if (!(atomicOr(&zb[(xt - lo) >> 5], bit) & bit)) gone = w[xt];
          }
          W -= wave_sum_u64(gone);
        }
      }
      int c = relaxed ? next_child(u + 1) : n;
      Ahead cur = fetch(c);
      while (c < n) {
        const int cn = next_child(c + 1);
        const Ahead nxt = fetch(cn);
        const int xt = cur.xt;
        const uint64_t r = draw_below(seed, step, (uint32_t)u, (uint32_t)trial, W);
        ++trial;
        uint64_t mass = in_range(xt) && !removed(xt) ? cur.wx : 0ull;
        int credit_n = 0;
        const int32_t* nb = knn + (int64_t)xt * knn_stride;
        // neighbour j = base + lane of batch bi: the fetched id and weight for the first two
        // batches, a load for later ones
        auto nbr = [&](int bi, int j, int jmax, uint64_t& wr) -> int {
          int y;
          if (bi < 2) {
            y = bi == 0 ? cur.y0 : cur.y1;
            wr = bi == 0 ? cur.w0 : cur.w1;
          } else {
            y = j <= jmax ? nb[j] : -1;
            wr = in_range(y) ? w[y] : 0ull;
          }
          return j <= jmax ? y : -1;
        };
        if (relaxed && xt < knn_rows) {
          // neighbours 1.. in order while the credited sum stays <= lim: the first j whose
          // running sum passes lim ends the run (a wave prefix sum per 64 neighbours)
          const uint64_t lim = (W * (uint64_t)delta_q) >> AS_DELTA_BITS;
          uint64_t extra = 0;
          credit_n = knn_k - 1;
          for (int bi = 0, base = 1; base < knn_k; ++bi, base += WAVE) {
            const int j = base + lane;
            uint64_t wr;
            const int y = nbr(bi, j, knn_k - 1, wr);
            const uint64_t wy = in_range(y) && !removed(y) ? wr : 0ull;
            const uint64_t inc = wave_incl_scan_u64(wy);
            const uint64_t past = __ballot(j < knn_k && extra + inc > lim);
            if (past) {
              const int f = __ffsll((long long)past) - 1;
              credit_n = base - 1 + f;
              if (f > 0) extra += shfl_u64(inc, f - 1);
              break;
            }
            extra += shfl_u64(inc, WAVE - 1);
          }
          mass += extra;
        }
        if (r < mass) {
          acc = c;
          break;
        }
        // rejected: x, then its credited neighbours, leave p; an id already removed (an earlier
        // sibling's credit, a repeat in the list, x itself) subtracts nothing
        uint64_t gone = 0;
        if (lane == 0 && in_range(xt)) {
          const uint32_t bit = 1u << ((xt - lo) & 31);
          if (!(atomicOr(&zb[(xt - lo) >> 5], bit) & bit)) gone = cur.wx;
        }
        for (int bi = 0, base = 1; base <= credit_n; ++bi, base += WAVE) {
          uint64_t wr;
          const int y = nbr(bi, base + lane, credit_n, wr);
          if (in_range(y)) {
            const uint32_t bit = 1u << ((y - lo) & 31);
            if (!(atomicOr(&zb[(y - lo) >> 5], bit) & bit)) gone += wr;
          }
        }
        W -= wave_sum_u64(gone);
        c = cn;
        cur = nxt;
      }
      if (lane == 0) {
        sh.accepted = acc;
        sh.trial = trial;
        sh.total = W;
        if (acc >= 0) {
          sh.a += 1;
          path[sh.a] = acc;
          sh.node = acc;
        }
      }
    }
    __syncthreads();
    if (sh.accepted >= 0) continue;
    // --- bonus from the residual: smallest id with prefix(w) > r
    const uint64_t W = sh.total;
    if (W == 0) {
      // residual empty: the top-1 id of p (largest z, lowest id)
      const int b = block_top1(x, lo, hi, T, sh);
      if (tid == 0) sh.bonus = b;
      __syncthreads();
      break;
    }
    const uint64_t r = draw_below(seed, step, (uint32_t)u, (uint32_t)sh.trial, W);
    int b0, b1;
    uint64_t own;
    chunk_scan(w, lo, hi, b0, b1, own, sh, zb);
    const int f = chunk_find(w, lo, b0, b1, own, r, sh, zb);
    if (f >= 0) sh.bonus = f;
    __syncthreads();
    break;
  }
  if (tid == 0) {
    *n_acc = sh.a;
    *bonus = sh.bonus;
  }
}

__device__ float block_sum_f32(float v, SampleShared& sh) {
  v = wave_sum(v);
  __syncthreads();
  if (threadIdx.x % WAVE == 0) sh.f32[threadIdx.x / WAVE] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < AS_THREADS / WAVE; ++i) s += sh.f32[i];
  __syncthreads();
  return s;
}

__device__ int block_max_i32(int v, SampleShared& sh) {
  for (int o = 32; o >= 1; o >>= 1) v = max(v, __shfl_xor(v, o, WAVE));
  __syncthreads();
  if (threadIdx.x % WAVE == 0) sh.u64[threadIdx.x / WAVE] = (uint64_t)(uint32_t)v;
  __syncthreads();
  int m = 0;
  for (int i = 0; i < AS_THREADS / WAVE; ++i) m = max(m, (int)(uint32_t)sh.u64[i]);
  __syncthreads();
  return m;
}

__device__ __forceinline__ int bitlen128(unsigned __int128 v) {
  const uint64_t hi = (uint64_t)(v >> 64), lo = (uint64_t)v;
  return hi ? 128 - __clzll(hi) : (lo ? 64 - __clzll(lo) : 0);
}

// ---------------------------------------------------------------------------- stochastic children
// One workgroup per frontier row: q's integer weights (as p's above), the log-sum-exp of the
// row at T = 1 over its allowed ids (the confidences that rank the frontier), then cnt draws
// r_j = floor(U_j W / 2^64), U_j at counter (step, parent tree index, j, 2), each resolved to
// the smallest id with prefix weight > r_j.
__global__ __launch_bounds__(AS_THREADS) void row_sample_kernel(const float* __restrict__ logits, int64_t ld, int V,
                                                                const int32_t* __restrict__ allowed,
                                                                const int32_t* __restrict__ front, int cnt, float T,
                                                                int top_k, uint64_t seed, uint32_t step,
                                                                uint64_t* __restrict__ wbuf, int32_t* __restrict__ top_id,
                                                                float* __restrict__ top_val, float* __restrict__ lse,
                                                                int kmax) {
  __shared__ SampleShared sh;
  const int r = blockIdx.x, tid = threadIdx.x;
  const float* x = logits + (int64_t)r * ld;
  uint64_t* w = wbuf + (int64_t)r * V;
  const int lo = max(0, min(allowed[2 * r], V)), hi = max(lo, min(allowed[2 * r + 1], V));
  const uint64_t W = build_weights(x, lo, hi, V, T, top_k, w, sh);
  float m1 = -INFINITY;
  for (int i = lo + tid; i < hi; i += AS_THREADS) m1 = fmaxf(m1, x[i]);
  m1 = block_max_f32(m1, sh);
  float e1 = 0.f;
  for (int i = lo + tid; i < hi; i += AS_THREADS) e1 += expf(x[i] - m1);
  e1 = block_sum_f32(e1, sh);
  int b0, b1;
  uint64_t own;
  chunk_scan(w, lo, hi, b0, b1, own, sh);
  const uint32_t node = front ? (uint32_t)(front[r] + 1) : 0u;
  for (int j = 0; j < cnt; ++j) {
    const uint64_t rj = __umul64hi(philox_u64(seed, step, node, (uint32_t)j, 2u), W);
    const int id = chunk_find(w, lo, b0, b1, own, rj, sh);
    if (id >= 0) {
      top_id[r * kmax + j] = id;
      top_val[r * kmax + j] = x[id];
    }
  }
  if (tid == 0) lse[r] = m1 + logf(e1);
}

adt_status launch_row_sample(const float* logits, int64_t ld, int V, const int32_t* allowed, int rows,
                             const int32_t* front, int cnt, float T, int top_k, uint64_t seed, uint32_t step,
                             uint64_t* w, int32_t* top_id, float* top_val, float* lse, int kmax, hipStream_t st) {
  ADT_CHECK_ARG(rows >= 1 && cnt >= 1 && cnt <= kmax, ADT_E_ARG, "row_sample: rows %d cnt %d", rows, cnt);
  row_sample_kernel<<<rows, AS_THREADS, 0, st>>>(logits, ld, V, allowed, front, cnt, T, top_k, seed, step, w, top_id,
                                                 top_val, lse, kmax);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

// ---------------------------------------------------------------------------- literal Eq. 1
// Multi-step acceptance for children drawn i.i.d. from q: at node u the children are tried in
// node order; child x is accepted iff u32 * q_w(x) * W_p < 2^32 * p_w(x) * W_q (u32 = the high
// half of the draw at counter (step, u, trial, 0)), i.e. with probability min(1, p(x) / q(x));
// after a rejection p_w(y) <- max(0, p_w(y) W_q - q_w(y) W_p) >> s, s the least shift leaving
// every weight below 2^32 (products in 128 bits); with all rejected the bonus is drawn from
// the residual, at a leaf from p.  q_w: the weights of draft-logit row q_row[u].
__global__ __launch_bounds__(AS_THREADS) void accept_mss_kernel(
    const float* __restrict__ logits, int64_t ld, int V, const int32_t* __restrict__ parent,
    const int32_t* __restrict__ token, const int32_t* __restrict__ allowed, const int32_t* __restrict__ n_nodes,
    int n_max, float T, int top_k, const float* __restrict__ q_logits, int64_t q_ld, const int32_t* __restrict__ q_row,
    int q_rows, uint64_t seed, uint32_t step, uint64_t* __restrict__ w, uint64_t* __restrict__ wq, int32_t* __restrict__ path,
    int32_t* __restrict__ n_acc, int32_t* __restrict__ bonus) {
  __shared__ SampleShared sh;
  const int tid = threadIdx.x;
  const int n = min(*n_nodes, n_max);
  if (tid == 0) {
    sh.node = 0;
    sh.a = 0;
    sh.bonus = 0;
    path[0] = 0;
  }
  __syncthreads();
  for (int guard = 0; guard < ADT_MAX_NODES; ++guard) {
    const int u = sh.node;
    const int lo = max(0, min(allowed[u * 2], V)), hi = max(lo, min(allowed[u * 2 + 1], V));
    const float* x = logits + (int64_t)u * ld;
    uint64_t Wp = build_weights(x, lo, hi, V, T, top_k, w, sh);
    int first = -1;
    for (int c = u + 1; c < n; ++c)
      if (parent[c] == u) {
        first = c;
        break;
      }
    const int qr = first >= 0 ? q_row[u] : -1;
    int trial = 0, accepted = -1;
    bool empty = false;
    if (qr >= 0 && qr < q_rows) {   // a node without a valid q row ends the walk (bonus from p)
      const uint64_t Wq = build_weights(q_logits + (int64_t)qr * q_ld, lo, hi, V, T, top_k, wq, sh);
      for (int c = first; c < n; ++c) {
        if (parent[c] != u) continue;
        const int xt = min(max(token[c], 0), V - 1);
        if (tid == 0) {
          const uint32_t u32 = (uint32_t)(philox_u64(seed, step, (uint32_t)u, (uint32_t)trial, 0u) >> 32);
          const unsigned __int128 lhs = (unsigned __int128)((uint64_t)u32 * wq[xt]) * Wp;
          const unsigned __int128 rhs = ((unsigned __int128)w[xt] * Wq) << 32;
          sh.accepted = lhs < rhs ? 1 : 0;
        }
        __syncthreads();
        ++trial;
        const int acc = sh.accepted;
        __syncthreads();
        if (acc) {
          accepted = c;
          break;
        }
        int bl = 0;
        for (int y = lo + tid; y < hi; y += AS_THREADS) {
          const unsigned __int128 a = (unsigned __int128)w[y] * Wq, b = (unsigned __int128)wq[y] * Wp;
          if (a > b) bl = max(bl, bitlen128(a - b));
        }
        bl = block_max_i32(bl, sh);
        const int shift = max(0, bl - 32);
        uint64_t part = 0;
        for (int y = lo + tid; y < hi; y += AS_THREADS) {
          const unsigned __int128 a = (unsigned __int128)w[y] * Wq, b = (unsigned __int128)wq[y] * Wp;
          const uint64_t v = a > b ? (uint64_t)((a - b) >> shift) : 0;
          w[y] = v;
          part += v;
        }
        Wp = block_sum_u64(part, sh);
        __threadfence_block();
        __syncthreads();
        if (Wp == 0) {   // p == q on the support: a rejection has probability zero; kept for safety
          empty = true;
          break;
        }
      }
    }
    if (accepted >= 0) {
      if (tid == 0) {
        sh.a += 1;
        path[sh.a] = accepted;
        sh.node = accepted;
      }
      __syncthreads();
      continue;
    }
    if (empty) {
      const int b = block_top1(x, lo, hi, T, sh);
      if (tid == 0) sh.bonus = b;
      __syncthreads();
      break;
    }
    const uint64_t r = draw_below(seed, step, (uint32_t)u, (uint32_t)trial, Wp);
    int b0, b1;
    uint64_t own;
    chunk_scan(w, lo, hi, b0, b1, own, sh);
    const int f = chunk_find(w, lo, b0, b1, own, r, sh);
    if (f >= 0) sh.bonus = f;
    __syncthreads();
    break;
  }
  if (tid == 0) {
    *n_acc = sh.a;
    *bonus = sh.bonus;
  }
}

size_t accept_ws_bytes(int V) { return (size_t)V * 16 + 4096; }

adt_status launch_accept_mss(const float* logits, int64_t ld, int V, const int32_t* parent, const int32_t* token,
                             const int32_t* allowed, const int32_t* n_nodes, int n_max, const adt_accept_cfg& cfg,
                             uint64_t step, int32_t* path, int32_t* n_acc, int32_t* bonus, void* ws, size_t ws_bytes,
                             hipStream_t st) {
  ADT_CHECK_ARG(ws_bytes >= (size_t)V * 16, ADT_E_CAPACITY, "accept_mss: workspace");
  ADT_CHECK_ARG(cfg.q_logits && cfg.q_row && cfg.q_ld >= V && cfg.q_rows >= 1, ADT_E_ARG, "accept_mss: q rows");
  uint64_t* w = (uint64_t*)ws;
  accept_mss_kernel<<<1, AS_THREADS, 0, st>>>(logits, ld, V, parent, token, allowed, n_nodes, n_max, cfg.temperature,
                                              cfg.top_k, cfg.q_logits, cfg.q_ld, cfg.q_row, cfg.q_rows, cfg.seed,
                                              (uint32_t)step,
                                              w, w + V, path, n_acc, bonus);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_accept_sample(const float* logits, int64_t ld, int V, const int32_t* parent, const int32_t* token,
                                const int32_t* allowed, const int32_t* n_nodes, int n_max, const adt_accept_cfg& cfg,
                                uint64_t step, int32_t* path, int32_t* n_acc, int32_t* bonus, void* ws, size_t ws_bytes,
                                hipStream_t st) {
  ADT_CHECK_ARG(ws_bytes >= (size_t)V * 8, ADT_E_CAPACITY, "accept_sample: workspace");
  ADT_CHECK_ARG(V <= AS_MAX_RANGE, ADT_E_UNSUPPORTED, "accept_sample: vocabulary %d above %d", V, AS_MAX_RANGE);
  const uint32_t dq = (uint32_t)lrintf(cfg.delta * (float)(1 << AS_DELTA_BITS));
  const int relaxed = cfg.mode == ADT_ACCEPT_RELAXED;
  accept_sample_kernel<<<1, AS_THREADS, 0, st>>>(logits, ld, V, parent, token, allowed, n_nodes, n_max, cfg.mode,
                                                 cfg.temperature, cfg.top_k, dq, relaxed ? cfg.knn_k : 1,
                                                 relaxed ? cfg.knn_rows : 0, cfg.knn_stride, cfg.knn, cfg.seed,
                                                 (uint32_t)step, (uint64_t*)ws, path, n_acc, bonus);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

}  // namespace adt
