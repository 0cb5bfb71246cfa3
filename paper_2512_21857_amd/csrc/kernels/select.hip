// Draft-tree expansion and greedy acceptance (Sec. 3.1; Sec. 4.2, Eq. 3-5).
//
// row_topk: per logits row, over its allowed id range, the top-k ids ordered by
//   (logit desc, id asc) and the log-sum-exp; one workgroup per row.  Each thread keeps a
//   sorted private list over a strided slice, then k rounds of a block-wide argmax merge.
// expand_level: children of the frontier rows (score = parent score + logit - lse, i.e. the
//   log of the product of confidences of Eq. 3), appended to the candidate pool, and the
//   next frontier (top-k of the new layer by (score desc, creation asc)); it also lays out
//   the next draft forward: tokens, parent-feature rows, positions, draft-cache tail masks.
// expand_finalize: top-N rerank of the pool by (score desc, depth asc, creation asc), BFS
//   order by (depth asc, score desc, creation asc), parent indices, masks, positions.
// accept_greedy: the accepted root path along target argmaxes, as a wave-level pass over the
//   parent array (matches, pointer doubling, ballot).
#include "../launch.h"

namespace adt {

constexpr int SEL_THREADS = 256;

__device__ __forceinline__ bool better(float a, int ia, float b, int ib) { return a > b || (a == b && ia < ib); }

constexpr int TOPK_THREADS = 1024;
constexpr int TOPK_WAVES = TOPK_THREADS / WAVE;

// Wave-wide argmax of (value desc, id asc) with the owning lane.
__device__ __forceinline__ void wave_best(float& v, int& id, int& lane) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float ov = __shfl_xor(v, o, WAVE);
    const int oi = __shfl_xor(id, o, WAVE), ol = __shfl_xor(lane, o, WAVE);
    if (better(ov, oi, v, id)) {
      v = ov;
      id = oi;
      lane = ol;
    }
  }
}

// Per row: top-k ids by (logit desc, id asc) over [lo, hi) and the log-sum-exp.  The
// thread's slice of the row (float4 j*4*T + 4*tid + {0..3}) is loaded into registers in one
// go, so the loads overlap; then each wave takes k rounds of "best remaining element of
// each lane" + shuffle argmax, and wave 0 merges the per-wave lists the same way.
template <int KMAX, int E4>
__global__ __launch_bounds__(TOPK_THREADS) void row_topk_kernel(const float* __restrict__ logits, int64_t ld, int V,
                                                                const int32_t* __restrict__ allowed, int k,
                                                                int32_t* __restrict__ top_id,
                                                                float* __restrict__ top_val, float* __restrict__ lse) {
  __shared__ float wv[TOPK_WAVES][KMAX];
  __shared__ int wi[TOPK_WAVES][KMAX];
  __shared__ float smx[TOPK_WAVES], ssum[TOPK_WAVES];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid % WAVE, wave = tid / WAVE;
  const int lo = max(0, min(allowed[row * 2], V)), hi = max(lo, min(allowed[row * 2 + 1], V));
  const float* x = logits + (int64_t)row * ld;
  const bool vec = ((ld & 3) == 0);
  float r[E4 * 4];
#pragma unroll
  for (int j = 0; j < E4; ++j) {
    const int base = j * 4 * TOPK_THREADS + 4 * tid;
    if (vec && base + 3 < V) {
      const float4 q = *reinterpret_cast<const float4*>(x + base);
      r[4 * j] = q.x;
      r[4 * j + 1] = q.y;
      r[4 * j + 2] = q.z;
      r[4 * j + 3] = q.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) r[4 * j + e] = (base + e < V) ? x[base + e] : -INFINITY;
    }
  }
  // mask to the allowed range
#pragma unroll
  for (int j = 0; j < E4; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = j * 4 * TOPK_THREADS + 4 * tid + e;
      if (i < lo || i >= hi) r[4 * j + e] = -INFINITY;
    }
  // log-sum-exp
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < E4 * 4; ++j) m = fmaxf(m, r[j]);
  const float M = wave_max(m);
  float sacc = 0.f;
  if (M != -INFINITY) {
#pragma unroll
    for (int j = 0; j < E4 * 4; ++j) sacc += (r[j] == -INFINITY) ? 0.f : expf(r[j] - M);
  }
  const float S = wave_sum(sacc);
  if (lane == 0) {
    smx[wave] = M;
    ssum[wave] = S;
  }
  const int kk = min(k, hi - lo);
  // wave-level selection
  for (int q = 0; q < kk; ++q) {
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int j = 0; j < E4 * 4; ++j) {
      const int i = (j / 4) * 4 * TOPK_THREADS + 4 * tid + (j % 4);
      if (better(r[j], i, bv, bi)) {
        bv = r[j];
        bi = i;
      }
    }
    if (bv == -INFINITY) bi = 0x7FFFFFFF;
    int bl = lane;
    float wvv = bv;
    int wii = bi;
    wave_best(wvv, wii, bl);
    if (lane == bl && wii != 0x7FFFFFFF) {
#pragma unroll
      for (int j = 0; j < E4 * 4; ++j) {
        const int i = (j / 4) * 4 * TOPK_THREADS + 4 * tid + (j % 4);
        if (i == wii) r[j] = -INFINITY;
      }
    }
    if (lane == 0) {
      wv[wave][q] = wvv;
      wi[wave][q] = wii;
    }
  }
  __syncthreads();
  if (wave != 0) return;
  if (lane == 0) {
    float gm = -INFINITY;
    for (int w = 0; w < TOPK_WAVES; ++w) gm = fmaxf(gm, smx[w]);
    float gs = 0.f;
    for (int w = 0; w < TOPK_WAVES; ++w)
      if (smx[w] != -INFINITY) gs += ssum[w] * expf(smx[w] - gm);
    lse[row] = gm + logf(gs);
  }
  int h2 = 0;
  for (int q = 0; q < kk; ++q) {
    float hv = -INFINITY;
    int hid = 0x7FFFFFFF;
    if (lane < TOPK_WAVES && h2 < kk) {
      hv = wv[lane][h2];
      hid = wi[lane][h2];
    }
    int bl = lane;
    wave_best(hv, hid, bl);
    if (lane == bl) ++h2;
    if (lane == 0) {
      top_id[row * KMAX + q] = hid;
      top_val[row * KMAX + q] = hv;
    }
  }
}

// Pool (see launch.h): device arrays of capacity C: token, score, depth, parent (pool index,
// -1 = root), drow (draft tree row of an expanded node, -1 otherwise); draft tree row j has a
// tail mask rmask[j][2] over draft tree rows.  Parent-feature sources of the next draft
// forward use the draft_input encoding: row r of the draft-feature buffer is fsrc = -2 - r.

// Order keys of the selections (smaller = better).  Scores are compared as written by
// fp32 arithmetic; a NaN score counts as -inf, so every key set is totally ordered and a
// selection of N takes exactly N nodes.
__device__ __forceinline__ uint32_t score_desc_bits(float sc) {
  const float v = (sc != sc) ? -INFINITY : sc + 0.f;                 // NaN -> -inf, -0 -> +0
  const uint32_t u = __float_as_uint(v);
  const uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);   // ascending with the value
  return ~asc;                                                       // descending
}
// rerank: (score desc, depth asc, creation asc)
__device__ __forceinline__ uint64_t rank_key(float sc, int depth, int idx) {
  return ((uint64_t)score_desc_bits(sc) << 32) | ((uint64_t)(depth & 0xFFF) << 20) | (uint32_t)(idx & 0xFFFFF);
}
// BFS order: (depth asc, score desc, creation asc)
__device__ __forceinline__ uint64_t bfs_key(float sc, int depth, int idx) {
  return ((uint64_t)(depth & 0xFFF) << 52) | ((uint64_t)score_desc_bits(sc) << 20) | (uint32_t)(idx & 0xFFFFF);
}

constexpr int LVL_MAX = ADT_MAX_WIDTH * ADT_MAX_WIDTH;   // candidates of one layer

// One block.  Frontier rows r < nf (pool indices front[r], or the root when front == null)
// with top_id/top_val/lse rows; creates cnt children each at pool indices base + r*cnt + c.
// The next frontier is the k_hat best of them by (score desc, creation asc), ranked by
// comparing each candidate's key against every other key in LDS.
__global__ __launch_bounds__(SEL_THREADS) void expand_level_kernel(
    Pool pool, const int32_t* __restrict__ front, int nf, int cnt, int base, int depth, int k_hat,
    const int32_t* __restrict__ top_id, const float* __restrict__ top_val, const float* __restrict__ lse, int kmax,
    int make_next, int L, int drow_base, int root_frow, int tree_frow0, int qrow_base, NextRows nx) {
  __shared__ uint64_t key[LVL_MAX];
  const int C = nf * cnt;
  const int tid = threadIdx.x;
  for (int i = tid; i < C; i += SEL_THREADS) {
    const int r = i / cnt, c = i % cnt;
    const int par = front ? front[r] : -1;
    const float ps = par >= 0 ? pool.score[par] : 0.f;
    const int idx = base + i;
    const float sc = ps + (top_val[r * kmax + c] - lse[r]);
    pool.token[idx] = top_id[r * kmax + c];
    pool.score[idx] = sc;
    pool.depth[idx] = depth;
    pool.parent[idx] = par;
    pool.drow[idx] = -1;
    pool.qrow[idx] = -1;
    key[i] = ((uint64_t)score_desc_bits(sc) << 32) | (uint32_t)idx;
  }
  __syncthreads();
  if (!make_next) return;
  for (int i = tid; i < C; i += SEL_THREADS) {
    const uint64_t ki = key[i];
    int rank = 0;
    for (int j = 0; j < C; ++j) rank += key[j] < ki ? 1 : 0;
    if (rank < k_hat) {
      const int ci = base + i;
      const int par = pool.parent[ci];
      const int jrow = drow_base + rank;
      pool.drow[ci] = jrow;
      pool.qrow[ci] = qrow_base + rank;
      nx.frontier[rank] = ci;
      nx.tok[rank] = pool.token[ci];
      nx.pos[rank] = L + depth;
      uint64_t w0 = 0, w1 = 0;
      if (par >= 0) {
        const int pr = pool.drow[par];
        nx.fsrc[rank] = -2 - (tree_frow0 + pr);
        w0 = pool.rmask[pr * 2];
        w1 = pool.rmask[pr * 2 + 1];
      } else {
        nx.fsrc[rank] = -2 - root_frow;
      }
      if (jrow < 64) w0 |= 1ull << jrow;
      else w1 |= 1ull << (jrow - 64);
      pool.rmask[jrow * 2] = w0;
      pool.rmask[jrow * 2 + 1] = w1;
      nx.mask[rank * 2] = w0;
      nx.mask[rank * 2 + 1] = w1;
    }
  }
}

// One block of FIN_THREADS: rerank + BFS + tree arrays.  allowed_img [n_image][2]; row i's
// successor sits at absolute position L + depth + 1, image cell L + depth + 1 - P.
// Rank keys of the whole pool sit in LDS; each candidate's rank is the number of smaller
// keys (one broadcast LDS read per compared key), the N best keep their rank as the slot of
// the selection, the selection is BFS-ordered the same way, parents are mapped through the
// pool-to-BFS table in LDS, and the ancestor masks are built by pointer doubling over the
// parent array (seven rounds cover 128 levels).  keep_all: every pool node, in creation
// order (already BFS).
constexpr int FIN_THREADS = 1024;

__global__ __launch_bounds__(FIN_THREADS) void expand_finalize_kernel(
    Pool pool, int C, int n_budget, int root_token, int L, int P, int n_image, const int32_t* __restrict__ allowed_img,
    int32_t* __restrict__ parent, int32_t* __restrict__ token, int32_t* __restrict__ depth, float* __restrict__ score,
    int32_t* __restrict__ pos, uint64_t* __restrict__ mask, int32_t* __restrict__ allowed_rows,
    int32_t* __restrict__ qrow, int32_t* __restrict__ n_out, int keep_all) {
  extern __shared__ uint64_t fin_smem[];
  uint64_t* key = fin_smem;                                          // [C]
  int32_t* bfs_of = reinterpret_cast<int32_t*>(key + C);             // [C]
  __shared__ int32_t sel[ADT_MAX_NODES];                             // pool index of the r-th best
  __shared__ uint64_t bk[ADT_MAX_NODES];
  __shared__ int32_t par_pool[ADT_MAX_NODES], par[ADT_MAX_NODES], jmp[ADT_MAX_NODES];
  __shared__ uint64_t mw[ADT_MAX_NODES][2];
  const int tid = threadIdx.x;
  const int N = keep_all ? C : min(n_budget, C);
  for (int i = tid; i < C; i += FIN_THREADS) {
    key[i] = rank_key(pool.score[i], pool.depth[i], i);
    bfs_of[i] = -1;
  }
  __syncthreads();
  if (keep_all) {
    for (int r = tid; r < N; r += FIN_THREADS) sel[r] = r;
  } else {
    for (int i = tid; i < C; i += FIN_THREADS) {
      const uint64_t ki = key[i];
      int rank = 0;
      for (int j = 0; j < C; ++j) rank += key[j] < ki ? 1 : 0;
      if (rank < N) sel[rank] = i;
    }
  }
  __syncthreads();
  for (int r = tid; r < N; r += FIN_THREADS) {
    const int i = sel[r];
    bk[r] = keep_all ? (uint64_t)i : bfs_key(pool.score[i], pool.depth[i], i);
  }
  __syncthreads();
  for (int r = tid; r < N; r += FIN_THREADS) {
    const uint64_t kr = bk[r];
    int b = 1;
    for (int t = 0; t < N; ++t) b += bk[t] < kr ? 1 : 0;
    const int i = sel[r];
    bfs_of[i] = b;
    token[b] = pool.token[i];
    depth[b] = pool.depth[i];
    score[b] = pool.score[i];
    qrow[b] = pool.qrow[i];
    par_pool[b] = pool.parent[i];
  }
  __syncthreads();
  // parents in BFS indices; a selection is closed under ancestors (a child's score never
  // exceeds its parent's, ties go to the shallower node), and an index outside it is clamped
  // to the root rather than read out of range
  for (int b = tid; b <= N; b += FIN_THREADS) {
    int pb = -1;
    if (b > 0) {
      const int pp = par_pool[b];
      pb = (pp < 0 || pp >= C) ? 0 : bfs_of[pp];
      pb = (pb < 0 || pb >= b) ? 0 : pb;
      parent[b] = pb;
    }
    par[b] = pb;
    jmp[b] = pb;
    mw[b][0] = b < 64 ? 1ull << b : 0ull;
    mw[b][1] = b < 64 ? 0ull : 1ull << (b - 64);
  }
  if (tid == 0) {
    parent[0] = -1;
    token[0] = root_token;
    depth[0] = 0;
    score[0] = 0.f;
    qrow[0] = 0;   // the root's children come from draft-logit row 0
    *n_out = N + 1;
  }
  __syncthreads();
  // mw[b] = OR of the bits from b up to (not including) jmp[b]; doubling jmp each round
  for (int round = 0; round < 7; ++round) {
    uint64_t n0 = 0, n1 = 0;
    int nj = -1;
    if (tid <= N) {
      const int a = jmp[tid];
      n0 = mw[tid][0];
      n1 = mw[tid][1];
      if (a >= 0) {
        n0 |= mw[a][0];
        n1 |= mw[a][1];
        nj = jmp[a];
      }
    }
    __syncthreads();
    if (tid <= N) {
      mw[tid][0] = n0;
      mw[tid][1] = n1;
      jmp[tid] = nj;
    }
    __syncthreads();
  }
  for (int i = tid; i <= N; i += FIN_THREADS) {
    mask[i * 2] = mw[i][0];
    mask[i * 2 + 1] = mw[i][1];
    const int dp = (i == 0) ? 0 : depth[i];
    pos[i] = L + dp;
    int cell = L + dp + 1 - P;
    cell = cell < 0 ? 0 : (cell >= n_image ? n_image - 1 : cell);
    allowed_rows[i * 2] = allowed_img[cell * 2];
    allowed_rows[i * 2 + 1] = allowed_img[cell * 2 + 1];
  }
}

// Greedy acceptance (one wave; lane l holds nodes l and l + 64): node i matches when its
// token is the argmax of its parent's row and it is the first such child of that parent (the
// walk takes the lowest index among equal siblings).  A node is accepted when it and all its
// ancestors match: ok[i] &= ok[jmp[i]], jmp[i] = jmp[jmp[i]], seven doubling rounds over the
// parent array.  The accepted nodes form one root path in BFS order; a ballot numbers them,
// and the bonus is the argmax of the deepest one.
__global__ __launch_bounds__(WAVE) void accept_greedy_kernel(const int32_t* __restrict__ argmax, int kmax,
                                                             const int32_t* __restrict__ parent,
                                                             const int32_t* __restrict__ token,
                                                             const int32_t* __restrict__ n_nodes, int n_max,
                                                             int32_t* __restrict__ path, int32_t* __restrict__ n_acc,
                                                             int32_t* __restrict__ bonus) {
  __shared__ int32_t jmp[ADT_MAX_NODES], ok[ADT_MAX_NODES], first[ADT_MAX_NODES];
  const int lane = threadIdx.x;
  const int n = min(min(*n_nodes, n_max), ADT_MAX_NODES);
  bool match[2] = {false, false};
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int i = lane + h * WAVE;
    first[i] = ADT_MAX_NODES;
    if (i < n && i > 0) {
      const int p = parent[i];
      match[h] = p >= 0 && p < i && token[i] == argmax[p * kmax];
      jmp[i] = (p >= 0 && p < i) ? p : -1;
    } else {
      jmp[i] = -1;
    }
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < 2; ++h)
    if (match[h]) atomicMin(&first[jmp[lane + h * WAVE]], lane + h * WAVE);
  __syncthreads();
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int i = lane + h * WAVE;
    ok[i] = (i == 0 && n > 0) ? 1 : ((match[h] && first[jmp[i]] == i) ? 1 : 0);
  }
  __syncthreads();
  for (int round = 0; round < 7; ++round) {
    int nok[2], nj[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int i = lane + h * WAVE, a = jmp[i];
      nok[h] = ok[i] & (a >= 0 ? ok[a] : 1);
      nj[h] = a >= 0 ? jmp[a] : -1;
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      ok[lane + h * WAVE] = nok[h];
      jmp[lane + h * WAVE] = nj[h];
    }
    __syncthreads();
  }
  const uint64_t b0 = __ballot(lane > 0 && lane < n && ok[lane]);
  const uint64_t b1 = __ballot(lane + WAVE < n && ok[lane + WAVE]);
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (WAVE - lane));
  const int c0 = __popcll(b0);
  if (lane > 0 && ((b0 >> lane) & 1ull)) path[1 + __popcll(b0 & below)] = lane;
  if ((b1 >> lane) & 1ull) path[1 + c0 + __popcll(b1 & below)] = lane + WAVE;
  if (lane == 0) {
    const int a = c0 + __popcll(b1);
    const int deepest = b1 ? WAVE + 63 - __clzll(b1) : (b0 ? 63 - __clzll(b0) : 0);
    path[0] = 0;
    *n_acc = a;
    *bonus = argmax[deepest * kmax];
  }
}

// ----------------------------------------------------------------------------- host
adt_status launch_row_topk(const float* logits, int64_t ld, int V, const int32_t* allowed, int rows, int k, int kmax,
                           int32_t* top_id, float* top_val, float* lse, hipStream_t st) {
  ADT_CHECK_ARG(k >= 1 && k <= kmax && (kmax == 1 || kmax == 16), ADT_E_UNSUPPORTED, "row_topk: k=%d kmax=%d", k, kmax);
  const int e4 = (V + 4 * TOPK_THREADS - 1) / (4 * TOPK_THREADS);
  ADT_CHECK_ARG(e4 <= 16, ADT_E_UNSUPPORTED, "row_topk: vocab %d above 65536", V);
#define ADT_TOPK(KM, E)                                                                                        \
  row_topk_kernel<KM, E><<<rows, TOPK_THREADS, 0, st>>>(logits, ld, V, allowed, k, top_id, top_val, lse)
#define ADT_TOPK_E(KM)            \
  if (e4 <= 1) ADT_TOPK(KM, 1);   \
  else if (e4 <= 2) ADT_TOPK(KM, 2); \
  else if (e4 <= 4) ADT_TOPK(KM, 4); \
  else if (e4 <= 8) ADT_TOPK(KM, 8); \
  else ADT_TOPK(KM, 16)
  if (kmax == 1) {
    ADT_TOPK_E(1);
  } else {
    ADT_TOPK_E(16);
  }
#undef ADT_TOPK_E
#undef ADT_TOPK
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_expand_level(const Pool& pool, const int32_t* front, int nf, int cnt, int base, int depth, int k_hat,
                               const int32_t* top_id, const float* top_val, const float* lse, int kmax, int make_next,
                               int L, int drow_base, int root_frow, int tree_frow0, int qrow_base, const NextRows& nx,
                               hipStream_t st) {
  ADT_CHECK_ARG(nf >= 1 && cnt >= 0 && nf * cnt <= LVL_MAX, ADT_E_CAPACITY, "expand_level: %d x %d candidates", nf, cnt);
  expand_level_kernel<<<1, SEL_THREADS, 0, st>>>(pool, front, nf, cnt, base, depth, k_hat, top_id, top_val, lse, kmax,
                                                 make_next, L, drow_base, root_frow, tree_frow0, qrow_base, nx);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_expand_finalize(const Pool& pool, int C, int n_budget, int root_token, int L, int P, int n_image,
                                  const int32_t* allowed_img, int32_t* parent,
                                  int32_t* token, int32_t* depth, float* score, int32_t* pos, uint64_t* mask,
                                  int32_t* allowed_rows, int32_t* qrow, int32_t* n_out, bool keep_all,
                                  hipStream_t st) {
  ADT_CHECK_ARG(C >= 1 && C <= EXPAND_MAX_POOL, ADT_E_CAPACITY, "expand_finalize: pool of %d candidates (at most %d)", C,
                EXPAND_MAX_POOL);
  ADT_CHECK_ARG(keep_all ? C <= ADT_MAX_NODES - 1 : n_budget <= ADT_MAX_NODES - 1, ADT_E_CAPACITY,
                "expand_finalize: tree of more than %d nodes", ADT_MAX_NODES);
  const size_t smem = (size_t)C * (sizeof(uint64_t) + sizeof(int32_t));
  expand_finalize_kernel<<<1, FIN_THREADS, smem, st>>>(pool, C, n_budget, root_token, L, P, n_image, allowed_img,
                                                       parent, token, depth, score, pos, mask, allowed_rows, qrow, n_out,
                                                       keep_all ? 1 : 0);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_accept_greedy(const int32_t* argmax, int kmax, const int32_t* parent, const int32_t* token,
                                const int32_t* n_nodes, int n_max, int32_t* path, int32_t* n_acc, int32_t* bonus,
                                hipStream_t st) {
  accept_greedy_kernel<<<1, 64, 0, st>>>(argmax, kmax, parent, token, n_nodes, n_max, path, n_acc, bonus);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

}  // namespace adt
