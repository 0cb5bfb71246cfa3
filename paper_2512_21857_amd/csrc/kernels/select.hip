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

ADT_DEVICE_ERROR_WORD(select)

__device__ __forceinline__ bool better(float a, int ia, float b, int ib) { return a > b || (a == b && ia < ib); }

constexpr int TOPK_THREADS = 256;
constexpr int TOPK_WAVES = TOPK_THREADS / WAVE;
constexpr int TOPK_CHUNK = 8 * TOPK_THREADS;   // logits per chunk workgroup (two float4 per thread)
constexpr int TOPK_MAX_CHUNKS = 32;            // vocabularies up to 65536

// (value desc, id asc) as one 64-bit key, larger = better: the value's bits made
// order-preserving (-0 taken as +0) above the id's complement.  For values that are not NaN
// this is the order of better().
__device__ __forceinline__ uint64_t best_key(float v, int id) {
  const uint32_t u = __float_as_uint(v + 0.f);
  const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)o << 32) | (0xFFFFFFFFu - (uint32_t)id);
}

// max(v, v of the lane that the DPP pattern CTRL names), in the rows of row mask RM
template <int CTRL, int RM>
__device__ __forceinline__ uint64_t dpp_key_max(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)v, CTRL, RM, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(v >> 32), CTRL, RM, 0xF, false);
  const uint64_t t = ((uint64_t)hi << 32) | lo;
  return t > v ? t : v;
}

// The largest key of the wave (all 64 lanes active), as a uniform value: DPP exchanges within
// quads, half rows and rows (VALU moves, instead of six dependent LDS-pipe permutes), then
// the row broadcasts carry the maximum to lane 63.
__device__ __forceinline__ uint64_t wave_max_key(uint64_t v) {
  v = dpp_key_max<0xB1, 0xF>(v);    // quad_perm [1, 0, 3, 2]
  v = dpp_key_max<0x4E, 0xF>(v);    // quad_perm [2, 3, 0, 1]
  v = dpp_key_max<0x141, 0xF>(v);   // row_half_mirror
  v = dpp_key_max<0x140, 0xF>(v);   // row_mirror
  v = dpp_key_max<0x142, 0xA>(v);   // row_bcast:15 into rows 1 and 3
  v = dpp_key_max<0x143, 0xC>(v);   // row_bcast:31 into rows 2 and 3
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
  return ((uint64_t)hi << 32) | lo;
}

// Wave-wide argmax of (value desc, id asc) over every lane's (v, id), none NaN: v and id
// become the winner's (v exactly as the lane held it) and owner the lowest lane holding it.
__device__ __forceinline__ void wave_best(float& v, int& id, int& owner) {
  const uint64_t key = best_key(v, id);
  const uint64_t top = wave_max_key(key);
  owner = __ffsll((long long)__ballot(key == top)) - 1;
  v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), owner));
  id = (int)(0xFFFFFFFFu - (uint32_t)top);
}

// k rounds of "best remaining value of each lane, then the wave's best" over N values per
// lane (vals / ids, consumed); round q's winner goes to out_v[q] / out_i[q] (from lane 0).
// Rounds past the live values give (-inf, 0x7FFFFFFF).
template <int N>
__device__ __forceinline__ void wave_select(float (&vals)[N], int (&ids)[N], int kk, float* out_v, int* out_i) {
  const int lane = threadIdx.x % WAVE;
  for (int q = 0; q < kk; ++q) {
    float bv = -INFINITY;
    int bi = 0x7FFFFFFF;
#pragma unroll
    for (int j = 0; j < N; ++j)
      if (better(vals[j], ids[j], bv, bi)) {
        bv = vals[j];
        bi = ids[j];
      }
    if (bv == -INFINITY) bi = 0x7FFFFFFF;
    int bl = lane;
    wave_best(bv, bi, bl);
    if (lane == bl && bi != 0x7FFFFFFF) {
#pragma unroll
      for (int j = 0; j < N; ++j)
        if (ids[j] == bi) vals[j] = -INFINITY;
    }
    if (lane == 0) {
      out_v[q] = bv;
      out_i[q] = bi;
    }
  }
}

// Top-k ids by (logit desc, id asc) over the allowed range [lo, hi) of each row, and the
// row's log-sum-exp, in two launches.  Stage 1, one workgroup per (2048-logit chunk, row):
// the chunk's per-wave (max, sum of exp) pairs and its own top-k (each wave selects from its
// 512 logits, wave 0 merges the four lists).  Stage 2, one wave per row: the row's top-k
// from the chunks' lists and the log-sum-exp from their pairs.  Spreading a row over
// V / 2048 workgroups keeps the selection rounds (k of them, each a scan and a shuffle
// argmax) short; one workgroup per row ran them over 64 values per lane on a few CUs.
template <int KMAX>
__global__ __launch_bounds__(TOPK_THREADS) void topk_chunk_kernel(const float* __restrict__ logits, int64_t ld, int V,
                                                                  const int32_t* __restrict__ allowed, int ulo,
                                                                  int uhi, int k, float* __restrict__ cand_v,
                                                                  int* __restrict__ cand_i,
                                                                  float2* __restrict__ cand_ms, int c0) {
  __shared__ float wv[TOPK_WAVES][KMAX];
  __shared__ int wi[TOPK_WAVES][KMAX];
  // workgroup x covers chunk c0 + x of the row (outputs at x)
  const int chunk = blockIdx.x, G = gridDim.x, row = blockIdx.y;
  const int tid = threadIdx.x, lane = tid % WAVE, wave = tid / WAVE;
  const int lo = max(0, min(allowed ? allowed[row * 2] : ulo, V));
  const int hi = max(lo, min(allowed ? allowed[row * 2 + 1] : uhi, V));
  const float* x = logits + (int64_t)row * ld;
  const bool vec = ((ld & 3) == 0);
  float r[8];
  int id[8];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int base = (c0 + chunk) * TOPK_CHUNK + j * 4 * TOPK_THREADS + 4 * tid;
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
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      id[4 * j + e] = base + e;
      if (base + e < lo || base + e >= hi) r[4 * j + e] = -INFINITY;
    }
  }
  // the wave's (max, sum of exp) pair
  float m = -INFINITY;
#pragma unroll
  for (int j = 0; j < 8; ++j) m = fmaxf(m, r[j]);
  const float M = wave_max(m);
  float sacc = 0.f;
  if (M != -INFINITY) {
#pragma unroll
    for (int j = 0; j < 8; ++j) sacc += (r[j] == -INFINITY) ? 0.f : expf(r[j] - M);
  }
  const float S = wave_sum(sacc);
  if (lane == 0) cand_ms[((int64_t)row * G + chunk) * TOPK_WAVES + wave] = make_float2(M, S);
  const int kk = min(k, hi - lo);
  wave_select(r, id, kk, wv[wave], wi[wave]);
  __syncthreads();
  if (wave != 0) return;
  // wave 0: the chunk's top-k from the four wave lists (lane w < 4 offers list w's head)
  float* ov = cand_v + ((int64_t)row * G + chunk) * KMAX;
  int* oi = cand_i + ((int64_t)row * G + chunk) * KMAX;
  int h = 0;
  for (int q = 0; q < kk; ++q) {
    float hv = -INFINITY;
    int hid = 0x7FFFFFFF;
    if (lane < TOPK_WAVES && h < kk) {
      hv = wv[lane][h];
      hid = wi[lane][h];
    }
    int bl = lane;
    wave_best(hv, hid, bl);
    if (lane == bl) ++h;
    if (lane == 0) {
      ov[q] = hv;
      oi[q] = hid;
    }
  }
}

// Stage 2: one wave per row over the G chunk lists (G * KMAX <= 8 * WAVE candidates).
template <int KMAX>
__global__ __launch_bounds__(WAVE) void topk_merge_kernel(const float* __restrict__ cand_v,
                                                          const int* __restrict__ cand_i,
                                                          const float2* __restrict__ cand_ms, int G, int V,
                                                          const int32_t* __restrict__ allowed, int ulo, int uhi,
                                                          int k, int32_t* __restrict__ top_id, float* __restrict__ top_val,
                                                          float* __restrict__ lse) {
  constexpr int N = TOPK_MAX_CHUNKS * KMAX / WAVE > 0 ? TOPK_MAX_CHUNKS * KMAX / WAVE : 1;
  const int row = blockIdx.x, lane = threadIdx.x;
  const int lo = max(0, min(allowed ? allowed[row * 2] : ulo, V));
  const int hi = max(lo, min(allowed ? allowed[row * 2 + 1] : uhi, V));
  const int kk = min(k, hi - lo);
  // chunk c's list holds its min(k, live) entries; the rest of a list is never read
  float vals[N];
  int ids[N];
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const int e = j * WAVE + lane, c = e / KMAX, q = e % KMAX;
    vals[j] = -INFINITY;
    ids[j] = 0x7FFFFFFF;
    if (c < G && q < kk) {
      vals[j] = cand_v[((int64_t)row * G) * KMAX + e];
      ids[j] = cand_i[((int64_t)row * G) * KMAX + e];
    }
  }
  // log-sum-exp from the G * 4 (max, sum) pairs, in pair order within the lane
  float pm[2 * TOPK_MAX_CHUNKS * TOPK_WAVES / WAVE], ps[2 * TOPK_MAX_CHUNKS * TOPK_WAVES / WAVE];
  float gm = -INFINITY;
#pragma unroll
  for (int j = 0; j < 2 * TOPK_MAX_CHUNKS * TOPK_WAVES / WAVE; ++j) {
    const int e = j * WAVE + lane;
    pm[j] = -INFINITY;
    ps[j] = 0.f;
    if (e < G * TOPK_WAVES) {
      const float2 p = cand_ms[(int64_t)row * G * TOPK_WAVES + e];
      pm[j] = p.x;
      ps[j] = p.y;
    }
    gm = fmaxf(gm, pm[j]);
  }
  gm = wave_max(gm);
  float gs = 0.f;
#pragma unroll
  for (int j = 0; j < 2 * TOPK_MAX_CHUNKS * TOPK_WAVES / WAVE; ++j)
    if (pm[j] != -INFINITY) gs += ps[j] * expf(pm[j] - gm);
  gs = wave_sum(gs);
  if (lane == 0) lse[row] = gm + logf(gs);
  wave_select(vals, ids, kk, top_val + row * KMAX, top_id + row * KMAX);
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
      if (!(p >= 0 && p < i)) dev_fail(DEVINV_PARENT);
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
size_t row_topk_ws_bytes(int rows, int kmax) {
  return (size_t)rows * TOPK_MAX_CHUNKS * (kmax * 8 + TOPK_WAVES * 8) + 256;
}

adt_status launch_row_topk(const float* logits, int64_t ld, int V, const int32_t* allowed, int rows, int k, int kmax,
                           int32_t* top_id, float* top_val, float* lse, void* ws, size_t ws_bytes, hipStream_t st,
                           int lo, int hi) {
  ADT_CHECK_ARG(k >= 1 && k <= kmax && (kmax == 1 || kmax == 16), ADT_E_UNSUPPORTED, "row_topk: k=%d kmax=%d", k, kmax);
  const int G = (V + TOPK_CHUNK - 1) / TOPK_CHUNK;
  ADT_CHECK_ARG(V >= 1 && G <= TOPK_MAX_CHUNKS, ADT_E_UNSUPPORTED, "row_topk: vocab %d above 65536", V);
  ADT_CHECK_ARG(ws && ws_bytes >= row_topk_ws_bytes(rows, kmax), ADT_E_CAPACITY, "row_topk: workspace %zu < %zu", ws_bytes,
                row_topk_ws_bytes(rows, kmax));
  float2* cms = (float2*)ws;
  float* cv = (float*)(cms + (size_t)rows * G * TOPK_WAVES);
  int* ci = (int*)(cv + (size_t)rows * G * kmax);
  // one range for every row: only the chunks it touches (the chunks past it held -inf only;
  // Anole's 8192 image codes of 65536 ids: 4 chunks instead of 32)
  int c0 = 0, Gr = G;
  const int ulo = max(0, min(lo, V)), uhi = max(ulo, min(hi, V));
  if (!allowed && uhi > ulo) {
    c0 = ulo / TOPK_CHUNK;
    Gr = (uhi - 1) / TOPK_CHUNK + 1 - c0;
  }
  const dim3 g1(Gr, rows);
  if (kmax == 1) {
    topk_chunk_kernel<1><<<g1, TOPK_THREADS, 0, st>>>(logits, ld, V, allowed, lo, hi, k, cv, ci, cms, c0);
    ADT_LAUNCH_CHECK();
    topk_merge_kernel<1><<<rows, WAVE, 0, st>>>(cv, ci, cms, Gr, V, allowed, lo, hi, k, top_id, top_val, lse);
  } else {
    topk_chunk_kernel<16><<<g1, TOPK_THREADS, 0, st>>>(logits, ld, V, allowed, lo, hi, k, cv, ci, cms, c0);
    ADT_LAUNCH_CHECK();
    topk_merge_kernel<16><<<rows, WAVE, 0, st>>>(cv, ci, cms, Gr, V, allowed, lo, hi, k, top_id, top_val, lse);
  }
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
