// Host-side launchers of the kernels in csrc/kernels (internal to the library).
#pragma once

#include "common.h"

namespace adt {

// Guidance branches of a forward (classifier-free guidance): row r is node r / nb of branch
// r % nb (branch 0 conditional, 1 unconditional; nb = 1 without guidance).  The token of row
// r is tok[node + branch * tok_boff] (tok_boff = 0: the branches share one token list); the
// caches of branch b start cache_sb elements after those of branch 0.
struct Branches {
  int nb = 1;
  int tok_boff = 0;
  int64_t cache_sb = 0;
};

// Device error words of the source files whose kernels test invariants (debug builds; 0 in
// release builds): read and cleared, with the current device synchronised by the copy.
uint32_t dev_errors_take_rows();
uint32_t dev_errors_take_select();
uint32_t dev_errors_take_attn();
uint32_t dev_errors_take_gemm();

// attn.hip
// Row of query qr of sequence b in q and out: b * rs_b + qr * rs_i (rows of H * Dh); its mask
// row: b * ms_b + qr.  Separate sequences: (nq_max, 1, nq_max).  Guidance branches of one
// tree interleaved node by node: (1, B, 0), one mask per node.  With row_off (device, [B])
// the rows of sequence b start at row_off[b] instead (packed trees of different sizes), for
// q, out and masks alike.  o_pk > 0 stores out (bf16) in the fragment layout of o_pk row
// blocks (the input layout of the O projection), else row-major.
struct AttnRows {
  int rs_b, rs_i, ms_b;
  const int32_t* row_off = nullptr;
  int o_pk = 0;
  __device__ __forceinline__ int64_t q_row(int b, int qr) const {
    return (row_off ? (int64_t)row_off[b] : (int64_t)b * rs_b) + (int64_t)qr * rs_i;
  }
  // element (head h, dim d) of query qr's output row
  __device__ __forceinline__ int64_t o_index(int b, int qr, int H, int DH, int h, int d) const {
    return act_index(q_row(b, qr), h * DH + d, (int64_t)H * DH, o_pk);
  }
  __device__ __forceinline__ int64_t m_row(int b, int qr) const {
    return (row_off ? (int64_t)row_off[b] : (int64_t)b * ms_b) + qr;
  }
};
size_t tree_attn_ws_bytes(int B, int H, int Dh, int nq_max, int kv_cap, int dtype);
// Exact scratch bytes one launch of these sizes uses (0 unless it splits the keys).
size_t tree_attn_ws_need(int B, int H, int Dh, int nq_max, int kv_cap, int dtype);
adt_status launch_tree_attn(const void* q, const void* k, const void* v, int64_t sb, int64_t sh, const int32_t* kv_len,
                            const int32_t* n_q, const int32_t* n_tail, const uint64_t* mask, AttnRows rl, int B, int H,
                            int Dh, int nq_max, int kv_cap, float scale, int dtype, void* out, void* ws,
                            size_t ws_bytes, hipStream_t st, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);

// gemm.hip
size_t packed_bytes(int total_rows, int K, int dtype);
adt_status launch_pack(const void* const* srcs, const int32_t* rows, int n_src, int K, int mode, int group, int dtype,
                       void* dst, hipStream_t st);
// bf16 projections at batch 1 (M <= 128 rows of bf16 input, weights packed): each workgroup
// owns T 16-column tiles and one of S contiguous K ranges; its eight waves split that range
// and their partial tiles are summed in LDS in wave order.  With S = 1 the finished tile
// runs the epilogue; EPI_PART stores the S range sums instead, for resid_norm to add in
// range order.  T and S come from gemm_rows_plan.
enum : int { EPI_STORE = 1, EPI_PART = 2, EPI_QKV = 3, EPI_SWIGLU = 4, EPI_RESID = 5 };
struct GemmEpi {
  int mode = EPI_STORE;
  // EPI_STORE: out[m][n] (fp32, leading dimension ldo)
  float* out = nullptr;
  int64_t ldo = 0;
  // EPI_PART: part[s][m][n] (fp32), the sum over K range s of S
  float* part = nullptr;
  size_t part_elems = 0;
  // EPI_QKV (weights packed with ADT_PACK_QKV): q to q[m][H*Dh] after RoPE at pos[m]; k (RoPE)
  // and v to cache slot (*slot0 + m), element (head, slot, :) at kc + head*stride_h + slot*Dh
  uint16_t* q = nullptr;
  uint16_t* kc = nullptr;
  uint16_t* vc = nullptr;
  int64_t stride_h = 0;
  const int32_t* slot0 = nullptr;
  const int32_t* pos = nullptr;
  const float2* rope = nullptr;
  int Dh = 0;
  int nb = 1;              // guidance branches: row m is node m / nb of branch m % nb, whose
  int64_t cache_sb = 0;    // caches sit cache_sb elements further; q keeps row m
  int slot_cap = 0;        // cache slots per head (> 0: rows whose slot would pass it are not
                           // stored; debug builds record them)
  // EPI_SWIGLU (weights packed with ADT_PACK_GATE_UP): act[m][N/2] = silu(gate) * up, in
  // the fragment layout of act_pk row blocks (0: row-major)
  uint16_t* act = nullptr;
  int act_pk = 0;
  // EPI_RESID (one K range): resid[m][n] (fp32, [M][N]) += Y (assign: = Y), then act[m][n] =
  // the new residual in bf16, layout act_pk
  float* resid = nullptr;
  int assign = 0;
  // norm_eps > 0 (not with EPI_PART or EPI_RESID): the input rows are un-normalised and every
  // output row is scaled by 1 / sqrt(mean of its input row's squares + norm_eps), the RMSNorm
  // (unit gain) of the bf16 rows the kernel reads
  float norm_eps = 0.f;
};
struct RowsPlan {
  int T, S;       // at most T 16-column tiles per workgroup, S K ranges
  int G;          // column groups: group c takes tiles [c tiles / G, (c + 1) tiles / G)
};
RowsPlan gemm_rows_plan(int M, int N, int K, bool partial, bool wide = false);
constexpr int GEMM_MAX_SPLITS = 8;
// fp32: part[M][N] = X . W^T (consumed by the row kernels).  bf16: the kernel above with the
// epilogue epi; *splits (if given) gets S.  bf16 X is row-major with leading dimension ldx, or
// with ldx == X_FRAG in the fragment layout of (M + 15) / 16 row blocks.
constexpr int X_FRAG = 0;
adt_status launch_gemm(const void* X, int ldx, const void* Wp, int M, int N, int K, int dtype, float* part,
                       const GemmEpi& epi, hipStream_t st, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr,
                       int* splits = nullptr);
// gemm_nt.hip: C[M][N] fp32 = X[M][K] . W[N][K]^T, bf16 row-major operands (MFMA-bound batches)
// (packed: W in the adt_pack_weight layout, ldw unused; rows in the packed order)
// part: fp32 scratch of part_elems for K-split partials of the packed path (null: no split);
// gemm_nt_part_elems gives what the packed path's plan uses with unlimited scratch.
adt_status launch_gemm_nt(const void* X, int64_t ldx, const void* W, int64_t ldw, int M, int N, int K, float* C,
                          int64_t ldc, hipStream_t st, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr,
                          bool packed = false, float* part = nullptr, size_t part_elems = 0);
size_t gemm_nt_part_elems(int M, int N, int K);
// rows.hip
// h = embedding rows, a = RMSNorm(h) (raw: h itself) in the model dtype (bf16: fragment
// layout of a_pk row blocks when a_pk > 0, else row-major).
adt_status launch_embed_norm(const void* E, const int32_t* tok, int M, int d, float eps, float* h, void* a, int dtype,
                             hipStream_t st, const Branches& br = Branches{}, int a_pk = 0, bool raw = false);
// The residual projection's finish, one row per workgroup: y = sum over s < S of part[s][m][:]
// (in s order), h[m] = y (assign) or h[m] + y, then RMSNorm(h[m]) in the model dtype into out
// (layout out_pk: the next projection's input, or the final features) and, if out2 is given,
// into out2 as well (layout out2_pk).
adt_status launch_resid_norm(const float* part, int S, int M, int d, int assign, float eps, float* h, void* out,
                             int out_pk, void* out2, int out2_pk, int dtype, hipStream_t st);
// The same finish without the norm (the next projection normalises its own input rows):
// h[m] = y (assign) or h[m] + y, out[m] = h[m] in bf16, fragment layout out_pk.  Elementwise,
// four columns per thread.
adt_status launch_resid_add(const float* part, int S, int M, int d, int assign, float* h, void* out, int out_pk,
                            hipStream_t st);
// x[m] = [E[token] ; parent feature]: fsrc >= 0 is a node of fa, -1 zeros, <= -2 node
// (-2 - fsrc) of fb; fa and fb hold the nb branch rows of a node consecutively.  x is [M][2d]
// row-major, or in the fragment layout of x_pk row blocks.
adt_status launch_draft_input(const void* E, const int32_t* tok, const int32_t* fsrc, const void* fa, const void* fb,
                              int M, int d, void* x, int dtype, hipStream_t st, const Branches& br = Branches{},
                              int x_pk = 0);
adt_status launch_add_norm(const float* part, int splits, int M, int d, int assign, float eps, float* h, void* a,
                           int dtype, hipStream_t st);
adt_status launch_rope_table(float2* tab, int positions, int Dh, double theta, hipStream_t st);
adt_status launch_qkv_rope(const float* part, int splits, int M, int H, int Dh, const int32_t* pos,
                           const int32_t* slot0, const float2* rope, void* qout, void* kc, void* vc, int64_t stride_h,
                           int dtype, hipStream_t st, const Branches& br = Branches{});
// Batched verify: RoPE and cache append from fp32 QKV products in ADT_PACK_QKV column order;
// row m belongs to sequence seq[m] (caches cache_sb elements apart), position pos[m], slot slot[m].
adt_status launch_qkv_rows(const float* C, int M, int H, int Dh, const int32_t* pos, const int32_t* slot,
                           const int32_t* seq, const float2* rope, void* qout, void* kc, void* vc, int64_t stride_h,
                           int64_t cache_sb, int dtype, hipStream_t st);
adt_status launch_swiglu(const float* part, int splits, int M, int F, void* out, int dtype, hipStream_t st);
adt_status launch_reduce_store(const float* part, int splits, int M, int N, float* out, int64_t ldo, hipStream_t st);
adt_status launch_gather_rows(const void* src, const int32_t* idx, int cnt, int d, void* dst, int dtype,
                              hipStream_t st);
adt_status launch_kv_compact(void* k, void* v, int B, int slices, int Dh, int64_t sb, int64_t ss, const int32_t* kv_len,
                             int kv_stride, const int32_t* path, int path_stride, const int32_t* n_acc, int acc_stride,
                             int a_max, int dtype, hipStream_t st);
// out[i] = u + scale (c - u) over V logits, c = raw[2i], u = raw[2i + 1] (rows of V floats).
adt_status launch_guide_rows(const float* raw, int rows, int V, float scale, float* out, int64_t ldo, hipStream_t st);
adt_status launch_tree_masks(const int32_t* parent, const int32_t* n_nodes, int B, int n_max, uint64_t* mask,
                             int32_t* depth, hipStream_t st);

// select.hip
struct Pool {
  int32_t* token;
  float* score;
  int32_t* depth;
  int32_t* parent;
  int32_t* drow;
  int32_t* qrow;   // draft-logit row that drew an expanded node's children (-1 otherwise)
  uint64_t* rmask;
};
struct NextRows {
  int32_t* tok;
  int32_t* fsrc;
  int32_t* pos;
  uint64_t* mask;
  int32_t* frontier;
};
// Top-k (ids and logits, rows of kmax) and log-sum-exp of each row over its allowed range
// (allowed: [rows][2] device pairs, or null for the range [lo, hi) of every row); ws holds
// row_topk_ws_bytes(rows, kmax) bytes of per-chunk candidates.
size_t row_topk_ws_bytes(int rows, int kmax);
adt_status launch_row_topk(const float* logits, int64_t ld, int V, const int32_t* allowed, int rows, int k, int kmax,
                           int32_t* top_id, float* top_val, float* lse, void* ws, size_t ws_bytes, hipStream_t st,
                           int lo = 0, int hi = 0);
adt_status launch_expand_level(const Pool& pool, const int32_t* front, int nf, int cnt, int base, int depth, int k_hat,
                               const int32_t* top_id, const float* top_val, const float* lse, int kmax, int make_next,
                               int L, int drow_base, int root_frow, int tree_frow0, int qrow_base, const NextRows& nx,
                               hipStream_t st);
// keep_all: every pool node in creation order (stochastic children), else the top-N rerank
adt_status launch_expand_finalize(const Pool& pool, int C, int n_budget, int root_token, int L, int P, int n_image,
                                  const int32_t* allowed_img, int32_t* parent, int32_t* token, int32_t* depth,
                                  float* score, int32_t* pos, uint64_t* mask, int32_t* allowed_rows, int32_t* qrow,
                                  int32_t* n_out, bool keep_all, hipStream_t st);
// Largest candidate pool the rerank holds in LDS.
constexpr int EXPAND_MAX_POOL = 4096;
adt_status launch_accept_greedy(const int32_t* argmax, int kmax, const int32_t* parent, const int32_t* token,
                                const int32_t* n_nodes, int n_max, int32_t* path, int32_t* n_acc, int32_t* bonus,
                                hipStream_t st);

// small.hip
struct SmallI32 {
  int32_t v[32];
};
adt_status launch_set_i32(int32_t* dst, const SmallI32& vals, int count, hipStream_t st);
adt_status launch_fill_pairs(int32_t* dst, int rows, int lo, int hi, hipStream_t st);
// The draft catch-up rows (cu <= 32): ctok = tok, cfsrc = 0..cu-1, cpos = Ld.., chain masks.
adt_status launch_catchup_rows(const SmallI32& tok, int cu, int Ld, int32_t* ctok, int32_t* cfsrc, int32_t* cpos,
                               uint64_t* cmask, hipStream_t st);
adt_status launch_table_rows(const int32_t* tok, int count, int depth, int rows, int32_t* idx, hipStream_t st);
adt_status launch_iota(int32_t* dst, int count, int start, int step, hipStream_t st);
adt_status launch_chain_masks(uint64_t* mask, int n, hipStream_t st);
adt_status launch_tree_rows(const int32_t* depth, const int32_t* n_nodes, int n_max, int L, int P, int n_image,
                            const int32_t* allowed_img, int32_t* pos, int32_t* allowed_rows, float* score,
                            hipStream_t st);

// accept_sample.hip
// Stochastic children: per frontier row r (pool index front[r], the root when front is null),
// cnt i.i.d. draws from q (the acceptance's integer weights at temperature T, top_k) with
// Philox counter (step, parent tree index, j, 2); top_id/top_val [rows][kmax] receive the ids
// and their logits, lse [rows] the log-sum-exp at T = 1 over the allowed ids.  w: rows * V
// uint64 of scratch.
adt_status launch_row_sample(const float* logits, int64_t ld, int V, const int32_t* allowed, int rows,
                             const int32_t* front, int cnt, float T, int top_k, uint64_t seed, uint32_t step,
                             uint64_t* w, int32_t* top_id, float* top_val, float* lse, int kmax, hipStream_t st);
size_t accept_ws_bytes(int V);
adt_status launch_accept_sample(const float* logits, int64_t ld, int V, const int32_t* parent, const int32_t* token,
                                const int32_t* allowed, const int32_t* n_nodes, int n_max, const adt_accept_cfg& cfg,
                                uint64_t step, int32_t* path, int32_t* n_acc, int32_t* bonus, void* ws, size_t ws_bytes,
                                hipStream_t st);
adt_status launch_accept_mss(const float* logits, int64_t ld, int V, const int32_t* parent, const int32_t* token,
                             const int32_t* allowed, const int32_t* n_nodes, int n_max, const adt_accept_cfg& cfg,
                             uint64_t step, int32_t* path, int32_t* n_acc, int32_t* bonus, void* ws, size_t ws_bytes,
                             hipStream_t st);

// knn.hip
size_t knn_ws_bytes(int n);
adt_status launch_codebook_knn(const float* cb, int n, int dim, int k, int32_t* out, void* ws, size_t ws_bytes,
                               hipStream_t st);

}  // namespace adt
