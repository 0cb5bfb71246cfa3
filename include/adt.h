/*
 * adt.h -- C ABI of the ADT-Tree draft-then-verify hot path on one MI355X (gfx950).
 *
 * The method is ADT-Tree, "Fast Inference of Visual Autoregressive Model with
 * Adjacency-Adaptive Dynamical Draft Trees" (arXiv 2512.21857).  One cycle: a draft head
 * proposes a tree whose depth and width are chosen per image-grid position (Sec. 4.1,
 * Sec. 4.2 Eq. 2), the target model verifies all tree nodes in one forward under the
 * ancestor mask (Sec. 3.1), the accepted root-to-node path plus one bonus token is
 * committed (Sec. 3.1 Eq. 1; greedy decoding at T = 0 per Sec. 5.1), and the KV cache
 * is compacted so the accepted nodes become the prefix.
 *
 * Conventions for every call:
 *  - Status: ADT_OK (0) or a negative ADT_E_* code.  On an error nothing is enqueued and
 *    adt_last_error() returns a message (thread-local).  No C++ exception crosses the ABI.
 *  - Ownership: the caller allocates and owns every device buffer (weights, caches, tree
 *    arrays, logits, outputs, workspaces).  The library keeps non-owning pointers and never
 *    allocates device memory.  Pointers marked [host] are host memory; all others device.
 *  - Streams: `stream` is a hipStream_t (NULL = default stream).  Calls are asynchronous on
 *    it unless marked "synchronises".
 *  - Dtypes: ADT_F32 (float) or ADT_BF16 (bfloat16 stored as uint16 bit patterns).
 *    Row-major layouts.  A KV cache is [slices][S_cap][Dh] with a slice per (layer, head).
 *  - Trees: node 0 is the root (the last committed token), nodes are in BFS order
 *    (parent[i] < i), at most ADT_MAX_NODES nodes.  Ancestor masks are packed uint64
 *    words, ADT_MASK_WORDS per node: bit j of node i set iff j is on the path root..i.
 */
#ifndef ADT_H_
#define ADT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t adt_status;

#define ADT_OK 0
#define ADT_E_ARG (-1)         /* null pointer, bad enum, bad scalar */
#define ADT_E_SHAPE (-2)       /* dimension not supported by the kernels (alignment, head size) */
#define ADT_E_CAPACITY (-3)    /* tree, cache or workspace too small */
#define ADT_E_HIP (-4)         /* a HIP runtime call failed */
#define ADT_E_UNSUPPORTED (-5) /* valid request outside what the library implements */
#define ADT_E_DEVICE_INVARIANT (-6) /* debug builds: a kernel found device data breaking an invariant */
#define ADT_E_STATE (-7)       /* session used out of order (e.g. step before prefill) */

#define ADT_F32 0
#define ADT_BF16 1

#define ADT_MAX_NODES 128
#define ADT_MASK_WORDS 2

#define ADT_ACCEPT_GREEDY 0
#define ADT_ACCEPT_EXACT 1
#define ADT_ACCEPT_RELAXED 2
#define ADT_ACCEPT_MSS 3

#define ADT_ALPHA_REAL 0
#define ADT_ALPHA_POISSON 1

/* Initial tree attributes (d~, k~) of a cycle (Sec. 4.1 and the alternatives of Sec. 5.3) */
#define ADT_INIT_HORIZONTAL 0   /* the record of the left cell (i, j-1) */
#define ADT_INIT_VERTICAL 1     /* the record of the cell above (i-1, j) */
#define ADT_INIT_RANDOM 2       /* uniform over the depth and width bounds */
#define ADT_INIT_TOKENFLOCK 3   /* weighted mean over recorded cells within radius delta (Eqs. 6-8) */

/* Width bounds after Eq. 2 (Sec. 4.2) */
#define ADT_KCLAMP_ALWAYS 0     /* k_hat always clamped to [k_lo, k_hi] */
#define ADT_KCLAMP_DEEP 1       /* clamped only when the adapted depth d~ +- l_d exceeds 1; a
                                   one-layer tree keeps k_hat in [1, ADT_MAX_WIDTH] */
#define ADT_MAX_WIDTH 16        /* widest top-k of one expansion layer */

int32_t adt_version(void);
/* Copies the last error message of this thread into buf (NUL-terminated, truncated to cap);
 * returns its full length. */
size_t adt_last_error(char* buf, size_t cap);

/* Device invariant checks.  The library is also built as libadt_debug.so (same ABI, built
 * with ADT_DEVICE_CHECKS=1), whose kernels test the device-side data the host cannot see
 * before launching: a tree's parents come before their children (parent[0] = -1,
 * 0 <= parent[i] < i; the BFS order of Sec. 4.2's tree arrays), the keys a launch reads or
 * appends stay inside the cache (kv_len + n <= S_cap), accepted-path entries lie inside the
 * tree.  A kernel that finds a violation records it in a device error word and continues
 * within bounds (masked or skipped), so no access leaves its buffers.
 * adt_device_checks_enabled() is 1 in the debug build, 0 otherwise.
 * adt_device_check(stream) synchronises `stream` and returns ADT_E_DEVICE_INVARIANT (with a
 * message naming the invariants) if any kernel of this library recorded a violation since
 * the last check, clearing the record; ADT_OK otherwise (always in the release build, which
 * records nothing).  Every session call that synchronises (prefill, adt_step,
 * adt_session_accept_commit, ...) runs the same check after its own synchronisation. */
int32_t adt_device_checks_enabled(void);
adt_status adt_device_check(void* stream);

/* ------------------------------------------------------------------ b2: tree attention
 * Sec. 3.1: node i attends to the committed prefix and to the nodes on its own
 * root-to-node path.  For sequence b and head h:
 *   O[b][i][h] = softmax(scale * q[b][i][h] . K_S^T) V_S,
 *   S = slots [0, kv_len[b]) (prefix, unmasked) plus slots kv_len[b] + j for every j < n_tail[b]
 *       whose bit j is set in anc_mask[b][i] (the tail holds the tree nodes' own K/V).
 * q:        [B][nq_max][H][Dh]        dtype; rows i < n_q[b] are used
 * k_cache, v_cache: element (b, h, slot, :) at base + b*stride_b + h*stride_h + slot*Dh
 * kv_len, n_q, n_tail: [B] int32 device arrays; n_q[b] <= n_tail[b] <= ADT_MAX_NODES and
 *   kv_len[b] + n_tail[b] <= kv_cap (host bound used to size the launch)
 * anc_mask: [B][nq_max][ADT_MASK_WORDS] uint64
 * out:      [B][nq_max][H][Dh] dtype (rows >= n_q[b] untouched)
 * workspace: adt_tree_attn_workspace_size() bytes (split-KV partials)
 * Dh must be 64 or 128.  bf16 uses MFMA with fp32 accumulation and fp32 softmax; f32 is
 * computed in fp32 on the vector units. */
size_t adt_tree_attn_workspace_size(int32_t B, int32_t H, int32_t Dh, int32_t nq_max, int32_t kv_cap);
adt_status adt_tree_attn(const void* q, const void* k_cache, const void* v_cache, int64_t stride_b,
                         int64_t stride_h, const int32_t* kv_len, const int32_t* n_q, const int32_t* n_tail,
                         const uint64_t* anc_mask, int32_t B, int32_t H, int32_t Dh, int32_t nq_max,
                         int32_t kv_cap, float scale, int32_t dtype, void* out, void* workspace,
                         size_t workspace_bytes, void* stream);
/* adt_tree_attn for callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same arguments without the
 * workspace, the same result and the same errors.  The key-split partials live in a 16 MiB
 * device array inside the library, one per device, whose address is looked up on the first
 * call on that device; a call whose partials need more (only fewer than 128 sequence-head pairs
 * split the keys, into about 256 / pairs ranges: e.g. 120 pairs of 128-row trees at head size
 * 128 over 10000 slots need 24 MB; 32 pairs of 61-row trees need 8.1 MB) returns
 * ADT_E_CAPACITY and enqueues nothing.  Allocates nothing.  Every call on a device shares that
 * device's array and leaves the last call's partials in it: calls that overlap on one device
 * (several streams or threads) race, so the caller must serialise them. */
adt_status adt_tree_attn_noalloc(const void* q, const void* k_cache, const void* v_cache, int64_t stride_b,
                                 int64_t stride_h, const int32_t* kv_len, const int32_t* n_q, const int32_t* n_tail,
                                 const uint64_t* anc_mask, int32_t B, int32_t H, int32_t Dh, int32_t nq_max,
                                 int32_t kv_cap, float scale, int32_t dtype, void* out, void* stream);

/* ------------------------------------------------------------------ a3 support: masks
 * Ancestor bitmask and depth of every node of B BFS-ordered trees (Sec. 3.1 tree mask):
 * mask[i] = mask[parent[i]] | bit(i), depth[i] = depth[parent[i]] + 1, root depth 0.
 * parent: [B][n_max] (parent[b][0] = -1), n_nodes: [B] device; mask: [B][n_max][ADT_MASK_WORDS];
 * depth may be NULL.  Rows >= n_nodes[b] are zeroed. */
adt_status adt_tree_masks(const int32_t* parent, const int32_t* n_nodes, int32_t B, int32_t n_max,
                          uint64_t* mask, int32_t* depth, void* stream);

/* ------------------------------------------------------------------ d1: KV compaction
 * Implicit in Sec. 3.1 (the accepted tokens become the prefix): for each sequence b and
 * each cache slice (layer x head), slot L + m <- slot L + path[b][m] for m = 1..n_acc[b],
 * L = kv_len[b].  path[b][0] is the root (0) and is not read; path[b][m] >= m is required
 * (BFS order of an accepted chain) so every source is at or after its destination; all
 * reads of a slice happen before its writes.  Both K and V caches are compacted.
 * Slice s of sequence b starts at base + b*stride_b + s*stride_slice; rows are Dh long.
 * n_acc[b] <= a_max <= ADT_MAX_NODES - 1, and a_max rows of one slice at most 64 KB
 * (a_max * Dh * element size <= 65536; ADT_E_UNSUPPORTED otherwise). */
adt_status adt_kv_compact(void* k_cache, void* v_cache, int32_t B, int32_t slices, int32_t Dh, int64_t stride_b,
                          int64_t stride_slice, const int32_t* kv_len, const int32_t* path, int32_t path_stride,
                          const int32_t* n_acc, int32_t a_max, int32_t dtype, void* stream);

/* ------------------------------------------------------------------ c1-c3: acceptance
 * Walk from the root of one verified tree (Sec. 3.1 Eq. 1; Sec. 5.1).
 *  GREEDY: t_u = argmax of logits row u over its allowed ids (lowest id on ties); move to
 *    the child whose token is t_u while one exists; the bonus is t_u of the last node.
 *  EXACT: Eq. 1 with the drafted top-k children read as point-mass proposals: child x is
 *    accepted with probability p(x) and on rejection removed from p; siblings are tried in
 *    node order; with all rejected the bonus is drawn from the residual.  p = softmax of
 *    logits / temperature over the allowed ids truncated to the top_k largest (0 = all),
 *    held as integer weights rint(exp(z - max z) * 2^32).
 *  RELAXED: as EXACT but x is credited with the weights of its nearest codebook neighbours
 *    knn[x][1..knn_k-1] taken in order while their sum stays <= delta * (remaining total);
 *    on rejection the credited set is removed.
 *  MSS: Eq. 1 as printed, for trees whose children are i.i.d. draws from q (stochastic
 *    children, Sec. 3.1: each selected node generates its children by sampling from the
 *    draft distribution; a session in this mode expands that way, see adt_tree_expand).
 *    At node u the children are tried in node order: child x is accepted iff
 *    u32 * qw(x) * Wp < 2^32 * pw(x) * Wq (probability min(1, p(x) / q(x))), u32 = U >> 32
 *    of the draw at (step, u, trial, 0); after a rejection pw(y) <- max(0, pw(y) Wq -
 *    qw(y) Wp) >> s with s the least shift leaving every weight below 2^32 (the residual
 *    norm(max(0, p - q)) of multi-step speculative sampling); with all rejected the bonus
 *    is drawn from the residual, at a leaf from p.  qw, Wq: the weights (same temperature
 *    and top_k as p) of row q_row[u] of q_logits, the draft row that drew u's children.
 *  Draws: r = floor(U * W / 2^64), U = Philox4x32-10(key = seed, counter = (step, node,
 *    trial, 0)) words (x1 << 32 | x0), W = remaining total weight.
 * logits: [n][ld] fp32 (row u gives the target distribution of u's successor)
 * parent, token: [n] BFS tree; allowed: [n][2] allowed id range [lo, hi) per row; n_nodes: device
 *   scalar n; n_max [host] = rows allocated in logits/parent/token/allowed (n <= n_max <= ADT_MAX_NODES)
 * path: [ADT_MAX_NODES] out, path[0] = 0 then v_1..v_a; n_acc, bonus: device scalars out.
 * workspace: adt_accept_workspace_size(); only sampling modes use it.  EXACT and RELAXED need
 *   V <= 65536 (ADT_E_UNSUPPORTED otherwise). */
typedef struct {
  int32_t mode;        /* ADT_ACCEPT_* */
  float temperature;   /* > 0 for sampling modes */
  int32_t top_k;       /* sampling truncation, 0 = none; <= 4096 */
  float delta;         /* relaxed-mode mass bound, in [0, 1) */
  int32_t knn_k;       /* neighbours per code used in relaxed mode (row 0 is the code itself) */
  int32_t knn_rows;    /* rows of the knn table (ids >= knn_rows have no neighbours) */
  int32_t knn_stride;  /* int32 per knn row */
  const int32_t* knn;  /* device [knn_rows][knn_stride] */
  uint64_t seed;
  int32_t children;    /* MSS sessions: children drawn per expanded node, in [1, 16] and <= n_budget */
  const float* q_logits;   /* MSS, adt_verify_accept: device [rows][q_ld] draft logits (sessions set their own) */
  int64_t q_ld;
  const int32_t* q_row;    /* MSS, adt_verify_accept: device [n] row of q_logits that drew node u's children;
                              an entry outside [0, q_rows) stops the walk at u (bonus drawn from p) */
  int32_t q_rows;          /* MSS, adt_verify_accept: rows of q_logits */
} adt_accept_cfg;

size_t adt_accept_workspace_size(int32_t V);
adt_status adt_verify_accept(const float* logits, int64_t ld, int32_t V, const int32_t* parent, const int32_t* token,
                             const int32_t* allowed, const int32_t* n_nodes, int32_t n_max,
                             const adt_accept_cfg* cfg /*[host]*/,
                             uint64_t step, int32_t* path, int32_t* n_acc, int32_t* bonus, void* workspace,
                             size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ c3 support: neighbours
 * Neighbour table of a VQ codebook for relaxed acceptance: out[x][0] = x, then the k-1
 * other codes of highest cosine similarity to code x (fp32, ties to the lower id).
 * codebook: [n][dim] fp32; out: [n][k] int32 (k <= 256); workspace:
 * adt_codebook_knn_workspace_size(n) bytes.  Set-up work, run once per codebook. */
size_t adt_codebook_knn_workspace_size(int32_t n);
adt_status adt_codebook_knn(const float* codebook, int32_t n, int32_t dim, int32_t k, int32_t* out, void* workspace,
                            size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ b3 for a batch of trees
 * The dense projections of the verification forward (Sec. 3.1) when the rows of several
 * trees are multiplied together (M = their total, in the hundreds), where the product is
 * bound by the matrix cores rather than by the weight stream: C[M][N] = X[M][K] . W[N][K]^T.
 * X, W: device bf16, row-major with K contiguous (leading dimensions ldx, ldw >= K,
 * multiples of 8 elements); C: device fp32 [M][ldc] (ldc >= N, a multiple of 4).  N must be
 * a multiple of 128 and K of 64; M >= 1.  Asynchronous on `stream`.  ADT_E_ARG on null
 * pointers, ADT_E_SHAPE on other shapes; nothing is enqueued on error. */
adt_status adt_gemm_bf16(const void* X, int64_t ldx, const void* W, int64_t ldw, int32_t M, int32_t N, int32_t K,
                         float* C, int64_t ldc, void* stream);

/* The same product with W in the packed layout of adt_pack_weight (ADT_PACK_STACK, bf16;
 * the layout every model weight is kept in), as the batched verification forward multiplies
 * it.  Wp: device, adt_packed_bytes(N, K, ADT_BF16) bytes, W's rows in their packed
 * order (C's columns follow that order).  workspace: NULL, or device scratch of
 * adt_gemm_bf16_packed_workspace_size(M, N, K) bytes (0 when the product needs none), with
 * which K is split across 2-4 workgroups per output block for a product of few blocks and
 * long K (K >= 8192), or for the columns of a last, at most half-full round of blocks, and
 * the fp32 partials are added to C in a fixed order (deterministic; rounding then differs
 * from the unsplit product by the reassociation of the K sum).  A NULL workspace splits
 * nothing; a smaller one splits only as far as it holds the partials.  Shapes, errors and
 * asynchrony as adt_gemm_bf16. */
size_t adt_gemm_bf16_packed_workspace_size(int32_t M, int32_t N, int32_t K);
adt_status adt_gemm_bf16_packed(const void* X, int64_t ldx, const void* Wp, int32_t M, int32_t N, int32_t K, float* C,
                                int64_t ldc, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ weights
 * Repacks row-major [rows][K] matrices (rows = output features) into the layout the GEMM
 * kernels stream.  srcs/rows: [host] arrays of n_src device pointers and their row counts.
 * Row order of the packed matrix:
 *   ADT_PACK_STACK    the sources stacked in order (lm_head, draft FC, O, down; the fp32 QKV);
 *   ADT_PACK_GATE_UP  n_src = 2 equal sources (gate, up) interleaved in blocks of 8 rows:
 *                     gate rows 8t..8t+7, then up rows 8t..8t+7, t = 0, 1, ... (both dtypes);
 *   ADT_PACK_QKV      the sources (q, k, v) stacked; inside every head of `group` rows
 *                     (= head_dim, a multiple of 16) each 16-row block u holds rows 8u..8u+7
 *                     of the head's first half then the same rows of its second half, so a
 *                     RoPE pair (j, j + head_dim/2) lands in one block (bf16 QKV weights).
 * group is ignored by the other modes.  bf16: rows and K multiples of 16 and 32, stored as
 * 16x32 tiles; dst holds sum(rows)*K bf16.  f32: the same row order, row-major.
 * adt_packed_bytes() gives the size.  ADT_E_ARG on a bad mode, ADT_E_SHAPE on shapes the
 * mode cannot tile. */
enum { ADT_PACK_STACK = 0, ADT_PACK_GATE_UP = 1, ADT_PACK_QKV = 2 };
size_t adt_packed_bytes(int32_t total_rows, int32_t K, int32_t dtype);
adt_status adt_pack_weight(const void* const* srcs, const int32_t* rows, int32_t n_src, int32_t K, int32_t mode,
                           int32_t group, int32_t dtype, void* dst, void* stream);

/* ------------------------------------------------------------------ a0: schedule (host)
 * A cycle's tree shape is found in two phases (Sec. 4): an initial (d~, k~) from the records
 * of committed cells (adt_schedule_init, Sec. 4.1 and Sec. 5.3), then the bisectional
 * adaptation of Eq. 2 and the bounds of Sec. 4.2 (adt_schedule_next).
 *
 * The record of an image cell is the (d_hat, k_hat) of the tree whose cycle committed it;
 * cells are numbered in raster order, cell = i * grid_w + j.  Rules (init_mode):
 *   HORIZONTAL: the record of cell - 1 (the raster predecessor at j = 0).
 *   VERTICAL:   the record of cell - grid_w; in the first row, or where that cell has no
 *               record, the HORIZONTAL value.
 *   RANDOM:     d~ = d_lo + floor(U0 * (d_hi - d_lo + 1) / 2^64),
 *               k~ = k_lo + floor(U1 * (k_hi - k_lo + 1) / 2^64), where (x0..x3) =
 *               Philox4x32-10(key = seed, counter = (cell, 0, 0, 1)), U0 = x1 << 32 | x0 and
 *               U1 = x3 << 32 | x2; every cycle, the first included.
 *   TOKENFLOCK: over the recorded cells c < cell with (dx^2 + dy^2) <= delta^2 (x = column,
 *               y = row), weights w = delta + 1 - dy normalised to sum 1; d~ and k~ are the
 *               weighted means rounded half up.
 * With no source (no record yet, or an empty TOKENFLOCK set) the tree starts from (d0, k0)
 * and skips Eq. 2.  fix_d / fix_k > 0 replace d~ / k~ by that constant (the fixed-base
 * ablations of Table V), the first tree included. */
typedef struct {
  int32_t d_lo, d_hi, k_lo, k_hi; /* inclusive bounds */
  int32_t l_d, l_k;               /* adjustment steps of Eq. 2 */
  float beta;                     /* positive threshold of Eq. 2 */
  int32_t n_budget;               /* draft nodes kept by the top-N rerank (Eq. 3) */
  int32_t d0, k0;                 /* first tree */
  int32_t alpha_source;           /* ADT_ALPHA_REAL or ADT_ALPHA_POISSON */
  int32_t init_mode;              /* ADT_INIT_* */
  int32_t grid_w;                 /* cells per grid row; >= 1 for VERTICAL and TOKENFLOCK */
  int32_t flock_delta;            /* TOKENFLOCK radius, >= 1 */
  int32_t fix_d, fix_k;           /* fixed initial depth / width, 0 = none */
  int32_t k_clamp;                /* ADT_KCLAMP_ALWAYS or ADT_KCLAMP_DEEP (needs d_lo = 1) */
  uint64_t seed;                  /* RANDOM key */
} adt_sched_cfg;

/* Initial (d~, k~) of the cycle whose first drafted token is image cell `cell`.
 * rec_d, rec_k, has_rec: [host] [n_cells] records (only entries below `cell` are read).
 * Writes have_init = 0 (start from (d0, k0) without adaptation) or 1 with (d_init, k_init).
 * ADT_E_ARG on null pointers, a cell outside [0, n_cells) or an invalid rule setting. */
adt_status adt_schedule_init(const adt_sched_cfg* cfg, int32_t cell, int32_t n_cells, const int32_t* rec_d,
                             const int32_t* rec_k, const int32_t* has_rec, int32_t* have_init, int32_t* d_init,
                             int32_t* k_init);

/* Eq. 2 and the bounds.  have_left: whether an initial value (d_left, k_left) exists (from
 * adt_schedule_init; 0 = start from (d0, k0) and skip Eq. 2); have_prev: whether a previous
 * tree exists, with a_prev accepted draft tokens at depth d_prev (alpha = a_prev / d_prev,
 * positive iff alpha >= beta); remaining = image tokens still to commit including this
 * cycle's bonus.  The depth is clamped to [d_lo, d_hi] and then cut to remaining - 1; the
 * width per k_clamp.  Writes (d_hat, k_hat); d_hat = 0 means a plain AR step. */
adt_status adt_schedule_next(const adt_sched_cfg* cfg, int32_t have_left, int32_t d_left, int32_t k_left,
                             int32_t have_prev, int32_t a_prev, int32_t d_prev, int32_t remaining, int32_t* d_hat,
                             int32_t* k_hat);

/* ------------------------------------------------------------------ model and session */
typedef struct adt_model_s adt_model;
typedef struct adt_session_s adt_session;

typedef struct {
  int32_t n_layers, d_model, n_heads, head_dim, ffn, vocab;
  int32_t dtype;
  float rope_theta, norm_eps;
  const void* embed;            /* [vocab][d_model] row-major, dtype */
  const void* lm_head;          /* packed [vocab][d_model] */
  const void* draft_fc;         /* packed [d_model][2 d_model] (input = [embedding ; parent feature]) */
  const void* const* w_qkv;     /* [host] n_layers + 1 packed [3d][d] (q, k, v): ADT_PACK_QKV with group =
                                   head_dim for bf16, ADT_PACK_STACK for f32; last = draft layer */
  const void* const* w_o;       /* [host] n_layers + 1 packed [d][d] */
  const void* const* w_gu;      /* [host] n_layers + 1 packed [2F][d], ADT_PACK_GATE_UP */
  const void* const* w_down;    /* [host] n_layers + 1 packed [d][F] */
} adt_model_desc;

adt_status adt_model_create(const adt_model_desc* desc, adt_model** out);
void adt_model_destroy(adt_model* m);

typedef struct {
  int32_t prefix_len;           /* committed prompt tokens before the image */
  int32_t n_image;              /* image tokens (grid cells, raster order) */
  int32_t s_cap;                /* cache slots; >= prefix_len + n_image + ADT_MAX_NODES */
  void* k_cache;                /* target [n_layers][n_heads][s_cap][head_dim] */
  void* v_cache;
  void* dk_cache;               /* draft  [n_heads][s_cap][head_dim] */
  void* dv_cache;
  const int32_t* allowed;       /* [host] [n_image][2] allowed id range [lo, hi) per image cell (copied) */
  adt_sched_cfg sched;
  adt_accept_cfg accept;
  const int32_t* poisson;       /* [host] [n_image] acceptance lengths for ADT_ALPHA_POISSON, else NULL */
  int32_t fixed_tree;           /* 1: skip the schedule, always (sched.d_hi, sched.k_hi) */
  /* Optional caller-supplied draft distribution instead of the draft head: the draft logits
   * of a row whose token is t at depth l (the root row has depth 0) are row
   * (l * 131 + t) mod draft_table_rows of draft_table [rows][vocab] fp32.  Used to drive the
   * expansion (a2, a3) with known logits; NULL = run the draft head. */
  const float* draft_table;
  int32_t draft_table_rows;
  /* 1: capture the verify and draft forwards as HIP graphs (one per tree shape, built on
   * first use on a private stream, replayed on the caller's stream); 0: plain launches. */
  int32_t use_graphs;
  /* Classifier-free guidance in target and draft (Sec. 3.1; Fig. 5 caption): guided = 1 runs
   * every forward over a conditional and an unconditional branch and uses the logits
   * l_u + guidance_scale (l_c - l_u) for drafting and acceptance.  Then the caches hold both
   * branches, branch 1 after branch 0 (k_cache / v_cache [2][n_layers][n_heads][s_cap]
   * [head_dim], dk_cache / dv_cache [2][n_heads][s_cap][head_dim]), the prompt passed to
   * adt_session_prefill is both prompts ([2][prefix_len]: conditional, then unconditional,
   * equally long), and a tree holds at most ADT_MAX_NODES / 2 nodes (n_budget <= 63). */
  int32_t guided;
  float guidance_scale;
  void* workspace;
  size_t workspace_bytes;
} adt_session_desc;

typedef struct {
  int32_t step;                 /* cycle index (1 for the first tree) */
  int32_t d_hat, k_hat;         /* tree shape chosen by the schedule */
  int32_t n_nodes;              /* verified rows, root included */
  int32_t n_accepted;           /* a */
  int32_t n_committed;          /* a + 1 */
  int32_t tokens[ADT_MAX_NODES];/* committed ids */
  int32_t done;                 /* 1 once every image token is committed */
} adt_step_out;

typedef struct {
  int32_t L;                    /* committed target KV length (root position) */
  int32_t Ld;                   /* valid draft KV length */
  int32_t step;                 /* next cycle index */
  int32_t n_tokens;             /* committed tokens, prompt included */
  int32_t n_nodes;              /* rows of the current tree */
  float* logits;                /* [ADT_MAX_NODES][vocab] last verify logits (unmasked; columns below) */
  void* feat;                   /* [ADT_MAX_NODES][d_model] last verify features */
  float* draft_logits;          /* [1 + (d_hi-1) k_hi][vocab] root row then frontier rows, per level */
  int32_t* parent; int32_t* token; int32_t* depth; float* score; uint64_t* mask;  /* current tree */
  int32_t* allowed_rows;        /* [ADT_MAX_NODES][2] allowed range of each row's successor */
  int32_t* path; int32_t* n_acc; int32_t* bonus;  /* last acceptance */
  const int32_t* tokens_host;   /* [host] committed ids */
  /* scratch of the last forward (last layer run): rotated queries [rows][d] dtype, attention
   * output [rows][d] dtype, normed activations [rows][d] dtype, residual stream [rows][d] fp32.
   * In bf16 sessions act holds the bf16 residual rows (each projection applies its RMSNorm
   * itself) except after a forward's last layer, where it holds the final norm; att and act
   * are then in the fragment layout of the projections' inputs: with
   * B = (rows + 15) / 16 row blocks, element (r, k) sits at
   * (((k / 32) * B + r / 16) * 64 + r % 16 + 16 * ((k % 32) / 8)) * 8 + k % 8. */
  void* q; void* att; void* act; float* resid;
  /* guidance: rows of the last forwards hold node i's branches at rows nb i + b (b = 0
   * conditional); feat is then [ADT_MAX_NODES / 2][2][d_model] and logits / draft_logits are
   * the guided ones */
  int32_t n_branches;
  float* branch_logits;         /* guided: [n][2][vocab] per-branch verify logits, else NULL */
  float* draft_branch_logits;   /* guided: [2][vocab] per-branch logits of the draft root row, else NULL */
  /* columns [logits_lo, logits_hi) of every logits row above are computed; the others are left
   * as they were.  bf16 sessions: the union of the image cells' allowed ranges, widened to
   * multiples of 16 (every step of the cycle reads a row's allowed range only); f32: the
   * whole vocabulary. */
  int32_t logits_lo, logits_hi;
} adt_session_view;

size_t adt_session_workspace_size(const adt_model* m, const adt_session_desc* desc);
adt_status adt_session_create(const adt_model* m, const adt_session_desc* desc, adt_session** out);
void adt_session_destroy(adt_session* s);
/* Target and draft over the prompt, then the first image token by one AR step (greedy or a
 * draw at step 0).  prefix: [host] prefix_len ids (guided: 2 * prefix_len, the conditional
 * prompt then the unconditional one).  Synchronises. */
adt_status adt_session_prefill(adt_session* s, const int32_t* prefix, int32_t* first_token, void* stream);
adt_status adt_session_get_view(const adt_session* s, adt_session_view* v);

/* Layer-by-layer record of the session's forwards, so that each decoder layer of the target
 * (Sec. 3.1, parallel verification) and of the draft head (Sec. 4.2; Fig. 5 caption) can be
 * compared with a reference evaluated from the same inputs.  For tests and debugging; off by
 * default.  While a capture is set the session's forwards run as plain launches (no graph
 * replay) and every forward appends, in order:
 *   resid:  fp32 snapshots of the residual stream, each [rows][d_model] (rows = nodes x
 *           branches, branch rows interleaved node by node): target forwards 2 n_layers + 1 of
 *           them (2l = the input of layer l, 2l + 1 = after layer l's attention block with the
 *           output projection added, 2 n_layers = the last layer's output, i.e. the final norm's
 *           input), draft forwards 3 (0 = the FC output, 1 = after the attention block, 2 = the
 *           layer output);
 *   xin:    draft forwards only: the FC input rows [rows][2 d_model] in the model dtype
 *           ([token embedding ; parent feature]);
 *   meta:   int32, per forward: token ids [nodes], positions [nodes], then the ancestor masks
 *           [nodes][ADT_MASK_WORDS] as uint64 (8-byte aligned).  Node r's K/V go to cache slot
 *           slot0 + r and it attends to slots [0, kv_prefix) plus kv_prefix + j for every set bit
 *           j of its mask.
 * The buffers are caller-owned device memory; a forward whose data would overrun one fails
 * with ADT_E_CAPACITY before it launches anything.  adt_session_set_capture resets the record
 * (NULL switches capture off); adt_session_capture_record returns forward i's offsets.  Not
 * used by the batched cycle. */
typedef struct {
  float* resid;
  size_t resid_elems;
  void* xin;
  size_t xin_bytes;
  int32_t* meta;
  size_t meta_elems;
} adt_capture;
typedef struct {
  int32_t draft;                /* 0 target forward, 1 draft-head forward */
  int32_t nodes, rows;          /* tree or prompt nodes; rows = nodes x branches */
  int32_t kv_prefix, slot0, n_tail;
  int32_t snapshots;            /* residual snapshots written (2 n_layers + 1, or 3) */
  int64_t resid_off;            /* first float of this forward in resid */
  int64_t xin_off;              /* first byte in xin (draft forwards) */
  int64_t meta_off;             /* first int32 in meta */
} adt_capture_rec;
adt_status adt_session_set_capture(adt_session* s, const adt_capture* cap);
int32_t adt_session_capture_count(const adt_session* s);
adt_status adt_session_capture_record(const adt_session* s, int32_t i, adt_capture_rec* rec);

/* a1-a3: the draft head's catch-up rows then d_hat - 1 frontier forwards (Sec. 4.2, Eq. 4),
 * top-k children scored by summed log-probability (Eq. 3), frontier select, top-N rerank and
 * the BFS tree arrays + masks of the session's current tree.  n_nodes_out [host] gets the
 * tree size (root included).
 * Sessions in ADT_ACCEPT_MSS mode draw the children instead (Sec. 3.1 read literally): every
 * expanded node takes accept.children i.i.d. draws from q (the acceptance's integer weights
 * of its draft row), child j of tree node u at r = floor(U W_q / 2^64), U at counter (step,
 * u, j, 2), the id the smallest with prefix weight > r.  All drawn children stay in the tree
 * (no rerank: the siblings must remain an i.i.d. sample of q); each later layer expands the
 * k_hat best nodes of the previous one by path confidence, as many as keep the tree within
 * n_budget draft nodes; nodes are in creation order (siblings in draw order). */
adt_status adt_tree_expand(adt_session* s, int32_t d_hat, int32_t k_hat, int32_t n_budget, int32_t* n_nodes_out,
                           void* stream);
/* Replaces the session's current tree with a caller tree: parent/token [host] n ids, BFS
 * ordered (parent[i] < i, parent[0] = -1), token[0] = the last committed token, 1 <= n <=
 * ADT_MAX_NODES.  Called right after adt_tree_expand it keeps that expansion's draft-cache
 * state (the root's draft row stays valid); otherwise the draft cache is left as it was.
 * Synchronises.  ADT_E_ARG on a malformed tree, ADT_E_CAPACITY past the cache capacity. */
adt_status adt_session_set_tree(adt_session* s, const int32_t* parent, const int32_t* token, int32_t n,
                                void* stream);
/* b1-b3: the target forward of the session's current tree at the committed length L:
 * K/V of node i go to slot L + i, logits and features into the session buffers. */
adt_status adt_verify_forward(adt_session* s, void* stream);
/* c + d1 for the session: accept on the last verify, compact both caches, commit.  Synchronises. */
adt_status adt_session_accept_commit(adt_session* s, int32_t d_hat, int32_t k_hat, adt_step_out* out, void* stream);
/* One full cycle: a0 + a1-a3 + b + c + d1.  Synchronises once (the accepted path). */
adt_status adt_step(adt_session* s, adt_step_out* out, void* stream);

/* ------------------------------------------------------------------ batched cycle
 * Several images decoded together (Sec. 3.1 verification applied to a batch of trees): each
 * session schedules and drafts its own tree as in adt_step, then ONE target forward verifies
 * every tree, its rows packed one tree after another (M = sum of tree sizes; the projections
 * run on the MFMA-tiled batched GEMM reading the packed weights, attention takes each tree
 * against its own cache), and each session accepts and commits from its rows.  Results equal
 * adt_step on each session up to floating-point order.
 * sessions: [host] B prefilled sessions of one bf16 model, unguided, equal s_cap, whose
 *   target caches are equally spaced: k_cache of session b = k_cache of session 0 +
 *   b * stride (the same stride for v_cache, at least n_layers*n_heads*s_cap*head_dim
 *   elements), i.e. one [B][n_layers][n_heads][s_cap][head_dim] allocation.  The batch
 *   keeps the pointers; the sessions must outlive it and not be stepped on their own while
 *   it is used.
 * workspace: device memory of adt_batch_workspace_size() bytes, owned by the caller.
 * adt_batch_step writes outs[b] for every session (done sessions report done = 1 and are
 * not verified).  ADT_E_ARG / ADT_E_SHAPE when the sessions do not satisfy the above. */
typedef struct adt_batch_s adt_batch;
size_t adt_batch_workspace_size(adt_session* const* sessions, int32_t B);
adt_status adt_batch_create(adt_session* const* sessions, int32_t B, void* workspace, size_t workspace_bytes,
                            adt_batch** out);
void adt_batch_destroy(adt_batch* b);
adt_status adt_batch_step(adt_batch* b, adt_step_out* outs, void* stream);

/* ------------------------------------------------------------------ profiling
 * Optional timing of the session's kernels by class, with HIP events recorded on the
 * caller's stream around each launch (adds a little host overhead while enabled).  Read
 * values accumulate until reset: launches, summed kernel milliseconds, algorithmic bytes
 * (what the method must move: weights once, inputs and outputs; prefix K/V once for
 * attention) and flops. */
#define ADT_PROF_GEMM 0     /* dense projections (bf16 MFMA or fp32) */
#define ADT_PROF_ATTN 1     /* tree attention + split merge */
#define ADT_PROF_COMPACT 2  /* KV compaction */
#define ADT_PROF_ROWS 3     /* finish of a residual projection: K-range sums, residual add, RMSNorm */
#define ADT_PROF_CLASSES 4
adt_status adt_profile_enable(int32_t on);
/* Probes of what the device sustains, to report beside the nominal peaks (HBM 8 TB/s, dense
 * bf16 MFMA 2.5 PFLOP/s).  adt_probe_hbm_read streams `bytes` (a multiple of 16, 16-byte
 * aligned device buffer) with 16-byte nontemporal loads and folds them into `sink`; adt_probe_mfma runs
 * `iters` rounds of back-to-back 32x32x16 bf16 MFMAs on register operands (no memory traffic)
 * and reports the flops it launched in *flops [host].  sink: device scratch of at least
 * adt_probe_sink_bytes() bytes.  Asynchronous on `stream`; the caller times them. */
size_t adt_probe_sink_bytes(void);
adt_status adt_probe_hbm_read(const void* buf, size_t bytes, void* sink, size_t sink_bytes, void* stream);
adt_status adt_probe_mfma(int32_t iters, void* sink, size_t sink_bytes, double* flops, void* stream);
/* The integer weights the sampling kernels (exact, relaxed and stochastic-children modes,
 * Sec. 3.1 Eq. 1) give to float32 exponents d = z - max z: w[i] = rint(exp(d[i]) * 2^32)
 * with exp evaluated by a fixed sequence of IEEE double operations (y = d log2 e, k = floor y,
 * f = y - k, 2^f by Horner's rule over the doubles nearest ln(2)^j / j!, j = 13..0, no fused
 * multiply-add), 0 for d < -40 or NaN.  Exposed so that a reference of the same definition
 * can be compared with the device's integers.  d, w: [n] device arrays; asynchronous on
 * `stream`; ADT_E_ARG for null pointers or n < 0. */
adt_status adt_probe_sample_weights(const float* d, int64_t n, uint64_t* w, void* stream);
adt_status adt_profile_read(int32_t cls, int64_t* launches, double* ms, double* bytes, double* flops, int32_t reset);

#ifdef __cplusplus
}
#endif
#endif /* ADT_H_ */
