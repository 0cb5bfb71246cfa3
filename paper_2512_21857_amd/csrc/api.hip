// C ABI of the ADT-Tree hot path: argument checks, the host-side schedule, workspace
// layout and the orchestration of one draft-then-verify cycle.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <vector>

#include "launch.h"

namespace adt {

static thread_local char g_err[512];

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

#define TRY(x)                \
  do {                        \
    adt_status e__ = (x);     \
    if (e__ != ADT_OK) return e__; \
  } while (0)

static inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct Bump {
  char* base;
  size_t off = 0;
  template <typename T>
  T* take(size_t count) {
    off = align_up(off, 256);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

// ---------------------------------------------------------------------------- profiling
// Optional per-kernel-class timing: HIP events recorded on the caller's stream around each
// launch of a class, read back at the next synchronisation of a cycle.  Off by default.
struct ProfRec {
  int cls;
  int e0, e1;
  double bytes, flops;
};
struct Profiler {
  bool on = false;
  std::vector<hipEvent_t> ev;
  int next = 0;
  std::vector<ProfRec> pending;
  double ms[ADT_PROF_CLASSES] = {};
  double bytes[ADT_PROF_CLASSES] = {};
  double flops[ADT_PROF_CLASSES] = {};
  int64_t launches[ADT_PROF_CLASSES] = {};
};
static Profiler g_prof;

static int prof_begin(hipStream_t st) {
  if (!g_prof.on || g_prof.next + 2 > (int)g_prof.ev.size()) return -1;
  const int e = g_prof.next;
  g_prof.next += 2;
  (void)hipEventRecord(g_prof.ev[e], st);
  return e;
}
static void prof_end(int e, int cls, double bytes, double flops, hipStream_t st) {
  if (e < 0) return;
  (void)hipEventRecord(g_prof.ev[e + 1], st);
  g_prof.pending.push_back({cls, e, e + 1, bytes, flops});
}
// An event pair for a launch that records its own start and end (hipExtLaunchKernelGGL).
static int prof_pair() {
  if (!g_prof.on || g_prof.next + 2 > (int)g_prof.ev.size()) return -1;
  const int e = g_prof.next;
  g_prof.next += 2;
  return e;
}
static void prof_done(int e, int cls, double bytes, double flops) {
  if (e >= 0) g_prof.pending.push_back({cls, e, e + 1, bytes, flops});
}
static void prof_collect() {
  if (!g_prof.on) return;
  for (const ProfRec& r : g_prof.pending) {
    float ms = 0.f;
    if (hipEventSynchronize(g_prof.ev[r.e1]) == hipSuccess && hipEventElapsedTime(&ms, g_prof.ev[r.e0], g_prof.ev[r.e1]) == hipSuccess) {
      g_prof.ms[r.cls] += ms;
      g_prof.bytes[r.cls] += r.bytes;
      g_prof.flops[r.cls] += r.flops;
      g_prof.launches[r.cls] += 1;
    }
  }
  g_prof.pending.clear();
  g_prof.next = 0;
}

}  // namespace adt

using namespace adt;

static constexpr int R = ADT_MAX_NODES;

extern "C" adt_status adt_profile_enable(int32_t on) {
  if (on && g_prof.ev.empty()) {
    g_prof.ev.resize(16384);
    for (auto& e : g_prof.ev) ADT_HIP(hipEventCreate(&e));
  }
  g_prof.on = on != 0;
  return ADT_OK;
}

extern "C" adt_status adt_profile_read(int32_t cls, int64_t* launches, double* ms, double* bytes, double* flops,
                                       int32_t reset) {
  ADT_CHECK_ARG(cls >= 0 && cls < ADT_PROF_CLASSES, ADT_E_ARG, "profile_read: class %d", cls);
  prof_collect();
  if (launches) *launches = g_prof.launches[cls];
  if (ms) *ms = g_prof.ms[cls];
  if (bytes) *bytes = g_prof.bytes[cls];
  if (flops) *flops = g_prof.flops[cls];
  if (reset) {
    g_prof.launches[cls] = 0;
    g_prof.ms[cls] = g_prof.bytes[cls] = g_prof.flops[cls] = 0.0;
  }
  return ADT_OK;
}

extern "C" int32_t adt_version(void) { return 1; }

extern "C" size_t adt_last_error(char* buf, size_t cap) {
  const size_t n = strlen(g_err);
  if (buf && cap) {
    const size_t c = n < cap - 1 ? n : cap - 1;
    memcpy(buf, g_err, c);
    buf[c] = 0;
  }
  return n;
}

static bool valid_dtype(int32_t dt) { return dt == ADT_F32 || dt == ADT_BF16; }
static size_t esize(int32_t dt) { return dt == ADT_BF16 ? 2 : 4; }

// ============================================================================ standalone calls
extern "C" size_t adt_tree_attn_workspace_size(int32_t B, int32_t H, int32_t Dh, int32_t nq_max, int32_t kv_cap) {
  return tree_attn_ws_bytes(B, H, Dh, nq_max, kv_cap, ADT_BF16);
}

static adt_status check_tree_attn(const void* q, const void* k_cache, const void* v_cache, int64_t stride_b,
                                  int64_t stride_h, const int32_t* kv_len, const int32_t* n_q, const int32_t* n_tail,
                                  const uint64_t* anc_mask, int32_t B, int32_t H, int32_t Dh, int32_t nq_max,
                                  int32_t kv_cap, float scale, int32_t dtype, void* out) {
  ADT_CHECK_ARG(q && k_cache && v_cache && kv_len && n_q && n_tail && anc_mask && out, ADT_E_ARG,
                "tree_attn: null pointer");
  ADT_CHECK_ARG(valid_dtype(dtype), ADT_E_ARG, "tree_attn: bad dtype %d", dtype);
  ADT_CHECK_ARG(B >= 1 && H >= 1 && kv_cap >= 1, ADT_E_ARG, "tree_attn: B=%d H=%d kv_cap=%d", B, H, kv_cap);
  ADT_CHECK_ARG(Dh == 64 || Dh == 128, ADT_E_SHAPE, "tree_attn: head_dim %d not in {64, 128}", Dh);
  ADT_CHECK_ARG(nq_max >= 1 && nq_max <= ADT_MAX_NODES, ADT_E_CAPACITY, "tree_attn: nq_max %d", nq_max);
  ADT_CHECK_ARG(stride_h >= (int64_t)kv_cap * Dh, ADT_E_SHAPE, "tree_attn: stride_h %lld < kv_cap*Dh",
                (long long)stride_h);
  ADT_CHECK_ARG(B == 1 || stride_b >= (int64_t)H * stride_h, ADT_E_SHAPE, "tree_attn: stride_b too small");
  ADT_CHECK_ARG(std::isfinite(scale) && scale > 0.f, ADT_E_ARG, "tree_attn: scale");
  return ADT_OK;
}

extern "C" adt_status adt_tree_attn(const void* q, const void* k_cache, const void* v_cache, int64_t stride_b,
                                    int64_t stride_h, const int32_t* kv_len, const int32_t* n_q, const int32_t* n_tail,
                                    const uint64_t* anc_mask, int32_t B, int32_t H, int32_t Dh, int32_t nq_max,
                                    int32_t kv_cap, float scale, int32_t dtype, void* out, void* workspace,
                                    size_t workspace_bytes, void* stream) {
  TRY(check_tree_attn(q, k_cache, v_cache, stride_b, stride_h, kv_len, n_q, n_tail, anc_mask, B, H, Dh, nq_max, kv_cap,
                      scale, dtype, out));
  return launch_tree_attn(q, k_cache, v_cache, stride_b, stride_h, kv_len, n_q, n_tail, anc_mask,
                          AttnRows{nq_max, 1, nq_max}, B, H, Dh, nq_max, kv_cap, scale, dtype, out, workspace,
                          workspace_bytes, (hipStream_t)stream);
}

// Scratch of adt_tree_attn_noalloc: the key-split partials of a launch live in this
// file-scope device array instead of a caller workspace.  Every device the library runs on
// holds its own copy until the process ends; host code reaches it only through the address
// hipGetSymbolAddress returns with that device current (kept per device below), never through
// the array's name, which in host code is a stand-in and not a device address.
constexpr size_t ATTN_SCRATCH_BYTES = (size_t)16 << 20;
constexpr int SCRATCH_MAX_DEVICES = 64;
static __device__ __align__(256) char scratch[ATTN_SCRATCH_BYTES];
static std::mutex g_scratch_mu;
static void* g_scratch_dev[SCRATCH_MAX_DEVICES];

static adt_status scratch_on_current_device(void** out) {
  int dev = -1;
  ADT_HIP(hipGetDevice(&dev));
  ADT_CHECK_ARG(dev >= 0 && dev < SCRATCH_MAX_DEVICES, ADT_E_UNSUPPORTED, "tree_attn_noalloc: device %d", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    ADT_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    ADT_CHECK_ARG(p != nullptr, ADT_E_HIP, "tree_attn_noalloc: no address for the scratch array");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return ADT_OK;
}

extern "C" adt_status adt_tree_attn_noalloc(const void* q, const void* k_cache, const void* v_cache, int64_t stride_b,
                                            int64_t stride_h, const int32_t* kv_len, const int32_t* n_q,
                                            const int32_t* n_tail, const uint64_t* anc_mask, int32_t B, int32_t H,
                                            int32_t Dh, int32_t nq_max, int32_t kv_cap, float scale, int32_t dtype,
                                            void* out, void* stream) {
  TRY(check_tree_attn(q, k_cache, v_cache, stride_b, stride_h, kv_len, n_q, n_tail, anc_mask, B, H, Dh, nq_max, kv_cap,
                      scale, dtype, out));
  const size_t need = tree_attn_ws_need(B, H, Dh, nq_max, kv_cap, dtype);
  ADT_CHECK_ARG(need <= ATTN_SCRATCH_BYTES, ADT_E_CAPACITY,
                "tree_attn_noalloc: the key-split partials need %zu bytes, the scratch holds %zu", need,
                ATTN_SCRATCH_BYTES);
  void* ws = nullptr;
  TRY(scratch_on_current_device(&ws));
  return launch_tree_attn(q, k_cache, v_cache, stride_b, stride_h, kv_len, n_q, n_tail, anc_mask,
                          AttnRows{nq_max, 1, nq_max}, B, H, Dh, nq_max, kv_cap, scale, dtype, out, ws,
                          ATTN_SCRATCH_BYTES, (hipStream_t)stream);
}

extern "C" adt_status adt_tree_masks(const int32_t* parent, const int32_t* n_nodes, int32_t B, int32_t n_max,
                                     uint64_t* mask, int32_t* depth, void* stream) {
  ADT_CHECK_ARG(parent && n_nodes && mask && B >= 1, ADT_E_ARG, "tree_masks: bad arguments");
  ADT_CHECK_ARG(n_max >= 1 && n_max <= ADT_MAX_NODES, ADT_E_CAPACITY, "tree_masks: n_max %d", n_max);
  return launch_tree_masks(parent, n_nodes, B, n_max, mask, depth, (hipStream_t)stream);
}

extern "C" adt_status adt_kv_compact(void* k_cache, void* v_cache, int32_t B, int32_t slices, int32_t Dh,
                                     int64_t stride_b, int64_t stride_slice, const int32_t* kv_len, const int32_t* path,
                                     int32_t path_stride, const int32_t* n_acc, int32_t a_max, int32_t dtype,
                                     void* stream) {
  ADT_CHECK_ARG(k_cache && v_cache && kv_len && path && n_acc, ADT_E_ARG, "kv_compact: null pointer");
  ADT_CHECK_ARG(valid_dtype(dtype) && B >= 1 && slices >= 1 && Dh >= 1, ADT_E_ARG, "kv_compact: bad sizes");
  ADT_CHECK_ARG(a_max >= 0 && a_max < ADT_MAX_NODES && path_stride >= a_max + 1, ADT_E_CAPACITY,
                "kv_compact: a_max %d path_stride %d", a_max, path_stride);
  if (a_max == 0) return ADT_OK;
  return launch_kv_compact(k_cache, v_cache, B, slices, Dh, stride_b, stride_slice, kv_len, 1, path, path_stride, n_acc,
                           1, a_max, dtype, (hipStream_t)stream);
}

extern "C" size_t adt_accept_workspace_size(int32_t V) {
  return align_up(accept_ws_bytes(V), 256) + (size_t)R * 16 * 8 + (size_t)R * 4 + align_up(row_topk_ws_bytes(R, 1), 256) +
         1024;
}

static adt_status accept_impl(const float* logits, int64_t ld, int V, const int32_t* parent, const int32_t* token,
                              const int32_t* allowed, const int32_t* n_nodes, int n_max, const adt_accept_cfg& cfg,
                              uint64_t step, int32_t* path, int32_t* n_acc, int32_t* bonus, void* ws, size_t ws_bytes,
                              hipStream_t st) {
  ADT_CHECK_ARG(ws && ws_bytes >= adt_accept_workspace_size(V), ADT_E_CAPACITY, "accept: workspace too small");
  Bump b{(char*)ws};
  int32_t* top_id = b.take<int32_t>((size_t)R * 16);
  float* top_val = b.take<float>((size_t)R * 16);
  float* lse = b.take<float>(R);
  void* rest = b.take<char>(accept_ws_bytes(V));
  const size_t tk_bytes = row_topk_ws_bytes(R, 1);
  void* tk = b.take<char>(tk_bytes);
  if (cfg.mode == ADT_ACCEPT_GREEDY) {
    adt_status e = launch_row_topk(logits, ld, V, allowed, n_max, 1, 1, top_id, top_val, lse, tk, tk_bytes, st);
    if (e) return e;
    return launch_accept_greedy(top_id, 1, parent, token, n_nodes, n_max, path, n_acc, bonus, st);
  }
  if (cfg.mode == ADT_ACCEPT_MSS)
    return launch_accept_mss(logits, ld, V, parent, token, allowed, n_nodes, n_max, cfg, step, path, n_acc, bonus, rest,
                             accept_ws_bytes(V), st);
  return launch_accept_sample(logits, ld, V, parent, token, allowed, n_nodes, n_max, cfg, step, path, n_acc, bonus,
                              rest, accept_ws_bytes(V), st);
}

static adt_status check_accept_cfg(const adt_accept_cfg* cfg) {
  ADT_CHECK_ARG(cfg != nullptr, ADT_E_ARG, "accept: null cfg");
  ADT_CHECK_ARG(cfg->mode >= ADT_ACCEPT_GREEDY && cfg->mode <= ADT_ACCEPT_MSS, ADT_E_ARG, "accept: mode %d",
                cfg->mode);
  if (cfg->mode != ADT_ACCEPT_GREEDY) {
    ADT_CHECK_ARG(cfg->temperature > 0.f && std::isfinite(cfg->temperature), ADT_E_ARG, "accept: temperature");
    ADT_CHECK_ARG(cfg->top_k >= 0 && cfg->top_k <= 4096, ADT_E_UNSUPPORTED, "accept: top_k %d", cfg->top_k);
  }
  if (cfg->mode == ADT_ACCEPT_RELAXED) {
    ADT_CHECK_ARG(cfg->delta >= 0.f && cfg->delta < 1.f, ADT_E_ARG, "accept: delta");
    ADT_CHECK_ARG(cfg->knn_k >= 1 && (cfg->knn_k == 1 || (cfg->knn && cfg->knn_stride >= cfg->knn_k)), ADT_E_ARG,
                  "accept: knn table");
  }
  return ADT_OK;
}

extern "C" adt_status adt_verify_accept(const float* logits, int64_t ld, int32_t V, const int32_t* parent,
                                        const int32_t* token, const int32_t* allowed, const int32_t* n_nodes,
                                        int32_t n_max, const adt_accept_cfg* cfg, uint64_t step, int32_t* path,
                                        int32_t* n_acc, int32_t* bonus, void* workspace, size_t workspace_bytes,
                                        void* stream) {
  ADT_CHECK_ARG(logits && parent && token && allowed && n_nodes && path && n_acc && bonus, ADT_E_ARG,
                "verify_accept: null pointer");
  ADT_CHECK_ARG(V >= 1 && ld >= V, ADT_E_ARG, "verify_accept: V %d ld %lld", V, (long long)ld);
  ADT_CHECK_ARG(n_max >= 1 && n_max <= ADT_MAX_NODES, ADT_E_CAPACITY, "verify_accept: n_max %d", n_max);
  adt_status e = check_accept_cfg(cfg);
  if (e) return e;
  ADT_CHECK_ARG(cfg->mode != ADT_ACCEPT_MSS || (cfg->q_logits && cfg->q_row && cfg->q_ld >= V && cfg->q_rows >= 1),
                ADT_E_ARG, "verify_accept: MSS needs q_logits, q_row, q_ld >= V and q_rows >= 1");
  return accept_impl(logits, ld, V, parent, token, allowed, n_nodes, n_max, *cfg, step, path, n_acc, bonus, workspace,
                     workspace_bytes, (hipStream_t)stream);
}

extern "C" size_t adt_codebook_knn_workspace_size(int32_t n) { return n > 0 ? knn_ws_bytes(n) : 0; }

extern "C" adt_status adt_codebook_knn(const float* codebook, int32_t n, int32_t dim, int32_t k, int32_t* out,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  ADT_CHECK_ARG(codebook && out && n >= 1 && dim >= 1, ADT_E_ARG, "codebook_knn: bad arguments");
  return launch_codebook_knn(codebook, n, dim, k, out, workspace, workspace_bytes, (hipStream_t)stream);
}

extern "C" adt_status adt_gemm_bf16(const void* X, int64_t ldx, const void* W, int64_t ldw, int32_t M, int32_t N,
                                    int32_t K, float* C, int64_t ldc, void* stream) {
  return launch_gemm_nt(X, ldx, W, ldw, M, N, K, C, ldc, (hipStream_t)stream);
}

extern "C" size_t adt_gemm_bf16_packed_workspace_size(int32_t M, int32_t N, int32_t K) {
  if (M < 1 || N < 256 || N % 256 != 0 || K < 64) return 0;
  return gemm_nt_part_elems(M, N, K) * sizeof(float);
}

extern "C" adt_status adt_gemm_bf16_packed(const void* X, int64_t ldx, const void* Wp, int32_t M, int32_t N, int32_t K,
                                           float* C, int64_t ldc, void* workspace, size_t workspace_bytes,
                                           void* stream) {
  return launch_gemm_nt(X, ldx, Wp, K, M, N, K, C, ldc, (hipStream_t)stream, nullptr, nullptr, true, (float*)workspace,
                        workspace ? workspace_bytes / sizeof(float) : 0);
}

extern "C" size_t adt_packed_bytes(int32_t total_rows, int32_t K, int32_t dtype) {
  return packed_bytes(total_rows, K, dtype);
}

extern "C" adt_status adt_pack_weight(const void* const* srcs, const int32_t* rows, int32_t n_src, int32_t K,
                                      int32_t mode, int32_t group, int32_t dtype, void* dst, void* stream) {
  ADT_CHECK_ARG(valid_dtype(dtype) && K >= 1, ADT_E_ARG, "pack: dtype/K");
  return launch_pack(srcs, rows, n_src, K, mode, group, dtype, dst, (hipStream_t)stream);
}

static adt_status check_sched_cfg(const adt_sched_cfg* c) {
  ADT_CHECK_ARG(c->d_lo >= 1 && c->d_lo <= c->d_hi && c->k_lo >= 1 && c->k_lo <= c->k_hi, ADT_E_ARG,
                "schedule: bad bounds");
  ADT_CHECK_ARG(c->init_mode >= ADT_INIT_HORIZONTAL && c->init_mode <= ADT_INIT_TOKENFLOCK, ADT_E_ARG,
                "schedule: init_mode %d", c->init_mode);
  ADT_CHECK_ARG(c->grid_w >= 1 || (c->init_mode != ADT_INIT_VERTICAL && c->init_mode != ADT_INIT_TOKENFLOCK),
                ADT_E_ARG, "schedule: grid_w %d", c->grid_w);
  ADT_CHECK_ARG(c->flock_delta >= 1 || c->init_mode != ADT_INIT_TOKENFLOCK, ADT_E_ARG, "schedule: flock_delta %d",
                c->flock_delta);
  ADT_CHECK_ARG(c->fix_d >= 0 && c->fix_k >= 0, ADT_E_ARG, "schedule: fixed bases");
  ADT_CHECK_ARG(c->k_clamp == ADT_KCLAMP_ALWAYS || (c->k_clamp == ADT_KCLAMP_DEEP && c->d_lo == 1), ADT_E_ARG,
                "schedule: k_clamp %d (the deep-only rule needs d_lo = 1)", c->k_clamp);
  return ADT_OK;
}

extern "C" adt_status adt_schedule_init(const adt_sched_cfg* c, int32_t cell, int32_t n_cells, const int32_t* rec_d,
                                        const int32_t* rec_k, const int32_t* has_rec, int32_t* have_init,
                                        int32_t* d_init, int32_t* k_init) {
  ADT_CHECK_ARG(c && rec_d && rec_k && has_rec && have_init && d_init && k_init, ADT_E_ARG,
                "schedule_init: null pointer");
  ADT_CHECK_ARG(cell >= 0 && cell < n_cells, ADT_E_ARG, "schedule_init: cell %d of %d", cell, n_cells);
  TRY(check_sched_cfg(c));
  int have = 0, d = 0, k = 0;
  auto take = [&](int g) {
    if (g >= 0 && g < cell && has_rec[g]) {
      have = 1;
      d = rec_d[g];
      k = rec_k[g];
    }
  };
  switch (c->init_mode) {
    case ADT_INIT_HORIZONTAL:
      take(cell - 1);
      break;
    case ADT_INIT_VERTICAL:
      take(cell - c->grid_w);
      if (!have) take(cell - 1);
      break;
    case ADT_INIT_RANDOM: {
      // two 64-bit draws from one Philox block; floor(U * span / 2^64) as a 128-bit product
      uint32_t x[4] = {(uint32_t)cell, 0u, 0u, 1u};
      philox4x32_10(x, (uint32_t)c->seed, (uint32_t)(c->seed >> 32));
      const uint64_t u0 = ((uint64_t)x[1] << 32) | x[0], u1 = ((uint64_t)x[3] << 32) | x[2];
      const uint64_t sd = (uint64_t)(c->d_hi - c->d_lo + 1), sk = (uint64_t)(c->k_hi - c->k_lo + 1);
      d = c->d_lo + (int)(((unsigned __int128)u0 * sd) >> 64);
      k = c->k_lo + (int)(((unsigned __int128)u1 * sk) >> 64);
      have = 1;
      break;
    }
    case ADT_INIT_TOKENFLOCK: {
      // Eqs. 6-8: only rows y - delta .. y and columns x - delta .. x + delta can lie within
      // the radius; the 1/delta of the weights cancels in the normalisation.
      const int W = c->grid_w, R2 = c->flock_delta * c->flock_delta;
      const int y = cell / W, x = cell % W;
      int64_t sw = 0, swd = 0, swk = 0;
      for (int dy = 0; dy <= c->flock_delta && dy <= y; ++dy)
        for (int dx = -c->flock_delta; dx <= c->flock_delta; ++dx) {
          const int xx = x + dx;
          if (xx < 0 || xx >= W || dx * dx + dy * dy > R2) continue;
          const int g = (y - dy) * W + xx;
          if (g >= cell || !has_rec[g]) continue;
          const int64_t w = c->flock_delta + 1 - dy;
          sw += w;
          swd += w * rec_d[g];
          swk += w * rec_k[g];
        }
      if (sw > 0) {
        have = 1;
        d = (int)((2 * swd + sw) / (2 * sw));   // round half up of swd / sw (all terms >= 0)
        k = (int)((2 * swk + sw) / (2 * sw));
      }
      break;
    }
  }
  if (c->fix_d > 0 || c->fix_k > 0) {
    if (!have) {
      d = c->d0;
      k = c->k0;
      have = 1;
    }
    if (c->fix_d > 0) d = c->fix_d;
    if (c->fix_k > 0) k = c->fix_k;
  }
  *have_init = have;
  *d_init = have ? d : 0;
  *k_init = have ? k : 0;
  return ADT_OK;
}

extern "C" adt_status adt_schedule_next(const adt_sched_cfg* c, int32_t have_left, int32_t d_left, int32_t k_left,
                                        int32_t have_prev, int32_t a_prev, int32_t d_prev, int32_t remaining,
                                        int32_t* d_hat, int32_t* k_hat) {
  ADT_CHECK_ARG(c && d_hat && k_hat, ADT_E_ARG, "schedule: null pointer");
  TRY(check_sched_cfg(c));
  ADT_CHECK_ARG(remaining >= 1, ADT_E_ARG, "schedule: nothing remains");
  int d, k;
  if (!have_left) {
    d = c->d0;
    k = c->k0;
  } else {
    d = d_left;
    k = k_left;
    if (have_prev && d_prev > 0) {
      // Eq. 2: alpha = a / d compared with beta exactly as a >= beta * d.
      if ((double)a_prev >= (double)c->beta * (double)d_prev) {
        d += c->l_d;
        k -= c->l_k;
      } else {
        d -= c->l_d;
        k += c->l_k;
      }
    }
  }
  if (c->k_clamp == ADT_KCLAMP_DEEP && d <= 1)
    k = std::max(1, std::min(ADT_MAX_WIDTH, k));
  else
    k = std::max(c->k_lo, std::min(c->k_hi, k));
  d = std::max(c->d_lo, std::min(c->d_hi, d));
  d = std::min(d, remaining - 1);
  *d_hat = d;
  *k_hat = k;
  return ADT_OK;
}

// ============================================================================ model
struct adt_model_s {
  adt_model_desc d;
  std::vector<const void*> qkv, o, gu, down;
};

extern "C" adt_status adt_model_create(const adt_model_desc* d, adt_model** out) {
  ADT_CHECK_ARG(d && out, ADT_E_ARG, "model_create: null pointer");
  ADT_CHECK_ARG(valid_dtype(d->dtype), ADT_E_ARG, "model_create: dtype");
  ADT_CHECK_ARG(d->n_layers >= 1 && d->n_heads >= 1 && d->ffn >= 1 && d->vocab >= 1, ADT_E_ARG, "model_create: dims");
  ADT_CHECK_ARG(d->head_dim == 64 || d->head_dim == 128, ADT_E_SHAPE, "model_create: head_dim %d", d->head_dim);
  ADT_CHECK_ARG(d->d_model == d->n_heads * d->head_dim, ADT_E_SHAPE, "model_create: d_model != heads*head_dim");
  if (d->dtype == ADT_BF16)
    ADT_CHECK_ARG(d->d_model % 32 == 0 && d->ffn % 32 == 0 && d->vocab % 16 == 0, ADT_E_SHAPE,
                  "model_create: bf16 needs d_model, ffn multiples of 32 and vocab of 16");
  ADT_CHECK_ARG(d->embed && d->lm_head && d->draft_fc && d->w_qkv && d->w_o && d->w_gu && d->w_down, ADT_E_ARG,
                "model_create: missing weights");
  adt_model_s* m = new (std::nothrow) adt_model_s();
  ADT_CHECK_ARG(m != nullptr, ADT_E_ARG, "model_create: out of host memory");
  m->d = *d;
  for (int l = 0; l <= d->n_layers; ++l) {
    if (!d->w_qkv[l] || !d->w_o[l] || !d->w_gu[l] || !d->w_down[l]) {
      delete m;
      set_error("model_create: layer %d weight missing", l);
      return ADT_E_ARG;
    }
    m->qkv.push_back(d->w_qkv[l]);
    m->o.push_back(d->w_o[l]);
    m->gu.push_back(d->w_gu[l]);
    m->down.push_back(d->w_down[l]);
  }
  m->d.w_qkv = m->d.w_o = m->d.w_gu = m->d.w_down = nullptr;
  *out = m;
  return ADT_OK;
}

extern "C" void adt_model_destroy(adt_model* m) { delete m; }

// ============================================================================ session
struct TreeBufs {
  int32_t *parent, *token, *depth, *pos, *allowed_rows, *n, *path, *nacc, *bonus;
  int32_t* qrow;   // draft-logit row that drew each node's children (stochastic children)
  float* score;
  uint64_t* mask;
};

struct adt_session_s {
  const adt_model_s* m;
  adt_session_desc d;
  int dt, Lr, dm, H, Dh, F, V, P, T;
  int C0;       // first draft-feature row of draft tree rows
  int DR;       // draft-feature rows
  int DLR;      // draft logits rows
  int KR;       // frontier rows capacity
  int C;        // pool capacity
  // guidance: nb = 2 branches (conditional, unconditional) interleaved node by node in every
  // forward's rows; caches of branch 1 sit tcache_sb / dcache_sb elements after branch 0
  int nb = 1;
  float gscale = 1.f;
  int64_t tcache_sb = 0, dcache_sb = 0;
  float* rawlog = nullptr;   // [R][V] per-branch verify logits (guided)
  float* draw = nullptr;     // [nb (1 + KR)][V] per-branch draft logits: root rows, then a level's rows
  // host state
  bool prefilled = false;
  bool expanded = false;   // the current tree came from adt_tree_expand (draft root row written)
  int L = 0, Ld = 0, step = 1, n_nodes = 0;
  std::vector<int32_t> tokens, allowed_h, poisson;
  // vocabulary columns [lm_lo, lm_hi) the bf16 LM head computes: the union of the image
  // cells' allowed ranges, widened to whole 16-row weight tiles (every consumer of the logits
  // reads a cell's allowed range only)
  int lm_lo = 0, lm_hi = 0;
  std::vector<int32_t> rec_d, rec_k, has_rec;
  bool have_prev = false;
  int a_prev = 0, d_prev = 0, prev_cell = 0;
  // device buffers
  float *h, *part, *logits, *dlogits;
  void *act, *xin, *q, *att, *sw, *feat, *cfeat, *dfeat;
  size_t part_elems;
  TreeBufs tr;
  int32_t* allowed_img;
  Pool pool;
  NextRows nx[2];
  int32_t *ctok, *cfsrc, *cpos, *idx;
  uint64_t* cmask;
  int32_t *top_id, *allowed_lvl, *scal;
  float2* rope;   // [s_cap][head_dim / 2] cos/sin table
  float *top_val, *lse;
  void* attn_ws;
  size_t attn_ws_bytes;
  void* topk_ws;          // per-chunk candidates of the expansions' top-k
  size_t topk_ws_bytes;
  void* acc_ws;
  size_t acc_ws_bytes;
  uint64_t* samp_w = nullptr;   // stochastic children: [KR][V] q weights of a level's rows
  // pinned host staging of an acceptance's readback: path [R], tokens [R], a, bonus
  int32_t* h_acc = nullptr;
  // layer-by-layer record (adt_session_set_capture): forwards run eagerly while it is set;
  // capt_cur indexes the record of the forward in progress (-1 outside a forward)
  bool capt_on = false;
  adt_capture capt{};
  std::vector<adt_capture_rec> capt_log;
  size_t capt_resid = 0, capt_xin = 0, capt_meta = 0;
  int capt_cur = -1;
  // HIP graphs of the forwards, keyed by shape; captured on a private stream, replayed on
  // the caller's stream.
  bool graphs = true;
  hipStream_t cap = nullptr;
  std::map<int64_t, hipGraphExec_t> gexec;
  ~adt_session_s() {
    for (auto& kv : gexec) (void)hipGraphExecDestroy(kv.second);
    if (cap) (void)hipStreamDestroy(cap);
    if (h_acc) (void)hipHostFree(h_acc);
  }
};

static void session_dims(adt_session_s* s, const adt_model_s* m, const adt_session_desc* d) {
  const adt_model_desc& md = m->d;
  s->m = m;
  s->d = *d;
  s->dt = md.dtype;
  s->Lr = md.n_layers;
  s->dm = md.d_model;
  s->H = md.n_heads;
  s->Dh = md.head_dim;
  s->F = md.ffn;
  s->V = md.vocab;
  s->P = d->prefix_len;
  s->T = d->n_image;
  s->nb = d->guided ? 2 : 1;
  s->gscale = d->guidance_scale;
  s->tcache_sb = (int64_t)md.n_layers * md.n_heads * d->s_cap * md.head_dim;
  s->dcache_sb = (int64_t)md.n_heads * d->s_cap * md.head_dim;
  const int dh = d->sched.d_hi, kh = d->sched.k_hi;
  s->C0 = dh + 2;
  s->DR = s->C0 + std::max(1, (dh - 1) * kh);
  s->DLR = 1 + std::max(0, (dh - 1) * kh);
  // a one-layer tree may be as wide as ADT_MAX_WIDTH under the deep-only width clamp
  const int kw = d->sched.k_clamp == ADT_KCLAMP_DEEP ? ADT_MAX_WIDTH : kh;
  s->KR = std::max(kh, 1);
  s->C = std::max(kw, kh + (dh - 1) * kh * kh);
  if (d->accept.mode == ADT_ACCEPT_MSS) s->C = std::max(s->C, R);   // every drawn child is kept
  // fp32 projections write [rows][N] products for the row kernels; bf16 residual projections
  // (O, down, draft FC) write up to GEMM_MAX_SPLITS K-range sums of [rows][d_model]
  size_t pe = (size_t)GEMM_MAX_SPLITS * R * s->dm;
  if (s->dt == ADT_F32)
    for (int n : {3 * s->dm, s->dm, 2 * s->F, s->V}) pe = std::max(pe, (size_t)R * n);
  s->part_elems = pe;
}

static size_t session_layout(adt_session_s* s, char* base) {
  Bump b{base};
  const size_t es = esize(s->dt);
  const int dm = s->dm;
  s->h = b.take<float>((size_t)R * dm);
  s->act = b.take<char>((size_t)R * dm * es);
  s->xin = b.take<char>((size_t)R * 2 * dm * es);
  s->q = b.take<char>((size_t)R * dm * es);
  s->att = b.take<char>((size_t)R * dm * es);
  s->sw = b.take<char>((size_t)R * s->F * es);
  s->feat = b.take<char>((size_t)R * dm * es);
  s->cfeat = b.take<char>((size_t)s->nb * s->C0 * dm * es);
  s->dfeat = b.take<char>((size_t)s->nb * s->DR * dm * es);
  s->part = b.take<float>(s->part_elems);
  s->logits = b.take<float>((size_t)R * s->V);
  s->dlogits = b.take<float>((size_t)s->DLR * s->V);
  if (s->nb > 1) {
    s->rawlog = b.take<float>((size_t)R * s->V);
    s->draw = b.take<float>((size_t)s->nb * (1 + s->KR) * s->V);
  }
  TreeBufs& t = s->tr;
  // path, tree tokens, accepted count and bonus are adjacent in the order of the host staging
  // (path [R], tokens [R], a, bonus), so one copy reads back an acceptance
  int32_t* acc = b.take<int32_t>(2 * R + 8);
  t.path = acc;
  t.token = acc + R;
  t.nacc = acc + 2 * R;
  t.bonus = acc + 2 * R + 1;
  t.parent = b.take<int32_t>(R);
  t.depth = b.take<int32_t>(R);
  t.pos = b.take<int32_t>(R);
  t.allowed_rows = b.take<int32_t>(2 * R);
  t.n = b.take<int32_t>(4);
  t.score = b.take<float>(R);
  t.mask = b.take<uint64_t>(2 * R);
  t.qrow = b.take<int32_t>(R);
  s->allowed_img = b.take<int32_t>((size_t)2 * s->T);
  s->pool.token = b.take<int32_t>(s->C);
  s->pool.score = b.take<float>(s->C);
  s->pool.depth = b.take<int32_t>(s->C);
  s->pool.parent = b.take<int32_t>(s->C);
  s->pool.drow = b.take<int32_t>(s->C);
  s->pool.qrow = b.take<int32_t>(s->C);
  s->pool.rmask = b.take<uint64_t>((size_t)2 * std::max(1, s->DR - s->C0));
  for (int i = 0; i < 2; ++i) {
    s->nx[i].tok = b.take<int32_t>(s->KR);
    s->nx[i].fsrc = b.take<int32_t>(s->KR);
    s->nx[i].pos = b.take<int32_t>(s->KR);
    s->nx[i].mask = b.take<uint64_t>(2 * s->KR);
    s->nx[i].frontier = b.take<int32_t>(s->KR);
  }
  s->ctok = b.take<int32_t>(2 * R);
  s->cfsrc = b.take<int32_t>(R);
  s->cpos = b.take<int32_t>(R);
  s->idx = b.take<int32_t>(R);
  s->cmask = b.take<uint64_t>(2 * R);
  s->top_id = b.take<int32_t>((size_t)R * 16);
  s->top_val = b.take<float>((size_t)R * 16);
  s->lse = b.take<float>(R);
  s->allowed_lvl = b.take<int32_t>(2 * R);
  s->scal = b.take<int32_t>(16);
  s->rope = b.take<float2>((size_t)s->d.s_cap * (s->Dh / 2));
  s->attn_ws_bytes = tree_attn_ws_bytes(s->nb, s->H, s->Dh, R / s->nb, s->d.s_cap, s->dt);
  s->attn_ws = b.take<char>(std::max<size_t>(s->attn_ws_bytes, 256));
  s->acc_ws_bytes = adt_accept_workspace_size(s->V);
  s->acc_ws = b.take<char>(s->acc_ws_bytes);
  s->topk_ws_bytes = row_topk_ws_bytes(R, 16);
  s->topk_ws = b.take<char>(s->topk_ws_bytes);
  if (s->d.accept.mode == ADT_ACCEPT_MSS) s->samp_w = b.take<uint64_t>((size_t)s->KR * s->V);
  return align_up(b.off, 256);
}

static adt_status check_session_desc(const adt_model* m, const adt_session_desc* d) {
  ADT_CHECK_ARG(m && d, ADT_E_ARG, "session: null pointer");
  ADT_CHECK_ARG(d->prefix_len >= 1 && d->prefix_len <= R, ADT_E_CAPACITY, "session: prefix_len %d not in [1,%d]",
                d->prefix_len, R);
  ADT_CHECK_ARG(d->n_image >= 1, ADT_E_ARG, "session: n_image");
  ADT_CHECK_ARG(d->s_cap >= d->prefix_len + d->n_image + R, ADT_E_CAPACITY, "session: s_cap %d too small", d->s_cap);
  ADT_CHECK_ARG(d->k_cache && d->v_cache && d->dk_cache && d->dv_cache && d->allowed, ADT_E_ARG,
                "session: caches / allowed table missing");
  const adt_sched_cfg& c = d->sched;
  TRY(check_sched_cfg(&c));
  ADT_CHECK_ARG(c.d_hi <= 30 && c.k_hi <= 16, ADT_E_UNSUPPORTED, "session: d_hi <= 30 and k_hi <= 16 supported");
  const int nb = d->guided ? 2 : 1;
  ADT_CHECK_ARG(d->guided == 0 || d->guided == 1, ADT_E_ARG, "session: guided %d", d->guided);
  ADT_CHECK_ARG(!d->guided || std::isfinite(d->guidance_scale), ADT_E_ARG, "session: guidance scale");
  ADT_CHECK_ARG(c.n_budget >= 1 && c.n_budget <= R / nb - 1, ADT_E_CAPACITY, "session: n_budget %d", c.n_budget);
  ADT_CHECK_ARG((c.d_hi - 1) * c.k_hi <= R, ADT_E_CAPACITY, "session: draft tree rows exceed %d", R);
  ADT_CHECK_ARG(c.k_hi + (c.d_hi - 1) * c.k_hi * c.k_hi <= EXPAND_MAX_POOL, ADT_E_CAPACITY,
                "session: candidate pool k_hi + (d_hi - 1) k_hi^2 = %d exceeds %d", c.k_hi + (c.d_hi - 1) * c.k_hi * c.k_hi,
                EXPAND_MAX_POOL);
  ADT_CHECK_ARG(c.alpha_source == ADT_ALPHA_REAL || (c.alpha_source == ADT_ALPHA_POISSON && d->poisson), ADT_E_ARG,
                "session: alpha source");
  ADT_CHECK_ARG(d->draft_table == nullptr || d->draft_table_rows >= 1, ADT_E_ARG, "session: draft table rows");
  for (int g = 0; g < d->n_image; ++g) {
    const int lo = d->allowed[2 * g], hi = d->allowed[2 * g + 1];
    ADT_CHECK_ARG(0 <= lo && lo < hi && hi <= m->d.vocab, ADT_E_ARG, "session: allowed range of cell %d", g);
  }
  TRY(check_accept_cfg(&d->accept));
  ADT_CHECK_ARG(d->accept.mode != ADT_ACCEPT_MSS ||
                    (d->accept.children >= 1 && d->accept.children <= 16 && d->accept.children <= c.n_budget),
                ADT_E_ARG, "session: MSS children %d (in [1, 16] and <= n_budget)", d->accept.children);
  return ADT_OK;
}

extern "C" size_t adt_session_workspace_size(const adt_model* m, const adt_session_desc* d) {
  if (check_session_desc(m, d)) return 0;
  adt_session_s s;
  session_dims(&s, m, d);
  return session_layout(&s, nullptr);
}

extern "C" adt_status adt_session_create(const adt_model* m, const adt_session_desc* d, adt_session** out) {
  adt_status e = check_session_desc(m, d);
  if (e) return e;
  ADT_CHECK_ARG(out != nullptr, ADT_E_ARG, "session_create: null out");
  adt_session_s* s = new (std::nothrow) adt_session_s();
  ADT_CHECK_ARG(s != nullptr, ADT_E_ARG, "session_create: out of host memory");
  session_dims(s, m, d);
  const size_t need = session_layout(s, nullptr);
  if (!d->workspace || d->workspace_bytes < need) {
    delete s;
    set_error("session_create: workspace %zu < %zu bytes", d->workspace_bytes, need);
    return ADT_E_CAPACITY;
  }
  session_layout(s, (char*)d->workspace);
  s->graphs = d->use_graphs != 0;
  s->allowed_h.assign(d->allowed, d->allowed + 2 * d->n_image);
  s->lm_lo = s->V;
  s->lm_hi = 0;
  for (int c = 0; c < d->n_image; ++c) {
    s->lm_lo = std::min(s->lm_lo, (int)s->allowed_h[2 * c]);
    s->lm_hi = std::max(s->lm_hi, (int)s->allowed_h[2 * c + 1]);
  }
  s->lm_lo = std::max(0, s->lm_lo / 16 * 16);
  s->lm_hi = std::min(s->V, (s->lm_hi + 15) / 16 * 16);
  if (s->dt != ADT_BF16 || s->lm_lo >= s->lm_hi) {
    s->lm_lo = 0;
    s->lm_hi = s->V;
  }
  if (d->poisson) s->poisson.assign(d->poisson, d->poisson + d->n_image);
  s->rec_d.assign(d->n_image, 0);
  s->rec_k.assign(d->n_image, 0);
  s->has_rec.assign(d->n_image, 0);
  s->d.allowed = nullptr;
  s->d.poisson = nullptr;
  // pinned host staging of every acceptance's readback, allocated once here (the cycle
  // itself allocates nothing)
  hipError_t he = hipHostMalloc((void**)&s->h_acc, sizeof(int32_t) * (2 * R + 2), hipHostMallocDefault);
  if (he == hipSuccess)
    he = hipMemcpy(s->allowed_img, s->allowed_h.data(), sizeof(int32_t) * 2 * s->T, hipMemcpyHostToDevice);
  if (he == hipSuccess && launch_rope_table(s->rope, s->d.s_cap, s->Dh, m->d.rope_theta, nullptr) == ADT_OK)
    he = hipDeviceSynchronize();
  if (he != hipSuccess) {
    delete s;
    set_error("session_create: %s", hipGetErrorString(he));
    return ADT_E_HIP;
  }
  *out = s;
  return ADT_OK;
}

extern "C" void adt_session_destroy(adt_session* s) { delete s; }

static SmallI32 small_of(const int32_t* v, int n) {
  SmallI32 s{};
  for (int i = 0; i < n && i < 32; ++i) s.v[i] = v[i];
  return s;
}

// Device scalars of a forward, one copy per guidance branch: scal[0..1] attention prefix
// length, [2..3] query rows, [4..5] tail rows; scal[6] first cache slot of the rows;
// scal[8..9] the committed length for compaction.
enum { SC_KV = 0, SC_NQ = 2, SC_TAIL = 4, SC_SLOT = 6, SC_CL = 8 };
static adt_status set_scalars(adt_session_s* s, int kv_len, int nq, int ntail, int slot0, hipStream_t st) {
  int32_t v[7] = {kv_len, kv_len, nq, nq, ntail, ntail, slot0};
  return launch_set_i32(s->scal, small_of(v, 7), 7, st);
}

// Runs body(stream) through a cached graph (captured on first use for this key).  Eager
// when graphs are off or the profiling hook is on (events cannot be recorded per kernel
// inside a replayed graph).
template <typename F>
static adt_status run_graph(adt_session_s* s, int64_t key, hipStream_t st, F&& body) {
  if (!s->graphs || g_prof.on || s->capt_on) return body(st);
  auto it = s->gexec.find(key);
  if (it == s->gexec.end()) {
    if (!s->cap) ADT_HIP(hipStreamCreateWithFlags(&s->cap, hipStreamNonBlocking));
    ADT_HIP(hipStreamBeginCapture(s->cap, hipStreamCaptureModeThreadLocal));
    const adt_status e = body(s->cap);
    hipGraph_t g = nullptr;
    const hipError_t he = hipStreamEndCapture(s->cap, &g);
    if (e != ADT_OK) {
      if (he == hipSuccess && g) (void)hipGraphDestroy(g);
      return e;
    }
    ADT_HIP(he);
    hipGraphExec_t ex = nullptr;
    const hipError_t ie = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    ADT_HIP(ie);
    it = s->gexec.emplace(key, ex).first;
  }
  ADT_HIP(hipGraphLaunch(it->second, st));
  return ADT_OK;
}

static int64_t gkey(int kind, int a, int b, int c) {
  return ((int64_t)kind << 48) | ((int64_t)a << 32) | ((int64_t)b << 16) | (int64_t)c;
}

// Algorithmic HBM bytes of a projection: weights once, the input rows, fp32 output rows.
static adt_status gemm_p(const void* X, int ldx, const void* W, int M, int N, int K, int dt, float* part,
                         hipStream_t st, const GemmEpi& epi = GemmEpi{}, int* splits = nullptr) {
  const int e = prof_pair();
  adt_status r = launch_gemm(X, ldx, W, M, N, K, dt, part, epi, st, e >= 0 ? g_prof.ev[e] : nullptr,
                             e >= 0 ? g_prof.ev[e + 1] : nullptr, splits);
  prof_done(e, ADT_PROF_GEMM, (double)N * K * esize(dt) + (double)M * K * esize(dt) + (double)M * N * 4.0,
            2.0 * M * N * K);
  return r;
}

// ---------------------------------------------------------------------------- capture
// Opens the record of one forward (adt_session_set_capture): checks that its residual
// snapshots, FC inputs and row metadata fit the caller's buffers, then copies the rows'
// tokens (branch 0), positions and ancestor masks.  Nothing is launched when a buffer is full.
static adt_status capt_begin(adt_session_s* s, bool draft, int M, int L_pre, int slot0, int n_tail,
                             const int32_t* tok, const int32_t* pos, const uint64_t* mask, hipStream_t st) {
  s->capt_cur = -1;
  if (!s->capt_on) return ADT_OK;
  adt_capture_rec r{};
  r.draft = draft ? 1 : 0;
  r.nodes = M;
  r.rows = s->nb * M;
  r.kv_prefix = L_pre;
  r.slot0 = slot0;
  r.n_tail = n_tail;
  r.snapshots = draft ? 3 : 2 * s->Lr + 1;
  r.resid_off = (int64_t)s->capt_resid;
  r.xin_off = (int64_t)s->capt_xin;
  r.meta_off = (int64_t)s->capt_meta;
  const size_t nres = (size_t)r.snapshots * r.rows * s->dm;
  const size_t nxin = draft ? (size_t)r.rows * 2 * s->dm * esize(s->dt) : 0;
  const size_t nmeta = (size_t)M * (2 + 2 * ADT_MASK_WORDS);
  ADT_CHECK_ARG(s->capt_resid + nres <= s->capt.resid_elems, ADT_E_CAPACITY,
                "capture: residual buffer holds %zu floats, %zu needed", s->capt.resid_elems, s->capt_resid + nres);
  ADT_CHECK_ARG(!draft || (s->capt.xin && s->capt_xin + nxin <= s->capt.xin_bytes), ADT_E_CAPACITY,
                "capture: FC input buffer holds %zu bytes, %zu needed", s->capt.xin_bytes, s->capt_xin + nxin);
  ADT_CHECK_ARG(s->capt.meta && s->capt_meta + nmeta <= s->capt.meta_elems, ADT_E_CAPACITY,
                "capture: metadata buffer holds %zu ints, %zu needed", s->capt.meta_elems, s->capt_meta + nmeta);
  int32_t* mt = s->capt.meta + s->capt_meta;
  ADT_HIP(hipMemcpyAsync(mt, tok, sizeof(int32_t) * M, hipMemcpyDeviceToDevice, st));
  ADT_HIP(hipMemcpyAsync(mt + M, pos, sizeof(int32_t) * M, hipMemcpyDeviceToDevice, st));
  ADT_HIP(hipMemcpyAsync(mt + 2 * M, mask, sizeof(uint64_t) * ADT_MASK_WORDS * M, hipMemcpyDeviceToDevice, st));
  s->capt_resid += nres;
  s->capt_xin += nxin;
  s->capt_meta += nmeta;
  s->capt_log.push_back(r);
  s->capt_cur = (int)s->capt_log.size() - 1;
  return ADT_OK;
}

// Residual snapshot idx of the forward in progress (no-op outside a captured forward).
static adt_status capt_snap(adt_session_s* s, int idx, hipStream_t st) {
  if (s->capt_cur < 0) return ADT_OK;
  const adt_capture_rec& r = s->capt_log[s->capt_cur];
  const size_t n = (size_t)r.rows * s->dm;
  ADT_HIP(hipMemcpyAsync(s->capt.resid + r.resid_off + (size_t)idx * n, s->h, sizeof(float) * n,
                         hipMemcpyDeviceToDevice, st));
  return ADT_OK;
}

// Finish of a bf16 residual projection: its K-range sums added to the residual rows (or
// assigned) and the rows' RMSNorm into out (layout out_pk) and, if given, out2 (layout out2_pk).
static adt_status resid_finish(adt_session_s* s, int splits, int rows, int assign, void* out, int out_pk, void* out2,
                               int out2_pk, hipStream_t st) {
  const int e = prof_begin(st);
  TRY(launch_resid_norm(s->part, splits, rows, s->dm, assign, s->m->d.norm_eps, s->h, out, out_pk, out2, out2_pk, s->dt,
                        st));
  prof_end(e, ADT_PROF_ROWS,
           (double)splits * rows * s->dm * 4.0 + rows * s->dm * (8.0 + (out2 ? 2.0 : 1.0) * esize(s->dt)), 0.0, st);
  return ADT_OK;
}

// bf16 forwards keep the inputs of their projections (act, att, sw, xin) in the fragment layout
// of this many 16-row blocks; fp32 forwards keep them row-major.
static int act_blocks(const adt_session_s* s, int rows) { return s->dt == ADT_BF16 ? (rows + 15) / 16 : 0; }

// A bf16 residual projection (O, down, draft FC) of the rows X (fragment layout, K columns)
// into the residual h (assign: h = Y): with one K range the product's epilogue adds it and
// leaves bf16(h) in act for the next projection, which normalises its own input; with
// several, the K-range sums and the element-wise finish.
static adt_status resid_proj(adt_session_s* s, const void* X, const void* W, int rows, int K, int assign,
                             hipStream_t st) {
  const int dm = s->dm, pk = act_blocks(s, rows);
  if (gemm_rows_plan(rows, dm, K, true).S == 1) {
    GemmEpi e;
    e.mode = EPI_RESID;
    e.resid = s->h;
    e.assign = assign;
    e.act = (uint16_t*)s->act;
    e.act_pk = pk;
    return gemm_p(X, X_FRAG, W, rows, dm, K, s->dt, s->part, st, e);
  }
  GemmEpi e;
  e.mode = EPI_PART;
  e.part = s->part;
  e.part_elems = s->part_elems;
  int sp = 1;
  TRY(gemm_p(X, X_FRAG, W, rows, dm, K, s->dt, s->part, st, e, &sp));
  const int ev = prof_begin(st);
  TRY(launch_resid_add(s->part, sp, rows, dm, assign, s->h, s->act, pk, st));
  prof_end(ev, ADT_PROF_ROWS, (double)sp * rows * dm * 4.0 + rows * dm * ((assign ? 4.0 : 8.0) + 2.0), 0.0, st);
  return ADT_OK;
}

// Decoder layers over the nb * M rows of M tree nodes (branches interleaved node by node).
// The final norm goes to final_out (row-major; bf16: act if null) and, with act_too (bf16),
// also to act.
static adt_status run_layers(adt_session_s* s, bool draft, int M, const int32_t* pos, int slot0, int L_pre, int n_tail,
                             const uint64_t* mask, void* final_out, bool act_too, hipStream_t st) {
  const adt_model_s* m = s->m;
  const int dm = s->dm, H = s->H, Dh = s->Dh, F = s->F, dt = s->dt, nb = s->nb, rows = nb * M;
  const int64_t cache_sb = draft ? s->dcache_sb : s->tcache_sb;
  const Branches br{nb, 0, cache_sb};
  const size_t es = esize(dt);
  const int64_t stride_h = (int64_t)s->d.s_cap * Dh;
  const float eps = m->d.norm_eps;
  const float scale = 1.f / std::sqrt((float)Dh);
  const int pk = act_blocks(s, rows);
  (void)slot0;
  const int l0 = draft ? s->Lr : 0, l1 = draft ? s->Lr + 1 : s->Lr;
  auto attention = [&](char* kc, char* vc) -> adt_status {
    // the prefix K/V once, tree Q/K/V in and O out, the masks
    const int e = prof_pair();
    AttnRows rl{1, nb, 0};
    rl.o_pk = pk;
    TRY(launch_tree_attn(s->q, kc, vc, cache_sb, stride_h, s->scal + SC_KV, s->scal + SC_NQ, s->scal + SC_TAIL, mask,
                         rl, nb, H, Dh, M, s->d.s_cap, scale, dt, s->att, s->attn_ws,
                         s->attn_ws_bytes, st, e >= 0 ? g_prof.ev[e] : nullptr, e >= 0 ? g_prof.ev[e + 1] : nullptr));
    prof_done(e, ADT_PROF_ATTN, nb * (2.0 * L_pre * H * Dh * es + 4.0 * M * H * Dh * es) + 16.0 * M,
              4.0 * rows * (L_pre + n_tail) * H * Dh);
    return ADT_OK;
  };
  if (dt == ADT_BF16) {
    // Per layer: QKV (RoPE + cache append) from the bf16 residual rows in act, normalised inside
    // the product; attention; O added to the residual (act = its new bf16 copy); gate/up
    // (the MLP's norm inside, SwiGLU); down added likewise, or after the last layer with the
    // final norm into final_out.
    GemmEpi pe;
    pe.mode = EPI_PART;
    pe.part = s->part;
    pe.part_elems = s->part_elems;
    for (int l = l0; l < l1; ++l) {
      char* kc = draft ? (char*)s->d.dk_cache : (char*)s->d.k_cache + (size_t)l * H * stride_h * es;
      char* vc = draft ? (char*)s->d.dv_cache : (char*)s->d.v_cache + (size_t)l * H * stride_h * es;
      TRY(capt_snap(s, 2 * (l - l0), st));
      GemmEpi qkv;
      qkv.mode = EPI_QKV;
      qkv.q = (uint16_t*)s->q;
      qkv.kc = (uint16_t*)kc;
      qkv.vc = (uint16_t*)vc;
      qkv.stride_h = stride_h;
      qkv.slot0 = s->scal + SC_SLOT;
      qkv.pos = pos;
      qkv.rope = s->rope;
      qkv.Dh = Dh;
      qkv.nb = nb;
      qkv.cache_sb = cache_sb;
      qkv.slot_cap = s->d.s_cap;
      qkv.norm_eps = eps;
      TRY(gemm_p(s->act, X_FRAG, m->qkv[l], rows, 3 * dm, dm, dt, s->part, st, qkv));
      TRY(attention(kc, vc));
      TRY(resid_proj(s, s->att, m->o[l], rows, dm, 0, st));
      TRY(capt_snap(s, 2 * (l - l0) + 1, st));
      GemmEpi sw;
      sw.mode = EPI_SWIGLU;
      sw.act = (uint16_t*)s->sw;
      sw.act_pk = pk;
      sw.norm_eps = eps;
      TRY(gemm_p(s->act, X_FRAG, m->gu[l], rows, 2 * F, dm, dt, s->part, st, sw));
      if (l + 1 < l1) {
        TRY(resid_proj(s, s->sw, m->down[l], rows, F, 0, st));
        continue;
      }
      int sp = 1;
      TRY(gemm_p(s->sw, X_FRAG, m->down[l], rows, dm, F, dt, s->part, st, pe, &sp));
      if (final_out)
        TRY(resid_finish(s, sp, rows, 0, final_out, 0, act_too ? s->act : nullptr, pk, st));
      else
        TRY(resid_finish(s, sp, rows, 0, s->act, pk, nullptr, 0, st));
    }
    TRY(capt_snap(s, 2 * (l1 - l0), st));
    return ADT_OK;
  }
  // fp32: products into part, row kernels finish each step
  for (int l = l0; l < l1; ++l) {
    char* kc = draft ? (char*)s->d.dk_cache : (char*)s->d.k_cache + (size_t)l * H * stride_h * es;
    char* vc = draft ? (char*)s->d.dv_cache : (char*)s->d.v_cache + (size_t)l * H * stride_h * es;
    TRY(capt_snap(s, 2 * (l - l0), st));
    TRY(gemm_p(s->act, dm, m->qkv[l], rows, 3 * dm, dm, dt, s->part, st));
    TRY(launch_qkv_rope(s->part, 1, rows, H, Dh, pos, s->scal + SC_SLOT, s->rope, s->q, kc, vc, stride_h, dt, st, br));
    TRY(attention(kc, vc));
    TRY(gemm_p(s->att, dm, m->o[l], rows, dm, dm, dt, s->part, st));
    TRY(launch_add_norm(s->part, 1, rows, dm, 0, eps, s->h, s->act, dt, st));
    TRY(capt_snap(s, 2 * (l - l0) + 1, st));
    TRY(gemm_p(s->act, dm, m->gu[l], rows, 2 * F, dm, dt, s->part, st));
    TRY(launch_swiglu(s->part, 1, rows, F, s->sw, dt, st));
    TRY(gemm_p(s->sw, F, m->down[l], rows, dm, F, dt, s->part, st));
    TRY(launch_add_norm(s->part, 1, rows, dm, 0, eps, s->h, l + 1 == l1 ? final_out : s->act, dt, st));
  }
  return capt_snap(s, 2 * (l1 - l0), st);
}

// Logits of M nodes (nb rows each) into out [M][V]; with guidance the per-branch rows go to
// raw [nb M][V] and out gets their combination.  feat_rows: row-major with ldx = d_model, or
// (bf16, ldx == X_FRAG) the fragment layout.
static adt_status lm_head(adt_session_s* s, const void* feat_rows, int ldx, int M, float* out, float* raw,
                          hipStream_t st) {
  const int rows = s->nb * M;
  float* dst = s->nb > 1 ? raw : out;
  if (s->dt == ADT_BF16) {
    // columns [lm_lo, lm_hi) only: their packed weight rows start lm_lo * d_model elements in
    GemmEpi e;
    e.mode = EPI_STORE;
    e.out = dst + s->lm_lo;
    e.ldo = s->V;
    const void* w = (const uint16_t*)s->m->d.lm_head + (size_t)s->lm_lo * s->dm;
    TRY(gemm_p(feat_rows, ldx, w, rows, s->lm_hi - s->lm_lo, s->dm, s->dt, s->part, st, e));
  } else {
    TRY(gemm_p(feat_rows, s->dm, s->m->d.lm_head, rows, s->V, s->dm, s->dt, s->part, st));
    TRY(launch_reduce_store(s->part, 1, rows, s->V, dst, s->V, st));
  }
  if (s->nb > 1) TRY(launch_guide_rows(raw, M, s->V, s->gscale, out, s->V, st));
  return ADT_OK;
}

// Target forward of M rows with tokens tok; features into s->feat; logits of rows
// [lm_row0, lm_row0 + lm_rows) into s->logits.
// (M nodes, nb rows each; tok_boff as in Branches: 0 = the branches share the tokens.)
static adt_status target_forward(adt_session_s* s, const int32_t* tok, int M, const int32_t* pos, int slot0, int L_pre,
                                 int n_tail, const uint64_t* mask, int lm_row0, int lm_rows, hipStream_t st,
                                 int64_t key = -1, int tok_boff = 0) {
  TRY(set_scalars(s, L_pre, M, n_tail, slot0, st));
  auto body = [&](hipStream_t cs) -> adt_status {
    TRY(capt_begin(s, false, M, L_pre, slot0, n_tail, tok, pos, mask, cs));
    const int pk = act_blocks(s, s->nb * M);
    // bf16: act takes the raw embedding rows (the first projection normalises them)
    TRY(launch_embed_norm(s->m->d.embed, tok, s->nb * M, s->dm, s->m->d.norm_eps, s->h, s->act, s->dt, cs,
                          Branches{s->nb, tok_boff, 0}, pk, pk > 0));
    // logits of every row read the final norm from act in the fragment layout
    const bool all = pk && lm_row0 == 0 && lm_rows == M;
    TRY(run_layers(s, false, M, pos, slot0, L_pre, n_tail, mask, s->feat, all, cs));
    if (all)
      TRY(lm_head(s, s->act, X_FRAG, lm_rows, s->logits, s->rawlog, cs));
    else if (lm_rows > 0)
      TRY(lm_head(s, (const char*)s->feat + (size_t)s->nb * lm_row0 * s->dm * esize(s->dt), s->dm, lm_rows,
                  s->logits, s->rawlog, cs));
    s->capt_cur = -1;
    return ADT_OK;
  };
  return key < 0 ? body(st) : run_graph(s, key, st, body);
}

// Draft-head forward: FC over [embedding ; parent feature], one decoder layer, final norm
// into feature rows fout (may be null), target LM head for rows [lm_row0, +lm_rows) into out.
// (M nodes, nb rows each; lraw takes the per-branch logits under guidance.)
static adt_status draft_forward(adt_session_s* s, const int32_t* tok, const int32_t* fsrc, const void* fa, int M,
                                const int32_t* pos, int slot0, int L_pre, int n_tail, const uint64_t* mask, void* fout,
                                int lm_row0, int lm_rows, float* lout, float* lraw, hipStream_t st, int64_t key = -1,
                                int tok_boff = 0) {
  const int dm = s->dm, dt = s->dt, rows = s->nb * M;
  TRY(set_scalars(s, L_pre, M, n_tail, slot0, st));
  auto body = [&](hipStream_t cs) -> adt_status {
    TRY(capt_begin(s, true, M, L_pre, slot0, n_tail, tok, pos, mask, cs));
    const int pk = act_blocks(s, rows);
    TRY(launch_draft_input(s->m->d.embed, tok, fsrc, fa, s->dfeat, rows, dm, s->xin, dt, cs,
                           Branches{s->nb, tok_boff, 0}, pk));
    if (s->capt_cur >= 0)   // the captured FC input is row-major
      TRY(launch_draft_input(s->m->d.embed, tok, fsrc, fa, s->dfeat, rows, dm,
                             (char*)s->capt.xin + s->capt_log[s->capt_cur].xin_off, dt, cs,
                             Branches{s->nb, tok_boff, 0}, 0));
    if (dt == ADT_BF16) {
      TRY(resid_proj(s, s->xin, s->m->d.draft_fc, rows, 2 * dm, 1, cs));
    } else {
      TRY(gemm_p(s->xin, 2 * dm, s->m->d.draft_fc, rows, dm, 2 * dm, dt, s->part, cs));
      TRY(launch_add_norm(s->part, 1, rows, dm, 1, s->m->d.norm_eps, s->h, s->act, dt, cs));
    }
    const bool all = pk && fout && lm_row0 == 0 && lm_rows == M;
    TRY(run_layers(s, true, M, pos, slot0, L_pre, n_tail, mask, fout, all, cs));
    if (all)
      TRY(lm_head(s, s->act, X_FRAG, lm_rows, lout, lraw, cs));
    else if (lm_rows > 0)
      TRY(lm_head(s, (const char*)fout + (size_t)s->nb * lm_row0 * dm * esize(dt), dm, lm_rows, lout, lraw, cs));
    s->capt_cur = -1;
    return ADT_OK;
  };
  return key < 0 ? body(st) : run_graph(s, key, st, body);
}

// Debug builds: the invariant violations the kernels recorded since the last look (cleared).
static adt_status device_errors() {
  if (!ADT_DEVICE_CHECKS) return ADT_OK;
  const uint32_t bits = dev_errors_take_rows() | dev_errors_take_select() | dev_errors_take_attn() |
                        dev_errors_take_gemm();
  ADT_CHECK_ARG(!(bits & 0x80000000u), ADT_E_HIP, "device check: the error words could not be read");
  ADT_CHECK_ARG(bits == 0, ADT_E_DEVICE_INVARIANT, "device invariant violated:%s%s%s",
                (bits & DEVINV_PARENT) ? " a parent not before its child" : "",
                (bits & DEVINV_KV_RANGE) ? " keys past the cache capacity" : "",
                (bits & DEVINV_PATH) ? " an accepted-path entry outside the tree" : "");
  return ADT_OK;
}

static adt_status sync_stream(hipStream_t st) {
  ADT_HIP(hipStreamSynchronize(st));
  prof_collect();
  return device_errors();
}

extern "C" int32_t adt_device_checks_enabled(void) { return ADT_DEVICE_CHECKS ? 1 : 0; }

extern "C" adt_status adt_device_check(void* stream) {
  ADT_HIP(hipStreamSynchronize((hipStream_t)stream));
  return device_errors();
}

static adt_status set_root_only_tree(adt_session_s* s, int root_token, int L, hipStream_t st) {
  int32_t v[1] = {1};
  TRY(launch_set_i32(s->tr.n, small_of(v, 1), 1, st));
  int32_t p[1] = {-1};
  TRY(launch_set_i32(s->tr.parent, small_of(p, 1), 1, st));
  int32_t t[1] = {root_token};
  TRY(launch_set_i32(s->tr.token, small_of(t, 1), 1, st));
  TRY(launch_tree_masks(s->tr.parent, s->tr.n, 1, R, s->tr.mask, s->tr.depth, st));
  TRY(launch_tree_rows(s->tr.depth, s->tr.n, R, L, s->P, s->T, s->allowed_img, s->tr.pos, s->tr.allowed_rows,
                       s->tr.score, st));
  s->n_nodes = 1;
  s->expanded = false;
  return ADT_OK;
}

// The session's acceptance settings; stochastic children read q from the session's own draft
// logit rows through the map its last expansion wrote.
static adt_accept_cfg session_accept_cfg(const adt_session_s* s) {
  adt_accept_cfg c = s->d.accept;
  c.q_logits = s->dlogits;
  c.q_ld = s->V;
  c.q_row = s->tr.qrow;
  c.q_rows = s->DLR;
  return c;
}

extern "C" adt_status adt_session_prefill(adt_session* s, const int32_t* prefix, int32_t* first_token, void* stream) {
  ADT_CHECK_ARG(s && prefix, ADT_E_ARG, "prefill: null pointer");
  ADT_CHECK_ARG(!s->prefilled, ADT_E_STATE, "prefill: already prefilled");
  hipStream_t st = (hipStream_t)stream;
  const int P = s->P, nb = s->nb;
  for (int i = 0; i < nb * P; ++i)
    ADT_CHECK_ARG(prefix[i] >= 0 && prefix[i] < s->V, ADT_E_ARG, "prefill: id %d", prefix[i]);
  // ctok = the prompts of all branches, branch after branch
  ADT_HIP(hipMemcpyAsync(s->ctok, prefix, sizeof(int32_t) * nb * P, hipMemcpyHostToDevice, st));
  TRY(sync_stream(st));
  TRY(launch_iota(s->cpos, P, 0, 1, st));
  TRY(launch_chain_masks(s->cmask, P, st));
  // Target and draft over the prompt in chunks of at most R rows (R / nb nodes).  Row p of the
  // draft takes the target feature of p - 1 (zeros for p = 0); the feature of the node before
  // a chunk is carried in draft-feature node 0.
  const int CH = R / nb;
  for (int c0 = 0; c0 < P; c0 += CH) {
    const int cn = std::min(CH, P - c0);
    const bool last = c0 + cn == P;
    TRY(target_forward(s, s->ctok + c0, cn, s->cpos + c0, c0, c0, cn, s->cmask, cn - 1, last ? 1 : 0, st, -1, P));
    TRY(launch_iota(s->cfsrc, cn, -1, 1, st));
    if (c0 > 0) {
      int32_t carry[1] = {-2};
      TRY(launch_set_i32(s->cfsrc, small_of(carry, 1), 1, st));
    }
    TRY(draft_forward(s, s->ctok + c0, s->cfsrc, s->feat, cn, s->cpos + c0, c0, c0, cn, s->cmask, nullptr, 0, 0,
                      nullptr, nullptr, st, -1, P));
    int32_t li[1] = {cn - 1};
    TRY(launch_set_i32(s->idx, small_of(li, 1), 1, st));
    TRY(launch_gather_rows(s->feat, s->idx, 1, nb * s->dm, last ? s->cfeat : s->dfeat, s->dt, st));
  }
  TRY(set_root_only_tree(s, prefix[P - 1], P - 1, st));
  // the root-only tree's successor is image cell 0
  TRY(launch_fill_pairs(s->tr.allowed_rows, 1, s->allowed_h[0], s->allowed_h[1], st));
  TRY(accept_impl(s->logits, s->V, s->V, s->tr.parent, s->tr.token, s->tr.allowed_rows, s->tr.n, 1, session_accept_cfg(s), 0,
                  s->tr.path, s->tr.nacc, s->tr.bonus, s->acc_ws, s->acc_ws_bytes, st));
  int32_t first = 0;
  ADT_HIP(hipMemcpyAsync(&first, s->tr.bonus, sizeof(int32_t), hipMemcpyDeviceToHost, st));
  TRY(sync_stream(st));
  s->tokens.assign(prefix, prefix + P);
  s->tokens.push_back(first);
  s->L = P;
  s->Ld = P;
  s->step = 1;
  s->prefilled = true;
  s->have_prev = false;
  if (first_token) *first_token = first;
  return ADT_OK;
}

static void cell_range(const adt_session_s* s, int cell, int& lo, int& hi) {
  cell = std::max(0, std::min(s->T - 1, cell));
  lo = s->allowed_h[2 * cell];
  hi = s->allowed_h[2 * cell + 1];
}

// Stochastic children (the session's acceptance is ADT_ACCEPT_MSS): the root's draft row is in
// dlogits row 0 and its allowed range in allowed_lvl[0].  Every expanded node draws ch children
// from q; level lvl expands the best nf nodes of the previous layer (nf <= k_hat, whole
// expansions within n_budget); the tree keeps every drawn child in creation order.
static adt_status expand_sampled(adt_session_s* s, int d_hat, int k_hat, int n_budget, int cu, bool table,
                                 int32_t* n_nodes_out, hipStream_t st) {
  const adt_sched_cfg& c = s->d.sched;
  const adt_accept_cfg& a = s->d.accept;
  const int V = s->V, L = s->L, P = s->P, ch = a.children;
  const uint32_t step = (uint32_t)s->step;
  TRY(launch_row_sample(s->dlogits, V, V, s->allowed_lvl, 1, nullptr, ch, a.temperature, a.top_k, a.seed, step,
                        s->samp_w, s->top_id, s->top_val, s->lse, 16, st));
  int pool_n = ch;
  int nf = d_hat > 1 ? std::min({k_hat, ch, (n_budget - pool_n) / ch}) : 0;
  TRY(launch_expand_level(s->pool, nullptr, 1, ch, 0, 1, std::max(nf, 1), s->top_id, s->top_val, s->lse, 16,
                          nf > 0 ? 1 : 0, L, 0, cu - 1, s->C0, 1, s->nx[0], st));
  int drow = 0, cur = 0;
  for (int lvl = 2; lvl <= d_hat && nf > 0; ++lvl) {
    const int dl_row = 1 + (lvl - 2) * c.k_hi;
    float* lrows = s->dlogits + (size_t)dl_row * V;
    void* fout = (char*)s->dfeat + (size_t)s->nb * (s->C0 + drow) * s->dm * esize(s->dt);
    if (table) {
      TRY(launch_table_rows(s->nx[cur].tok, nf, lvl - 1, s->d.draft_table_rows, s->idx, st));
      TRY(launch_gather_rows(s->d.draft_table, s->idx, nf, V, lrows, ADT_F32, st));
    } else {
      TRY(draft_forward(s, s->nx[cur].tok, s->nx[cur].fsrc, s->cfeat, nf, s->nx[cur].pos, L + 1 + drow, L + 1,
                        drow + nf, s->nx[cur].mask, fout, 0, nf, lrows, s->draw ? s->draw + (size_t)s->nb * s->V : nullptr,
                        st, gkey(3, lvl, nf, drow)));
    }
    int lo, hi;
    cell_range(s, L + lvl - P, lo, hi);
    TRY(launch_fill_pairs(s->allowed_lvl, nf, lo, hi, st));
    TRY(launch_row_sample(lrows, V, V, s->allowed_lvl, nf, s->nx[cur].frontier, ch, a.temperature, a.top_k, a.seed,
                          step, s->samp_w, s->top_id, s->top_val, s->lse, 16, st));
    const int made = nf * ch;
    const int nf_next = lvl < d_hat ? std::min({k_hat, made, (n_budget - pool_n - made) / ch}) : 0;
    TRY(launch_expand_level(s->pool, s->nx[cur].frontier, nf, ch, pool_n, lvl, std::max(nf_next, 1), s->top_id,
                            s->top_val, s->lse, 16, nf_next > 0 ? 1 : 0, L, drow + nf, cu - 1, s->C0,
                            1 + (lvl - 1) * c.k_hi, s->nx[cur ^ 1], st));
    pool_n += made;
    drow += nf;
    nf = nf_next;
    cur ^= 1;
  }
  TRY(launch_expand_finalize(s->pool, pool_n, pool_n, s->tokens[L], L, P, s->T, s->allowed_img,
                             s->tr.parent, s->tr.token, s->tr.depth, s->tr.score, s->tr.pos, s->tr.mask,
                             s->tr.allowed_rows, s->tr.qrow, s->tr.n, true, st));
  s->n_nodes = pool_n + 1;
  s->expanded = true;
  if (n_nodes_out) *n_nodes_out = s->n_nodes;
  return ADT_OK;
}

extern "C" adt_status adt_tree_expand(adt_session* s, int32_t d_hat, int32_t k_hat, int32_t n_budget,
                                      int32_t* n_nodes_out, void* stream) {
  ADT_CHECK_ARG(s != nullptr, ADT_E_ARG, "tree_expand: null session");
  ADT_CHECK_ARG(s->prefilled, ADT_E_STATE, "tree_expand: session not prefilled");
  const adt_sched_cfg& c = s->d.sched;
  const int k_top = (c.k_clamp == ADT_KCLAMP_DEEP && d_hat == 1) ? ADT_MAX_WIDTH : c.k_hi;
  ADT_CHECK_ARG(d_hat >= 1 && d_hat <= c.d_hi && k_hat >= 1 && k_hat <= k_top, ADT_E_ARG,
                "tree_expand: (d,k)=(%d,%d) outside the session bounds", d_hat, k_hat);
  ADT_CHECK_ARG(n_budget >= 1 && n_budget <= R / s->nb - 1, ADT_E_CAPACITY, "tree_expand: n_budget %d", n_budget);
  const int L = s->L, Ld = s->Ld, P = s->P;
  ADT_CHECK_ARG(L + 1 + d_hat - P <= s->T, ADT_E_ARG, "tree_expand: depth %d runs past the image", d_hat);
  hipStream_t st = (hipStream_t)stream;
  const int V = s->V;
  // catch-up rows: committed positions Ld..L, the root last
  const int cu = L - Ld + 1;
  ADT_CHECK_ARG(cu >= 1 && cu <= std::min(32, s->C0), ADT_E_STATE, "tree_expand: %d catch-up rows", cu);
  std::vector<int32_t> ctok(s->tokens.begin() + Ld, s->tokens.begin() + L + 1);
  const bool table = s->d.draft_table != nullptr;
  const int trows = s->d.draft_table_rows;
  if (table) {
    TRY(launch_set_i32(s->ctok, small_of(ctok.data(), cu), cu, st));
    TRY(launch_table_rows(s->ctok + (cu - 1), 1, 0, trows, s->idx, st));
    TRY(launch_gather_rows(s->d.draft_table, s->idx, 1, V, s->dlogits, ADT_F32, st));
  } else {
    TRY(launch_catchup_rows(small_of(ctok.data(), cu), cu, Ld, s->ctok, s->cfsrc, s->cpos, s->cmask, st));
    TRY(draft_forward(s, s->ctok, s->cfsrc, s->cfeat, cu, s->cpos, Ld, Ld, cu, s->cmask, s->dfeat, cu - 1, 1,
                      s->dlogits, s->draw, st, gkey(2, 0, 0, cu)));
  }
  int lo, hi;
  cell_range(s, L + 1 - P, lo, hi);
  if (s->d.accept.mode == ADT_ACCEPT_MSS) {
    ADT_CHECK_ARG(n_budget >= s->d.accept.children, ADT_E_ARG, "tree_expand: n_budget %d below the %d children of one node",
                  n_budget, s->d.accept.children);
    TRY(launch_fill_pairs(s->allowed_lvl, 1, lo, hi, st));
    return expand_sampled(s, d_hat, k_hat, n_budget, cu, table, n_nodes_out, st);
  }
  // layer 1: the root's top-k children
  TRY(launch_row_topk(s->dlogits, V, V, nullptr, 1, k_hat, 16, s->top_id, s->top_val, s->lse, s->topk_ws,
                      s->topk_ws_bytes, st, lo, hi));
  int cnt = std::min(k_hat, hi - lo);
  TRY(launch_expand_level(s->pool, nullptr, 1, cnt, 0, 1, k_hat, s->top_id, s->top_val, s->lse, 16, d_hat > 1 ? 1 : 0,
                          L, 0, cu - 1, s->C0, 1, s->nx[0], st));
  int pool_n = cnt, nf = std::min(k_hat, cnt), drow = 0, cur = 0;
  for (int lvl = 2; lvl <= d_hat; ++lvl) {
    const int dl_row = 1 + (lvl - 2) * c.k_hi;
    float* lrows = s->dlogits + (size_t)dl_row * V;
    void* fout = (char*)s->dfeat + (size_t)s->nb * (s->C0 + drow) * s->dm * esize(s->dt);
    if (table) {
      TRY(launch_table_rows(s->nx[cur].tok, nf, lvl - 1, trows, s->idx, st));
      TRY(launch_gather_rows(s->d.draft_table, s->idx, nf, V, lrows, ADT_F32, st));
    } else {
      TRY(draft_forward(s, s->nx[cur].tok, s->nx[cur].fsrc, s->cfeat, nf, s->nx[cur].pos, L + 1 + drow, L + 1,
                        drow + nf, s->nx[cur].mask, fout, 0, nf, lrows, s->draw ? s->draw + (size_t)s->nb * s->V : nullptr,
                        st, gkey(3, lvl, nf, drow)));
    }
    cell_range(s, L + lvl - P, lo, hi);
    TRY(launch_row_topk(lrows, V, V, nullptr, nf, k_hat, 16, s->top_id, s->top_val, s->lse, s->topk_ws,
                        s->topk_ws_bytes, st, lo, hi));
    cnt = std::min(k_hat, hi - lo);
    TRY(launch_expand_level(s->pool, s->nx[cur].frontier, nf, cnt, pool_n, lvl, k_hat, s->top_id, s->top_val, s->lse,
                            16, lvl < d_hat ? 1 : 0, L, drow + nf, cu - 1, s->C0, 1 + (lvl - 1) * c.k_hi,
                            s->nx[cur ^ 1], st));
    pool_n += nf * cnt;
    drow += nf;
    nf = std::min(k_hat, nf * cnt);
    cur ^= 1;
  }
  TRY(launch_expand_finalize(s->pool, pool_n, n_budget, s->tokens[L], L, P, s->T, s->allowed_img,
                             s->tr.parent, s->tr.token, s->tr.depth, s->tr.score, s->tr.pos, s->tr.mask,
                             s->tr.allowed_rows, s->tr.qrow, s->tr.n, false, st));
  s->n_nodes = std::min(n_budget, pool_n) + 1;
  s->expanded = true;
  if (n_nodes_out) *n_nodes_out = s->n_nodes;
  return ADT_OK;
}

extern "C" adt_status adt_session_set_tree(adt_session* s, const int32_t* parent, const int32_t* token, int32_t n,
                                           void* stream) {
  ADT_CHECK_ARG(s && parent && token, ADT_E_ARG, "set_tree: null pointer");
  ADT_CHECK_ARG(s->prefilled, ADT_E_STATE, "set_tree: session not prefilled");
  ADT_CHECK_ARG(n >= 1 && n <= R / s->nb, ADT_E_CAPACITY, "set_tree: n %d (at most %d)", n, R / s->nb);
  ADT_CHECK_ARG(parent[0] == -1, ADT_E_ARG, "set_tree: node 0 must be the root");
  ADT_CHECK_ARG(s->d.accept.mode != ADT_ACCEPT_MSS, ADT_E_UNSUPPORTED,
                "set_tree: stochastic-children sessions verify their own expansions (the q rows of a given tree "
                "are unknown); use adt_verify_accept with q rows");
  std::vector<int> dep(n, 0);
  for (int i = 1; i < n; ++i) {
    ADT_CHECK_ARG(parent[i] >= 0 && parent[i] < i, ADT_E_ARG, "set_tree: parent[%d]=%d not BFS ordered", i, parent[i]);
    ADT_CHECK_ARG(token[i] >= 0 && token[i] < s->V, ADT_E_ARG, "set_tree: token[%d]", i);
    dep[i] = dep[parent[i]] + 1;
  }
  const int dmax = *std::max_element(dep.begin(), dep.end());
  ADT_CHECK_ARG(s->L + 1 + dmax - s->P <= s->T, ADT_E_ARG, "set_tree: tree deeper than the image remainder");
  ADT_CHECK_ARG(s->L + n <= s->d.s_cap, ADT_E_CAPACITY, "set_tree: cache capacity");
  ADT_CHECK_ARG(token[0] == s->tokens[s->L], ADT_E_ARG, "set_tree: token[0] must be the root token %d",
                s->tokens[s->L]);
  hipStream_t st = (hipStream_t)stream;
  ADT_HIP(hipMemcpyAsync(s->tr.parent, parent, sizeof(int32_t) * n, hipMemcpyHostToDevice, st));
  ADT_HIP(hipMemcpyAsync(s->tr.token, token, sizeof(int32_t) * n, hipMemcpyHostToDevice, st));
  int32_t v[1] = {n};
  TRY(launch_set_i32(s->tr.n, small_of(v, 1), 1, st));
  TRY(launch_tree_masks(s->tr.parent, s->tr.n, 1, R, s->tr.mask, s->tr.depth, st));
  TRY(launch_tree_rows(s->tr.depth, s->tr.n, R, s->L, s->P, s->T, s->allowed_img, s->tr.pos, s->tr.allowed_rows,
                       s->tr.score, st));
  TRY(sync_stream(st));
  s->n_nodes = n;
  // s->expanded is kept: after adt_tree_expand the draft cache covers the root whichever tree
  // is verified next, and the node rows past it are rewritten by the next catch-up.
  return ADT_OK;
}

extern "C" adt_status adt_verify_forward(adt_session* s, void* stream) {
  ADT_CHECK_ARG(s != nullptr, ADT_E_ARG, "verify: null session");
  ADT_CHECK_ARG(s->prefilled && s->n_nodes >= 1, ADT_E_STATE, "verify: no tree");
  ADT_CHECK_ARG(s->L + s->n_nodes <= s->d.s_cap, ADT_E_CAPACITY, "verify: cache capacity");
  const int n = s->n_nodes;
  return target_forward(s, s->tr.token, n, s->tr.pos, s->L, s->L, n, s->tr.mask, 0, n, (hipStream_t)stream,
                        gkey(1, 0, 0, n));
}

// Acceptance on the last verify and the readback of its result into the session's pinned
// staging (asynchronous on st); accept_finish commits once st has been synchronised.
static adt_status accept_launch(adt_session_s* s, hipStream_t st) {
  const int n = s->n_nodes;
  TRY(accept_impl(s->logits, s->V, s->V, s->tr.parent, s->tr.token, s->tr.allowed_rows, s->tr.n, n, session_accept_cfg(s),
                  (uint64_t)s->step, s->tr.path, s->tr.nacc, s->tr.bonus, s->acc_ws, s->acc_ws_bytes, st));
  ADT_HIP(hipMemcpyAsync(s->h_acc, s->tr.path, sizeof(int32_t) * (2 * R + 2), hipMemcpyDeviceToHost, st));
  return ADT_OK;
}

static adt_status accept_finish(adt_session_s* s, int32_t d_hat, int32_t k_hat, adt_step_out* out, hipStream_t st);

extern "C" adt_status adt_session_accept_commit(adt_session* s, int32_t d_hat, int32_t k_hat, adt_step_out* out,
                                                void* stream) {
  ADT_CHECK_ARG(s != nullptr, ADT_E_ARG, "accept_commit: null session");
  ADT_CHECK_ARG(s->prefilled && s->n_nodes >= 1, ADT_E_STATE, "accept_commit: no verified tree");
  hipStream_t st = (hipStream_t)stream;
  TRY(accept_launch(s, st));
  TRY(sync_stream(st));
  return accept_finish(s, d_hat, k_hat, out, st);
}

// c + d1 after the acceptance's readback has landed: compaction, catch-up features, records
static adt_status accept_finish(adt_session_s* s, int32_t d_hat, int32_t k_hat, adt_step_out* out, hipStream_t st) {
  const int n = s->n_nodes, L = s->L, P = s->P;
  const int32_t* path = s->h_acc;
  const int32_t* tok = s->h_acc + R;
  const int32_t a = s->h_acc[2 * R], bonus = s->h_acc[2 * R + 1];
  ADT_CHECK_ARG(a >= 0 && a < n, ADT_E_STATE, "accept_commit: accepted length %d out of range", a);
  // Catch-up features are kept for committed positions Ld-1 .. L_new-1.  After an expansion
  // the draft cache covers the root, so the next catch-up starts at L + 1.
  const int new_Ld = s->expanded ? L + 1 : s->Ld;
  const int frow0 = L - (new_Ld - 1);
  ADT_CHECK_ARG(frow0 >= 0 && frow0 + a + 1 <= s->C0, ADT_E_CAPACITY,
                "accept_commit: %d catch-up rows exceed %d (too many cycles without expansion)", frow0 + a + 1, s->C0);
  if (a > 0) {
    int32_t lv[1] = {L};
    TRY(launch_set_i32(s->scal + SC_CL, small_of(lv, 1), 1, st));
    const int e = prof_begin(st);
    // every guidance branch moves the same accepted nodes
    TRY(launch_kv_compact(s->d.k_cache, s->d.v_cache, s->nb, s->Lr * s->H, s->Dh, s->tcache_sb,
                          (int64_t)s->d.s_cap * s->Dh, s->scal + SC_CL, 0, s->tr.path, 0, s->tr.nacc, 0, a, s->dt, st));
    prof_end(e, ADT_PROF_COMPACT, 4.0 * s->nb * a * s->Lr * s->H * s->Dh * esize(s->dt), 0.0, st);
  }
  TRY(launch_gather_rows(s->feat, s->tr.path, a + 1, s->nb * s->dm,
                         (char*)s->cfeat + (size_t)s->nb * frow0 * s->dm * esize(s->dt), s->dt, st));
  const int cell0 = L + 1 - P;
  std::vector<int32_t> committed;
  for (int m = 1; m <= a; ++m) committed.push_back(tok[path[m]]);
  committed.push_back(bonus);
  for (int c = 0; c < (int)committed.size(); ++c)
    if (cell0 + c < s->T) {
      s->rec_d[cell0 + c] = d_hat;
      s->rec_k[cell0 + c] = k_hat;
      s->has_rec[cell0 + c] = 1;
    }
  s->have_prev = true;
  s->a_prev = a;
  s->d_prev = d_hat;
  s->prev_cell = cell0;
  s->tokens.insert(s->tokens.end(), committed.begin(), committed.end());
  s->Ld = new_Ld;
  s->L = L + 1 + a;
  s->expanded = false;
  if (out) {
    out->step = s->step;
    out->d_hat = d_hat;
    out->k_hat = k_hat;
    out->n_nodes = n;
    out->n_accepted = a;
    out->n_committed = a + 1;
    for (int i = 0; i <= a; ++i) out->tokens[i] = committed[i];
    out->done = ((int)s->tokens.size() - P >= s->T) ? 1 : 0;
  }
  s->step += 1;
  return ADT_OK;
}

static adt_status schedule_for(adt_session_s* s, int& d_hat, int& k_hat) {
  const adt_sched_cfg& c = s->d.sched;
  const int cell = s->L + 1 - s->P;
  const int remaining = s->T - cell;
  if (s->d.fixed_tree) {
    d_hat = std::min(c.d_hi, remaining - 1);
    k_hat = c.k_hi;
    return ADT_OK;
  }
  int have = 0, d0 = 0, k0 = 0;
  TRY(adt_schedule_init(&c, cell, s->T, s->rec_d.data(), s->rec_k.data(), s->has_rec.data(), &have, &d0, &k0));
  int a_prev = s->a_prev;
  if (c.alpha_source == ADT_ALPHA_POISSON && s->have_prev) a_prev = std::min(s->poisson[s->prev_cell], s->d_prev);
  return adt_schedule_next(&c, have, d0, k0, s->have_prev ? 1 : 0, a_prev, s->d_prev, remaining, &d_hat, &k_hat);
}

extern "C" adt_status adt_step(adt_session* s, adt_step_out* out, void* stream) {
  ADT_CHECK_ARG(s != nullptr, ADT_E_ARG, "step: null session");
  ADT_CHECK_ARG(s->prefilled, ADT_E_STATE, "step: session not prefilled");
  hipStream_t st = (hipStream_t)stream;
  if ((int)s->tokens.size() - s->P >= s->T) {
    if (out) {
      memset(out, 0, sizeof(*out));
      out->done = 1;
    }
    return ADT_OK;
  }
  int d_hat = 0, k_hat = 0;
  TRY(schedule_for(s, d_hat, k_hat));
  if (d_hat >= 1) {
    TRY(adt_tree_expand(s, d_hat, k_hat, s->d.sched.n_budget, nullptr, st));
  } else {
    TRY(set_root_only_tree(s, s->tokens[s->L], s->L, st));
  }
  TRY(adt_verify_forward(s, st));
  return adt_session_accept_commit(s, d_hat, k_hat, out, st);
}

// ============================================================================ batched cycle
struct adt_batch_s {
  std::vector<adt_session_s*> ss;
  int B = 0, Mmax = 0, Nmax = 0;
  int64_t cache_sb = 0;        // elements between consecutive sessions' target caches
  float *h = nullptr, *C = nullptr;
  void *a = nullptr, *q = nullptr, *att = nullptr, *sw = nullptr, *feat = nullptr;
  int32_t *tok, *pos, *slot, *seq, *row_off, *kv_len, *nq;
  uint64_t* mask;
  void* attn_ws = nullptr;
  size_t attn_ws_bytes = 0;
  float* gemm_part = nullptr;   // fp32 partials of the projections' K splits
  size_t gemm_part_elems = 0;
  // The sessions' draft expansions are independent chains of small kernels; they run on
  // BATCH_STREAMS streams of their own (default priority), joined to the caller's stream by
  // events, so several overlap on the GPU.
  static constexpr int BATCH_STREAMS = 4;
  hipStream_t aux[BATCH_STREAMS] = {};
  hipEvent_t ev_fork = nullptr, ev_join[BATCH_STREAMS] = {};
  ~adt_batch_s() {
    for (int j = 0; j < BATCH_STREAMS; ++j) {
      if (aux[j]) (void)hipStreamDestroy(aux[j]);
      if (ev_join[j]) (void)hipEventDestroy(ev_join[j]);
    }
    if (ev_fork) (void)hipEventDestroy(ev_fork);
  }
};

static adt_status batch_streams(adt_batch_s* bt) {
  if (bt->ev_fork) return ADT_OK;
  for (int j = 0; j < adt_batch_s::BATCH_STREAMS; ++j) {
    ADT_HIP(hipStreamCreateWithFlags(&bt->aux[j], hipStreamNonBlocking));
    ADT_HIP(hipEventCreateWithFlags(&bt->ev_join[j], hipEventDisableTiming));
  }
  ADT_HIP(hipEventCreateWithFlags(&bt->ev_fork, hipEventDisableTiming));
  return ADT_OK;
}

static adt_status check_batch(adt_session* const* ss, int B, int64_t& cache_sb) {
  ADT_CHECK_ARG(ss && B >= 1 && B <= 256, ADT_E_ARG, "batch: %d sessions", B);
  for (int b = 0; b < B; ++b) ADT_CHECK_ARG(ss[b] != nullptr, ADT_E_ARG, "batch: session %d is null", b);
  const adt_session_s* s0 = ss[0];
  const int64_t per = (int64_t)s0->Lr * s0->H * s0->d.s_cap * s0->Dh;
  cache_sb = B > 1 ? ((const char*)ss[1]->d.k_cache - (const char*)s0->d.k_cache) / (int64_t)esize(s0->dt) : per;
  ADT_CHECK_ARG(cache_sb >= per, ADT_E_SHAPE, "batch: target caches closer than one session's size");
  for (int b = 0; b < B; ++b) {
    const adt_session_s* s = ss[b];
    ADT_CHECK_ARG(s->m == s0->m && s->dt == ADT_BF16 && s->nb == 1, ADT_E_ARG,
                  "batch: session %d is not an unguided bf16 session of the first one's model", b);
    ADT_CHECK_ARG(s->prefilled && s->d.s_cap == s0->d.s_cap, ADT_E_ARG, "batch: session %d not prefilled or s_cap", b);
    ADT_CHECK_ARG((const char*)s->d.k_cache == (const char*)s0->d.k_cache + b * cache_sb * esize(s->dt) &&
                      (const char*)s->d.v_cache == (const char*)s0->d.v_cache + b * cache_sb * esize(s->dt),
                  ADT_E_SHAPE, "batch: caches of session %d not at the common stride", b);
  }
  const int dm = s0->dm, F = s0->F, V = s0->V;
  ADT_CHECK_ARG(dm % 128 == 0 && F % 128 == 0 && V % 128 == 0 && F % 64 == 0, ADT_E_SHAPE,
                "batch: d_model, ffn and vocab must be multiples of 128");
  return ADT_OK;
}

static size_t batch_layout(adt_batch_s* bt, const adt_session_s* s0, char* base) {
  Bump b{base};
  const int M = bt->Mmax, dm = s0->dm;
  bt->h = b.take<float>((size_t)M * dm);
  bt->C = b.take<float>((size_t)M * bt->Nmax);
  bt->a = b.take<uint16_t>((size_t)M * dm);
  bt->q = b.take<uint16_t>((size_t)M * dm);
  bt->att = b.take<uint16_t>((size_t)M * dm);
  bt->sw = b.take<uint16_t>((size_t)M * s0->F);
  bt->feat = b.take<uint16_t>((size_t)M * dm);
  bt->tok = b.take<int32_t>(M);
  bt->pos = b.take<int32_t>(M);
  bt->slot = b.take<int32_t>(M);
  bt->seq = b.take<int32_t>(M);
  bt->row_off = b.take<int32_t>(bt->B + 1);
  bt->kv_len = b.take<int32_t>(bt->B);
  bt->nq = b.take<int32_t>(bt->B);
  bt->mask = b.take<uint64_t>((size_t)M * ADT_MASK_WORDS);
  bt->attn_ws_bytes = tree_attn_ws_bytes(bt->B, s0->H, s0->Dh, R, s0->d.s_cap, s0->dt);
  bt->attn_ws = b.take<char>(std::max<size_t>(bt->attn_ws_bytes, 256));
  // scratch for the K splits the packed-GEMM plan takes, at the most any row count needs
  const int F = s0->F;
  const int shapes[5][2] = {{3 * dm, dm}, {dm, dm}, {2 * F, dm}, {dm, F}, {s0->V, dm}};
  size_t part = 0;
  for (int m = 1; m <= M; ++m)
    for (const auto& sh : shapes) part = std::max(part, gemm_nt_part_elems(m, sh[0], sh[1]));
  bt->gemm_part_elems = part;
  bt->gemm_part = part ? b.take<float>(part) : nullptr;
  return align_up(b.off, 256);
}

static void batch_dims(adt_batch_s* bt, adt_session* const* ss, int B) {
  const adt_session_s* s0 = ss[0];
  bt->B = B;
  bt->Mmax = B * R;
  bt->Nmax = std::max({3 * s0->dm, 2 * s0->F, s0->V});
}

extern "C" size_t adt_batch_workspace_size(adt_session* const* sessions, int32_t B) {
  int64_t sb = 0;
  if (check_batch(sessions, B, sb)) return 0;
  adt_batch_s bt;
  batch_dims(&bt, sessions, B);
  return batch_layout(&bt, sessions[0], nullptr);
}

extern "C" adt_status adt_batch_create(adt_session* const* sessions, int32_t B, void* workspace,
                                       size_t workspace_bytes, adt_batch** out) {
  ADT_CHECK_ARG(out != nullptr, ADT_E_ARG, "batch_create: null out");
  int64_t sb = 0;
  TRY(check_batch(sessions, B, sb));
  adt_batch_s* bt = new (std::nothrow) adt_batch_s();
  ADT_CHECK_ARG(bt != nullptr, ADT_E_ARG, "batch_create: out of host memory");
  batch_dims(bt, sessions, B);
  const size_t need = batch_layout(bt, sessions[0], nullptr);
  if (!workspace || workspace_bytes < need) {
    delete bt;
    set_error("batch_create: workspace %zu < %zu bytes", workspace_bytes, need);
    return ADT_E_CAPACITY;
  }
  batch_layout(bt, sessions[0], (char*)workspace);
  bt->ss.assign(sessions, sessions + B);
  bt->cache_sb = sb;
  *out = bt;
  return ADT_OK;
}

extern "C" void adt_batch_destroy(adt_batch* b) { delete b; }

// The batched GEMM over packed weights, timed like the single-tree projections.
static adt_status gemm_b(const adt_batch_s* bt, const void* X, int ldx, const void* W, int M, int N, int K,
                         hipStream_t st) {
  const int e = prof_pair();
  adt_status r = launch_gemm_nt(X, ldx, W, 0, M, N, K, bt->C, N, st, e >= 0 ? g_prof.ev[e] : nullptr,
                                e >= 0 ? g_prof.ev[e + 1] : nullptr, true, bt->gemm_part, bt->gemm_part_elems);
  prof_done(e, ADT_PROF_GEMM, (double)N * K * 2.0 + (double)M * K * 2.0 + (double)M * N * 4.0, 2.0 * M * N * K);
  return r;
}

// One target forward over the packed rows of every tree: embedding + norm, per layer the
// QKV projection with RoPE and cache append, tree attention per sequence, the output
// projection with residual add and norm, gate/up with SwiGLU, down with residual add and
// norm, then the LM head.  Norm outputs, Q/K/V, attention output and SwiGLU product are
// rounded to bf16 where the single-tree path rounds them; the residual stays fp32.
static adt_status batch_forward(adt_batch_s* bt, int M, int nq_max, hipStream_t st) {
  const adt_session_s* s0 = bt->ss[0];
  const adt_model_s* m = s0->m;
  const int dm = s0->dm, H = s0->H, Dh = s0->Dh, F = s0->F, V = s0->V, dt = s0->dt;
  const float eps = m->d.norm_eps, scale = 1.f / std::sqrt((float)Dh);
  const int64_t stride_h = (int64_t)s0->d.s_cap * Dh;
  TRY(launch_embed_norm(m->d.embed, bt->tok, M, dm, eps, bt->h, bt->a, dt, st));
  for (int l = 0; l < s0->Lr; ++l) {
    char* kc = (char*)s0->d.k_cache + (size_t)l * H * stride_h * 2;
    char* vc = (char*)s0->d.v_cache + (size_t)l * H * stride_h * 2;
    TRY(gemm_b(bt, bt->a, dm, m->qkv[l], M, 3 * dm, dm, st));
    TRY(launch_qkv_rows(bt->C, M, H, Dh, bt->pos, bt->slot, bt->seq, s0->rope, bt->q, kc, vc, stride_h, bt->cache_sb,
                        dt, st));
    const int e = prof_pair();
    TRY(launch_tree_attn(bt->q, kc, vc, bt->cache_sb, stride_h, bt->kv_len, bt->nq, bt->nq, bt->mask,
                         AttnRows{0, 1, 0, bt->row_off}, bt->B, H, Dh, nq_max, s0->d.s_cap, scale, dt, bt->att,
                         bt->attn_ws, bt->attn_ws_bytes, st, e >= 0 ? g_prof.ev[e] : nullptr,
                         e >= 0 ? g_prof.ev[e + 1] : nullptr));
    prof_done(e, ADT_PROF_ATTN, 0.0, 0.0);
    TRY(gemm_b(bt, bt->att, dm, m->o[l], M, dm, dm, st));
    TRY(launch_add_norm(bt->C, 1, M, dm, 0, eps, bt->h, bt->a, dt, st));
    TRY(gemm_b(bt, bt->a, dm, m->gu[l], M, 2 * F, dm, st));
    TRY(launch_swiglu(bt->C, 1, M, F, bt->sw, dt, st));
    TRY(gemm_b(bt, bt->sw, F, m->down[l], M, dm, F, st));
    TRY(launch_add_norm(bt->C, 1, M, dm, 0, eps, bt->h, l + 1 == s0->Lr ? bt->feat : bt->a, dt, st));
  }
  return gemm_b(bt, bt->feat, dm, m->d.lm_head, M, V, dm, st);
}

extern "C" adt_status adt_batch_step(adt_batch* bt, adt_step_out* outs, void* stream) {
  ADT_CHECK_ARG(bt != nullptr && outs != nullptr, ADT_E_ARG, "batch_step: null pointer");
  hipStream_t st = (hipStream_t)stream;
  const int B = bt->B;
  std::vector<int> dh(B, 0), kh(B, 0), n(B, 0), active(B, 0);
  // each session's schedule and draft tree, as in adt_step; the expansions of different
  // sessions run on the auxiliary streams, after everything already on the caller's stream
  TRY(batch_streams(bt));
  constexpr int NS = adt_batch_s::BATCH_STREAMS;
  ADT_HIP(hipEventRecord(bt->ev_fork, st));
  for (int j = 0; j < NS; ++j) ADT_HIP(hipStreamWaitEvent(bt->aux[j], bt->ev_fork, 0));
  adt_status fail = ADT_OK;
  for (int b = 0; b < B && fail == ADT_OK; ++b) {
    adt_session_s* s = bt->ss[b];
    if ((int)s->tokens.size() - s->P >= s->T) continue;
    active[b] = 1;
    hipStream_t sb = bt->aux[b % NS];
    fail = schedule_for(s, dh[b], kh[b]);
    if (fail == ADT_OK)
      fail = dh[b] >= 1 ? adt_tree_expand(s, dh[b], kh[b], s->d.sched.n_budget, nullptr, sb)
                        : set_root_only_tree(s, s->tokens[s->L], s->L, sb);
    n[b] = s->n_nodes;
  }
  // join before anything else (also on failure, so no stream is left ahead of the caller's)
  for (int j = 0; j < NS; ++j) {
    ADT_HIP(hipEventRecord(bt->ev_join[j], bt->aux[j]));
    ADT_HIP(hipStreamWaitEvent(st, bt->ev_join[j], 0));
  }
  if (fail != ADT_OK) return fail;
  // packed rows: tree b at rows [off_b, off_b + n_b); node i at cache slot L_b + i
  std::vector<int32_t> off(B + 1, 0), kv(B, 0), slot, seq;
  int nq_max = 1;
  for (int b = 0; b < B; ++b) {
    off[b + 1] = off[b] + n[b];
    kv[b] = bt->ss[b]->L;
    nq_max = std::max(nq_max, n[b]);
    for (int i = 0; i < n[b]; ++i) {
      slot.push_back(bt->ss[b]->L + i);
      seq.push_back(b);
    }
  }
  const int M = off[B];
  if (M > 0) {
    for (int b = 0; b < B; ++b) {
      if (!n[b]) continue;
      const adt_session_s* s = bt->ss[b];
      ADT_CHECK_ARG(s->L + n[b] <= s->d.s_cap, ADT_E_CAPACITY, "batch_step: cache capacity of session %d", b);
      ADT_HIP(hipMemcpyAsync(bt->tok + off[b], s->tr.token, sizeof(int32_t) * n[b], hipMemcpyDeviceToDevice, st));
      ADT_HIP(hipMemcpyAsync(bt->pos + off[b], s->tr.pos, sizeof(int32_t) * n[b], hipMemcpyDeviceToDevice, st));
      ADT_HIP(hipMemcpyAsync(bt->mask + (size_t)off[b] * ADT_MASK_WORDS, s->tr.mask,
                             sizeof(uint64_t) * ADT_MASK_WORDS * n[b], hipMemcpyDeviceToDevice, st));
    }
    ADT_HIP(hipMemcpyAsync(bt->slot, slot.data(), sizeof(int32_t) * M, hipMemcpyHostToDevice, st));
    ADT_HIP(hipMemcpyAsync(bt->seq, seq.data(), sizeof(int32_t) * M, hipMemcpyHostToDevice, st));
    ADT_HIP(hipMemcpyAsync(bt->row_off, off.data(), sizeof(int32_t) * (B + 1), hipMemcpyHostToDevice, st));
    ADT_HIP(hipMemcpyAsync(bt->kv_len, kv.data(), sizeof(int32_t) * B, hipMemcpyHostToDevice, st));
    ADT_HIP(hipMemcpyAsync(bt->nq, n.data(), sizeof(int32_t) * B, hipMemcpyHostToDevice, st));
    TRY(batch_forward(bt, M, nq_max, st));
  }
  // each session accepts from its own rows: every acceptance first (on the auxiliary streams,
  // after the forward), one synchronisation, then each session commits
  for (int b = 0; b < B; ++b) {
    adt_session_s* s = bt->ss[b];
    if (!active[b]) continue;
    ADT_HIP(hipMemcpyAsync(s->logits, bt->C + (size_t)off[b] * s->V, sizeof(float) * s->V * n[b],
                           hipMemcpyDeviceToDevice, st));
    ADT_HIP(hipMemcpyAsync(s->feat, (char*)bt->feat + (size_t)off[b] * s->dm * 2, (size_t)s->dm * 2 * n[b],
                           hipMemcpyDeviceToDevice, st));
  }
  ADT_HIP(hipEventRecord(bt->ev_fork, st));
  for (int j = 0; j < NS; ++j) ADT_HIP(hipStreamWaitEvent(bt->aux[j], bt->ev_fork, 0));
  for (int b = 0; b < B && fail == ADT_OK; ++b)
    if (active[b]) fail = accept_launch(bt->ss[b], bt->aux[b % NS]);
  for (int j = 0; j < NS; ++j) {
    ADT_HIP(hipEventRecord(bt->ev_join[j], bt->aux[j]));
    ADT_HIP(hipStreamWaitEvent(st, bt->ev_join[j], 0));
  }
  if (fail != ADT_OK) return fail;
  TRY(sync_stream(st));
  for (int b = 0; b < B; ++b) {
    if (!active[b]) {
      memset(&outs[b], 0, sizeof(outs[b]));
      outs[b].done = 1;
      continue;
    }
    TRY(accept_finish(bt->ss[b], dh[b], kh[b], &outs[b], st));
  }
  return ADT_OK;
}

extern "C" adt_status adt_session_set_capture(adt_session* s, const adt_capture* cap) {
  ADT_CHECK_ARG(s != nullptr, ADT_E_ARG, "set_capture: null session");
  const bool on = cap != nullptr && cap->resid != nullptr;
  ADT_CHECK_ARG(!on || cap->meta != nullptr, ADT_E_ARG, "set_capture: metadata buffer missing");
  s->capt_log.clear();
  s->capt_resid = s->capt_xin = s->capt_meta = 0;
  s->capt_cur = -1;
  s->capt_on = on;
  s->capt = on ? *cap : adt_capture{};
  return ADT_OK;
}

extern "C" int32_t adt_session_capture_count(const adt_session* s) { return s ? (int32_t)s->capt_log.size() : 0; }

extern "C" adt_status adt_session_capture_record(const adt_session* s, int32_t i, adt_capture_rec* rec) {
  ADT_CHECK_ARG(s && rec, ADT_E_ARG, "capture_record: null pointer");
  ADT_CHECK_ARG(i >= 0 && i < (int32_t)s->capt_log.size(), ADT_E_ARG, "capture_record: %d of %zu", i,
                s->capt_log.size());
  *rec = s->capt_log[i];
  return ADT_OK;
}

extern "C" adt_status adt_session_get_view(const adt_session* s, adt_session_view* v) {
  ADT_CHECK_ARG(s && v, ADT_E_ARG, "get_view: null pointer");
  v->L = s->L;
  v->Ld = s->Ld;
  v->step = s->step;
  v->n_tokens = (int32_t)s->tokens.size();
  v->n_nodes = s->n_nodes;
  v->logits = s->logits;
  v->feat = s->feat;
  v->draft_logits = s->dlogits;
  v->parent = s->tr.parent;
  v->token = s->tr.token;
  v->depth = s->tr.depth;
  v->score = s->tr.score;
  v->mask = s->tr.mask;
  v->allowed_rows = s->tr.allowed_rows;
  v->path = s->tr.path;
  v->n_acc = s->tr.nacc;
  v->bonus = s->tr.bonus;
  v->tokens_host = s->tokens.data();
  v->q = s->q;
  v->att = s->att;
  v->act = s->act;
  v->resid = s->h;
  v->n_branches = s->nb;
  v->branch_logits = s->rawlog;
  v->draft_branch_logits = s->draw;
  v->logits_lo = s->lm_lo;
  v->logits_hi = s->lm_hi;
  return ADT_OK;
}
