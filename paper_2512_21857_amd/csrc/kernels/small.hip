// Tiny device-side setters: scalars and index arrays are written by kernels that take the
// values as arguments, so a cycle needs no host-to-device copies.
#include "../launch.h"

namespace adt {

__global__ void set_i32_kernel(int32_t* dst, SmallI32 vals, int count) {
  const int i = threadIdx.x;
  if (i < count) dst[i] = vals.v[i];
}

__global__ void fill_pairs_kernel(int32_t* dst, int rows, int lo, int hi) {
  for (int i = threadIdx.x; i < rows; i += blockDim.x) {
    dst[i * 2] = lo;
    dst[i * 2 + 1] = hi;
  }
}

__global__ void iota_kernel(int32_t* dst, int count, int start, int step) {
  for (int i = threadIdx.x; i < count; i += blockDim.x) dst[i] = start + i * step;
}

// Masks of a chain (causal block): row i has bits 0..i.
__global__ void chain_masks_kernel(uint64_t* mask, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    const int b = i + 1;
    mask[i * 2] = b >= 64 ? ~0ull : ((1ull << b) - 1);
    mask[i * 2 + 1] = b <= 64 ? 0ull : (b >= 128 ? ~0ull : ((1ull << (b - 64)) - 1));
  }
}

// The draft's catch-up rows in one launch: tokens from the arguments, feature sources
// 0..cu-1, positions Ld..Ld+cu-1 and the chain masks of cu rows (row i sees rows 0..i).
__global__ void catchup_rows_kernel(SmallI32 tok, int cu, int Ld, int32_t* ctok, int32_t* cfsrc, int32_t* cpos,
                                    uint64_t* cmask) {
  const int i = threadIdx.x;
  if (i >= cu) return;
  ctok[i] = tok.v[i];
  cfsrc[i] = i;
  cpos[i] = Ld + i;
  const int b = i + 1;
  cmask[i * 2] = b >= 64 ? ~0ull : ((1ull << b) - 1);
  cmask[i * 2 + 1] = b <= 64 ? 0ull : (b >= 128 ? ~0ull : ((1ull << (b - 64)) - 1));
}

// Positions, successor allowed ranges and zero scores of a caller-supplied tree.
__global__ void tree_rows_kernel(const int32_t* depth, const int32_t* n_nodes, int n_max, int L, int P, int n_image,
                                 const int32_t* allowed_img, int32_t* pos, int32_t* allowed_rows, float* score) {
  const int n = min(*n_nodes, n_max);
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    pos[i] = L + depth[i];
    int cell = L + depth[i] + 1 - P;
    cell = cell < 0 ? 0 : (cell >= n_image ? n_image - 1 : cell);
    allowed_rows[i * 2] = allowed_img[cell * 2];
    allowed_rows[i * 2 + 1] = allowed_img[cell * 2 + 1];
    score[i] = 0.f;
  }
}

// Row indices of a caller-supplied draft-logit table: (depth * 131 + token) mod rows.
__global__ void table_rows_kernel(const int32_t* tok, int count, int depth, int rows, int32_t* idx) {
  for (int i = threadIdx.x; i < count; i += blockDim.x) idx[i] = (int)(((int64_t)depth * 131 + tok[i]) % rows);
}

adt_status launch_table_rows(const int32_t* tok, int count, int depth, int rows, int32_t* idx, hipStream_t st) {
  table_rows_kernel<<<1, 128, 0, st>>>(tok, count, depth, rows, idx);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

adt_status launch_set_i32(int32_t* dst, const SmallI32& vals, int count, hipStream_t st) {
  ADT_CHECK_ARG(count >= 0 && count <= 32, ADT_E_ARG, "set_i32: count %d", count);
  if (count == 0) return ADT_OK;
  set_i32_kernel<<<1, 32, 0, st>>>(dst, vals, count);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}
adt_status launch_catchup_rows(const SmallI32& tok, int cu, int Ld, int32_t* ctok, int32_t* cfsrc, int32_t* cpos,
                               uint64_t* cmask, hipStream_t st) {
  ADT_CHECK_ARG(cu >= 1 && cu <= 32, ADT_E_ARG, "catchup_rows: %d rows", cu);
  catchup_rows_kernel<<<1, 32, 0, st>>>(tok, cu, Ld, ctok, cfsrc, cpos, cmask);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}
adt_status launch_fill_pairs(int32_t* dst, int rows, int lo, int hi, hipStream_t st) {
  fill_pairs_kernel<<<1, 128, 0, st>>>(dst, rows, lo, hi);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}
adt_status launch_iota(int32_t* dst, int count, int start, int step, hipStream_t st) {
  iota_kernel<<<1, 128, 0, st>>>(dst, count, start, step);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}
adt_status launch_chain_masks(uint64_t* mask, int n, hipStream_t st) {
  chain_masks_kernel<<<1, 128, 0, st>>>(mask, n);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}
adt_status launch_tree_rows(const int32_t* depth, const int32_t* n_nodes, int n_max, int L, int P, int n_image,
                            const int32_t* allowed_img, int32_t* pos, int32_t* allowed_rows, float* score,
                            hipStream_t st) {
  tree_rows_kernel<<<1, 128, 0, st>>>(depth, n_nodes, n_max, L, P, n_image, allowed_img, pos, allowed_rows, score);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

}  // namespace adt
