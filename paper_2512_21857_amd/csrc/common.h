// Shared device/host helpers of the ADT-Tree HIP library (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/adt.h"

namespace adt {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;   // an LDS operand of a transpose load

constexpr int WAVE = 64;
constexpr float LOG2E = 1.4426950408889634f;

// float -> bfloat16 bits, round to nearest even (gfx950 converts in hardware,
// v_cvt_pk_bf16_f32, two values per instruction when paired).
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ static __forceinline__ float load(const float* p, int64_t i) { return p[i]; }
  __device__ static __forceinline__ void store(float* p, int64_t i, float v) { p[i] = v; }
};
template <> struct Elem<uint16_t> {
  __device__ static __forceinline__ float load(const uint16_t* p, int64_t i) { return bf2f(p[i]); }
  __device__ static __forceinline__ void store(uint16_t* p, int64_t i, float v) { p[i] = f2bf(v); }
};
// Four consecutive values at p (aligned to four elements): one vector store.
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
}
__device__ __forceinline__ void store4(uint16_t* p, float a, float b, float c, float d) {
  *reinterpret_cast<u16x4*>(p) = u16x4{f2bf(a), f2bf(b), f2bf(c), f2bf(d)};
}

// Fragment layout of a bf16 activation matrix (rows r < 16 pk, K columns, K % 32 == 0): the
// 16 x 32 block (r / 16, k / 32) is 1 KB contiguous in the order a wave hands it to the
// 16x16x32 MFMA as its B operand (lane (r % 16) + 16 ((k % 32) / 8) holds 8 consecutive
// columns), and blocks follow each other row block fastest: block (k / 32) pk + r / 16.  A
// wave then reads a block with one contiguous 16-byte load per lane, where the row-major
// layout needs sixteen half-used 128-byte lines.  pk = 0 selects row-major with leading
// dimension ld.  Runs of up to 8 columns starting at a multiple of their length stay
// contiguous in both layouts.
__host__ __device__ __forceinline__ int64_t frag_index(int64_t r, int k, int pk) {
  return (((int64_t)(k >> 5) * pk + (r >> 4)) * 64 + (r & 15) + ((k & 31) >> 3) * 16) * 8 + (k & 7);
}
__host__ __device__ __forceinline__ int64_t act_index(int64_t r, int k, int64_t ld, int pk) {
  return pk ? frag_index(r, k, pk) : r * ld + k;
}

// Debug builds (ADT_DEVICE_CHECKS=1) test invariants of device-side inputs; a kernel that finds
// one broken sets its bit in the error word of its source file and goes on within bounds.
#ifndef ADT_DEVICE_CHECKS
#define ADT_DEVICE_CHECKS 0
#endif
enum : uint32_t {
  DEVINV_PARENT = 1u,     // parent[0] != -1 or parent[i] outside [0, i)
  DEVINV_KV_RANGE = 2u,   // kv_len + n beyond the cache capacity
  DEVINV_PATH = 4u,       // an accepted-path entry outside the tree
};
// One error word per source file (each file is its own device code object): file-scope
// `dev_err_word`, set by dev_fail, read and cleared by the file's dev_errors_take_*.
#define ADT_DEVICE_ERROR_WORD(tag)                                                               \
  static __device__ uint32_t dev_err_word;                                                       \
  __device__ __forceinline__ void dev_fail(uint32_t bit) {                                       \
    if (ADT_DEVICE_CHECKS) atomicOr(&dev_err_word, bit);                                         \
  }                                                                                              \
  uint32_t dev_errors_take_##tag() {                                                             \
    if (!ADT_DEVICE_CHECKS) return 0;                                                            \
    void* p = nullptr;                                                                           \
    uint32_t v = 0;                                                                              \
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(dev_err_word)) != hipSuccess || !p) return 0x80000000u; \
    if (hipMemcpy(&v, p, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess) return 0x80000000u;    \
    if (v && hipMemset(p, 0, sizeof(v)) != hipSuccess) return 0x80000000u;                        \
    return v;                                                                                    \
  }

// Philox4x32-10 (Salmon et al., SC'11): ten rounds over counter (c0..c3) with key (k0, k1);
// host and device share it (acceptance draws on the GPU, the Random tree initialisation on
// the host).
__host__ __device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)M0 * c[0], p1 = (uint64_t)M1 * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0, n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = (uint32_t)p1;
    c[2] = n2;
    c[3] = (uint32_t)p0;
    k0 += W0;
    k1 += W1;
  }
}

// One butterfly step over lanes l ^ 32 or l ^ 16 on gfx950's lane-swap instructions (VALU,
// no LDS round trip): the swap of a value with itself leaves x[l] and x[l ^ 32] (x[l ^ 16])
// in the two results, in an order that depends on the lane, so only a commutative combine of
// the two is taken (it equals x[l] op x[l ^ m] exactly).
__device__ __forceinline__ float xor32_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor16_max(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_add(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor16_add(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Sampling weight w = rint(exp(d) * 2^32) of a float32 exponent d = z - max z <= 0, with
// exp(d) evaluated by a fixed sequence of IEEE double operations and no fused multiply-add,
// so that any implementation following the same sequence gets the same integer: y = d log2(e),
// k = floor(y), f = y - k, 2^f by Horner's rule over the doubles nearest ln(2)^j / j!
// (j = 13 .. 0), exp(d) = 2^f 2^k; d < -40 gives 0 (exp(d) 2^32 < 2^-25 there).
__device__ inline uint64_t quantised_exp_weight(float d) {
#pragma clang fp contract(off)
  if (!(d >= -40.f)) return 0;
  const double y = (double)d * 0x1.71547652b82fep+0;
  const double k = floor(y);
  const double f = y - k;
  double p = 0x1.816193166d0f9p-40;
  p = p * f + 0x1.c3bd650fc2986p-36;
  p = p * f + 0x1.e8cac7351bb25p-32;
  p = p * f + 0x1.e4cf5158b8ecap-28;
  p = p * f + 0x1.b5253d395e7c4p-24;
  p = p * f + 0x1.62c0223a5c824p-20;
  p = p * f + 0x1.ffcbfc588b0c7p-17;
  p = p * f + 0x1.430912f86c787p-13;
  p = p * f + 0x1.5d87fe78a6731p-10;
  p = p * f + 0x1.3b2ab6fba4e77p-7;
  p = p * f + 0x1.c6b08d704a0c0p-5;
  p = p * f + 0x1.ebfbdff82c58fp-3;
  p = p * f + 0x1.62e42fefa39efp-1;
  p = p * f + 0x1.0p+0;
  return (uint64_t)rint(ldexp(p, (int)k + 32));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 (<= 1024); `red` holds >= 16 floats.
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, nw = blockDim.x / WAVE;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}

}  // namespace adt

// ----------------------------------------------------------------------------- host side
namespace adt {
void set_error(const char* fmt, ...);
}

#define ADT_CHECK_ARG(cond, code, ...)        \
  do {                                        \
    if (!(cond)) {                            \
      adt::set_error(__VA_ARGS__);            \
      return (code);                          \
    }                                         \
  } while (0)

#define ADT_HIP(call)                                                                 \
  do {                                                                                \
    hipError_t e_ = (call);                                                           \
    if (e_ != hipSuccess) {                                                           \
      adt::set_error("HIP error %s at %s:%d", hipGetErrorString(e_), __FILE__, __LINE__); \
      return ADT_E_HIP;                                                               \
    }                                                                                 \
  } while (0)

#define ADT_LAUNCH_CHECK() ADT_HIP(hipGetLastError())
