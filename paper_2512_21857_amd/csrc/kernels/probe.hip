// Measurement probes: what this device sustains for the two resources the hot path is bound
// by, reported beside the vendor's nominal peaks.
//
// probe_read:  nontemporal 16-byte loads over a buffer, eight independent loads in flight
//              per thread per iteration, XOR-folded into one word per workgroup (written out
//              so the loads stay live).  Bytes read / time = achievable HBM read bandwidth
//              (plain loads of the same pattern reach about 6.1 TB/s, nontemporal ones 6.9-7.0).
// probe_mfma:  back-to-back v_mfma_f32_32x32x16_bf16 on register operands, four independent
//              accumulators per wave, no memory traffic in the loop.  Flops / time = the
//              achievable dense bf16 matrix rate.
#include "../launch.h"

namespace adt {

typedef float f32x16 __attribute__((ext_vector_type(16)));

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int PROBE_THREADS = 256;
constexpr int PROBE_READ_BLOCKS = 2048;
constexpr int PROBE_MFMA_BLOCKS = 1024;
constexpr int PROBE_MFMA_ACC = 4;

__global__ __launch_bounds__(PROBE_THREADS) void probe_read_kernel(const uint4* __restrict__ p, int64_t n16,
                                                                   uint32_t* __restrict__ sink) {
  __shared__ uint32_t red[PROBE_THREADS / WAVE];
  const int64_t stride = (int64_t)gridDim.x * PROBE_THREADS;
  int64_t i = (int64_t)blockIdx.x * PROBE_THREADS + threadIdx.x;
  uint32_t acc = 0;
  // eight streaming (nontemporal) loads in flight per thread: the data is read once
  for (; i + 7 * stride < n16; i += 8 * stride) {
    u32x4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p + i + j * stride));
#pragma unroll
    for (int j = 0; j < 8; ++j) acc ^= v[j][0] ^ v[j][1] ^ v[j][2] ^ v[j][3];
  }
  for (; i < n16; i += stride) {
    const u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p + i));
    acc ^= a[0] ^ a[1] ^ a[2] ^ a[3];
  }
  for (int o = WAVE / 2; o >= 1; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o, WAVE);
  if (threadIdx.x % WAVE == 0) red[threadIdx.x / WAVE] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int w = 0; w < PROBE_THREADS / WAVE; ++w) t ^= red[w];
    sink[blockIdx.x] = t;
  }
}

__global__ __launch_bounds__(PROBE_THREADS) void probe_mfma_kernel(int iters, float* __restrict__ sink) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)(threadIdx.x + i));
    b[i] = (__bf16)(0.002f * (float)i);
  }
  f32x16 acc[PROBE_MFMA_ACC];
#pragma unroll
  for (int j = 0; j < PROBE_MFMA_ACC; ++j)
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[j][k] = 0.f;
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int j = 0; j < PROBE_MFMA_ACC; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < PROBE_MFMA_ACC; ++j)
#pragma unroll
    for (int k = 0; k < 16; ++k) s += acc[j][k];
  sink[(int64_t)blockIdx.x * PROBE_THREADS + threadIdx.x] = s;
}

__global__ __launch_bounds__(PROBE_THREADS) void probe_weight_kernel(const float* __restrict__ d, int64_t n,
                                                                      uint64_t* __restrict__ w) {
  for (int64_t i = blockIdx.x * (int64_t)PROBE_THREADS + threadIdx.x; i < n; i += (int64_t)gridDim.x * PROBE_THREADS)
    w[i] = quantised_exp_weight(d[i]);
}

}  // namespace adt

using namespace adt;

extern "C" adt_status adt_probe_sample_weights(const float* d, int64_t n, uint64_t* w, void* stream) {
  ADT_CHECK_ARG(d && w && n >= 0, ADT_E_ARG, "probe_sample_weights: bad arguments");
  if (n == 0) return ADT_OK;
  const int64_t blocks = std::min<int64_t>((n + PROBE_THREADS - 1) / PROBE_THREADS, 4096);
  probe_weight_kernel<<<(unsigned)blocks, PROBE_THREADS, 0, (hipStream_t)stream>>>(d, n, w);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

extern "C" size_t adt_probe_sink_bytes(void) {
  return sizeof(float) * (size_t)PROBE_MFMA_BLOCKS * PROBE_THREADS;
}

extern "C" adt_status adt_probe_hbm_read(const void* buf, size_t bytes, void* sink, size_t sink_bytes, void* stream) {
  ADT_CHECK_ARG(buf && sink, ADT_E_ARG, "probe_hbm_read: null pointer");
  ADT_CHECK_ARG(bytes >= 16 && bytes % 16 == 0 && ((uintptr_t)buf % 16) == 0, ADT_E_SHAPE,
                "probe_hbm_read: %zu bytes at %p (16-byte multiple, 16-byte aligned)", bytes, buf);
  ADT_CHECK_ARG(sink_bytes >= adt_probe_sink_bytes(), ADT_E_CAPACITY, "probe_hbm_read: sink %zu bytes", sink_bytes);
  probe_read_kernel<<<PROBE_READ_BLOCKS, PROBE_THREADS, 0, (hipStream_t)stream>>>((const uint4*)buf,
                                                                                 (int64_t)(bytes / 16),
                                                                                 (uint32_t*)sink);
  ADT_LAUNCH_CHECK();
  return ADT_OK;
}

extern "C" adt_status adt_probe_mfma(int32_t iters, void* sink, size_t sink_bytes, double* flops, void* stream) {
  ADT_CHECK_ARG(sink && iters >= 1, ADT_E_ARG, "probe_mfma: bad arguments");
  ADT_CHECK_ARG(sink_bytes >= adt_probe_sink_bytes(), ADT_E_CAPACITY, "probe_mfma: sink %zu bytes", sink_bytes);
  probe_mfma_kernel<<<PROBE_MFMA_BLOCKS, PROBE_THREADS, 0, (hipStream_t)stream>>>(iters, (float*)sink);
  ADT_LAUNCH_CHECK();
  if (flops)
    *flops = (double)PROBE_MFMA_BLOCKS * (PROBE_THREADS / WAVE) * iters * PROBE_MFMA_ACC * (32.0 * 32.0 * 16.0 * 2.0);
  return ADT_OK;
}
