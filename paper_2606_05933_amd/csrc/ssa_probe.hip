// Probe kernels for gfx950: the achievable HBM read rate and bf16 MFMA rate
// (include/ssa_probe.h), against which the library's kernels are measured.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ssa_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kInFlight = 8;  // 16-byte loads per thread before their first use

// Grid-stride over 16-byte chunks, kInFlight per thread per step, XOR-folded.
__global__ __launch_bounds__(kThreads) void hbm_read_kernel(const u32x4* src, size_t chunks,
                                                            uint32_t* out) {
  __shared__ uint32_t part[kThreads / 64];
  const size_t stride = (size_t)gridDim.x * kThreads;
  size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
  u32x4 acc = {0, 0, 0, 0};
  for (; i + (kInFlight - 1) * stride < chunks; i += kInFlight * stride) {
    u32x4 v[kInFlight];
#pragma unroll
    for (int j = 0; j < kInFlight; ++j) v[j] = __builtin_nontemporal_load(src + i + j * stride);
#pragma unroll
    for (int j = 0; j < kInFlight; ++j) acc ^= v[j];
  }
  for (; i < chunks; i += stride) acc ^= src[i];
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

// 16 independent accumulation chains per wave on register operands.
__global__ __launch_bounds__(kThreads) void mfma_bf16_kernel(int iters, float* out) {
  __shared__ float part[kThreads / 64];
  const float s = (float)(threadIdx.x & 7) * 0.125f;
  bf16x8 a, b;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    a[j] = (__bf16)(s + 0.01f * j);
    b[j] = (__bf16)(0.5f - 0.01f * j);
  }
  f32x4 acc[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < 16; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[c], 0, 0, 0);
  }
  float x = 0.f;
#pragma unroll
  for (int c = 0; c < 16; ++c) x += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = part[0] + part[1] + part[2] + part[3];
}

}  // namespace

extern "C" {

int ssa_probe_hbm_read(const void* src, size_t bytes, uint32_t* out, int32_t workgroups,
                       void* stream) {
  if (bytes == 0 || bytes % 16 || workgroups < 1 || workgroups > 65536) return SSA_ERR_ARG;
  if (!src || !out) return SSA_ERR_NULL;
  if ((uintptr_t)src % 16) return SSA_ERR_ARG;
  (void)hipGetLastError();
  hipLaunchKernelGGL(hbm_read_kernel, dim3(workgroups), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(src), bytes / 16,
                     out);
  return hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

int ssa_probe_mfma_bf16(int32_t iters, int32_t workgroups, float* out, void* stream) {
  if (iters < 1 || iters > (1 << 20) || workgroups < 1 || workgroups > 65536) return SSA_ERR_ARG;
  if (!out) return SSA_ERR_NULL;
  (void)hipGetLastError();
  hipLaunchKernelGGL(mfma_bf16_kernel, dim3(workgroups), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), iters, out);
  return hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

}  // extern "C"
