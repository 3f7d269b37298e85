// Probe kernels for gfx950: the achievable HBM read rate (a linear stream and a
// gather of whole chunks) and bf16 MFMA rate (include/ssa_probe.h), against
// which the library's kernels are measured.
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

// Gather: each wave reads kGatherLoads 1 KB rows per step, made of whole
// chunks of LPC rows (LPC KB each) at the positions the index array names, in
// the index array's order (wave w takes chunks w * CPS .., then a grid stride).
// Indices are clamped into the buffer; past the end of the array a wave
// re-reads the last chunk, so its step stays whole.
constexpr int kGatherLoads = 16;  // 16 KB in flight per wave per step
// KEY_ROWS (4 KB chunks only): each load instruction reads 64 B of each of 16
// rows of 256 B instead of one whole 1 KB row, the attention kernel's key-row
// pattern (lane l: row l % 16, bytes 16 (l / 16) .. of the instruction's 64).
template <int LPC, bool KEY_ROWS = false>
__global__ __launch_bounds__(kThreads) void hbm_gather_kernel(const uint8_t* src, int64_t src_chunks,
                                                              const int32_t* index, int32_t n,
                                                              uint32_t* out) {
  constexpr int CPS = kGatherLoads / LPC;
  __shared__ uint32_t part[kThreads / 64];
  const int lane = threadIdx.x & 63;
  const int wave = blockIdx.x * (kThreads / 64) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int waves = gridDim.x * (kThreads / 64);
  u32x4 acc = {0, 0, 0, 0};
  for (int64_t c0 = (int64_t)wave * CPS; c0 < n; c0 += (int64_t)waves * CPS) {
    u32x4 v[kGatherLoads];
#pragma unroll
    for (int k = 0; k < CPS; ++k) {
      const int64_t c = c0 + k < n ? c0 + k : n - 1;
      int64_t id = index[c];
      id = id < 0 ? 0 : (id >= src_chunks ? src_chunks - 1 : id);
      const uint8_t* chunk = src + id * (LPC * 1024);
#pragma unroll
      for (int j = 0; j < LPC; ++j) {
        const int off = KEY_ROWS ? (lane & 15) * 256 + j * 64 + (lane >> 4) * 16 : j * 1024 + lane * 16;
        v[k * LPC + j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(chunk + off));
      }
    }
#pragma unroll
    for (int j = 0; j < kGatherLoads; ++j) acc ^= v[j];
  }
  uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o, 64);
  if (lane == 0) part[threadIdx.x >> 6] = x;
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

int ssa_probe_hbm_gather(const void* src, size_t src_bytes, const int32_t* chunk_index,
                         int32_t n_chunks, int32_t chunk_bytes, int32_t pattern, uint32_t* out,
                         int32_t workgroups, void* stream) {
  if (chunk_bytes != 1024 && chunk_bytes != 2048 && chunk_bytes != 4096 && chunk_bytes != 8192 &&
      chunk_bytes != 16384)
    return SSA_ERR_ARG;
  if (pattern != 0 && !(pattern == 1 && chunk_bytes == 4096)) return SSA_ERR_ARG;
  if (n_chunks < 1 || workgroups < 1 || workgroups > 65536 || src_bytes < (size_t)chunk_bytes)
    return SSA_ERR_ARG;
  if (!src || !chunk_index || !out) return SSA_ERR_NULL;
  if ((uintptr_t)src % 16) return SSA_ERR_ARG;
  (void)hipGetLastError();
  const int64_t src_chunks = (int64_t)(src_bytes / (size_t)chunk_bytes);
  const uint8_t* s = static_cast<const uint8_t*>(src);
  hipStream_t st = static_cast<hipStream_t>(stream);
  const dim3 grid(workgroups), block(kThreads);
  switch (chunk_bytes) {
    case 1024: hipLaunchKernelGGL(hbm_gather_kernel<1>, grid, block, 0, st, s, src_chunks, chunk_index, n_chunks, out); break;
    case 2048: hipLaunchKernelGGL(hbm_gather_kernel<2>, grid, block, 0, st, s, src_chunks, chunk_index, n_chunks, out); break;
    case 4096:
      if (pattern == 1)
        hipLaunchKernelGGL((hbm_gather_kernel<4, true>), grid, block, 0, st, s, src_chunks, chunk_index, n_chunks, out);
      else
        hipLaunchKernelGGL(hbm_gather_kernel<4>, grid, block, 0, st, s, src_chunks, chunk_index, n_chunks, out);
      break;
    case 8192: hipLaunchKernelGGL(hbm_gather_kernel<8>, grid, block, 0, st, s, src_chunks, chunk_index, n_chunks, out); break;
    default: hipLaunchKernelGGL(hbm_gather_kernel<16>, grid, block, 0, st, s, src_chunks, chunk_index, n_chunks, out); break;
  }
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
