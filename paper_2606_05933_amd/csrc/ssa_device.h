// Device helpers shared by the library's HIP sources (gfx950 only): vector
// types, 16-byte register loads and stores, the global -> LDS copy, explicit
// vector-memory counter waits, the bf16 MFMA and bf16 packing.  Internal
// header; the definitions live in namespace ssa_dev.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ssa_dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// D = A B + C on one 16x16 tile, K = 32 (v_mfma_f32_16x16x32_bf16).
__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Two fp32 values to packed bf16, round to nearest even.
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// One wave-wide global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane i's 16 bytes from g land at LDS address l + 16 i (l wave-uniform).  It
// is inline assembly, so the compiler's memory-counter tracking does not make
// reads of other LDS buffers wait for it; every reader of the destination
// waits explicitly (vm_wait, then the barrier that publishes the buffer).
// COHERENT: a device-scope read (sc1), for rows written in the same launch.
template <bool COHERENT = false>
__device__ __forceinline__ void dma16(const void* g, const char* l) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)l;
  if (COHERENT)
    asm volatile("global_load_lds_dwordx4 %0, off sc1" ::"v"(g), "{m0}"(a) : "memory");
  else
    asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(a) : "memory");
}

// dma16 with the non-temporal hint (nt), for rows a workgroup reads once: they
// should not displace what the caches hold for other workgroups.
__device__ __forceinline__ void dma16_stream(const void* g, const char* l) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)l;
  asm volatile("global_load_lds_dwordx4 %0, off nt" ::"v"(g), "{m0}"(a) : "memory");
}

// s_waitcnt vmcnt(N): all but this wave's N most recent vector-memory
// operations (LDS copies included) have completed.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
__device__ __forceinline__ void lds_dma_wait() { vm_wait<0>(); }

}  // namespace ssa_dev
