// HIP kernel for gfx950 converting a value pool between two page layouts
// (include/ssa.h, ssa_v_pool_convert): token-major pages ([num_pages, Hkv, P,
// D]: P slots of D values, the key pool's layout) and the dim-major pages the
// attention kernels read ([num_pages, Hkv, D, P]: D rows of P slots).  A tile
// is one page of one kv head (P x D values).  One workgroup moves 8 KB of
// tiles: 16-byte loads into LDS, a barrier, then each thread gathers the 8
// values of one 16-byte piece of the destination and stores it.  Bytes are
// moved unchanged.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ssa.h"
#include "ssa_device.h"

namespace {
using namespace ssa_dev;

constexpr int kPoolThreads = 256;
constexpr int kPoolWgBytes = 8192;
constexpr int kPieces = kPoolWgBytes / 16 / kPoolThreads;  // 16-byte pieces per thread

template <int D, bool TO_DIM_MAJOR>
__global__ __launch_bounds__(kPoolThreads) void v_pool_convert_kernel(const uint16_t* src,
                                                                      uint16_t* dst,
                                                                      int64_t num_tiles) {
  constexpr int P = SSA_PAGE_SIZE;
  constexpr int TILE = P * D;                         // values per tile
  constexpr int TPW = kPoolWgBytes / (2 * TILE);      // tiles per workgroup
  static_assert(TPW * TILE * 2 == kPoolWgBytes, "whole tiles per workgroup");
  __shared__ __attribute__((aligned(16))) uint16_t lds[TPW * TILE];
  const int64_t tile0 = (int64_t)blockIdx.x * TPW;
  const int ntile = (int)(num_tiles - tile0 < TPW ? num_tiles - tile0 : TPW);
  const int npiece = ntile * TILE / 8;  // 16-byte pieces this workgroup moves
  const uint16_t* s = src + tile0 * TILE;
  uint16_t* d = dst + tile0 * TILE;
  u32x4 v[kPieces];
#pragma unroll
  for (int k = 0; k < kPieces; ++k) {
    const int c = threadIdx.x + k * kPoolThreads;
    if (c < npiece) v[k] = ld16(s + c * 8);
  }
#pragma unroll
  for (int k = 0; k < kPieces; ++k) {
    const int c = threadIdx.x + k * kPoolThreads;
    if (c < npiece) st16(lds + c * 8, v[k]);
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kPieces; ++k) {
    const int c = threadIdx.x + k * kPoolThreads;
    if (c >= npiece) continue;
    const int e0 = c * 8;  // first destination value of the piece (within the workgroup)
    const uint16_t* t = lds + (e0 / TILE) * TILE;
    const int j = e0 % TILE;
    uint16_t e[8];
    if constexpr (TO_DIM_MAJOR) {
      // destination row r, slots s0..s0+7  <-  source slot s, value r at s * D + r
      const int r = j / P, s0 = j % P;
#pragma unroll
      for (int i = 0; i < 8; ++i) e[i] = t[(s0 + i) * D + r];
    } else {
      // destination slot s, values r0..r0+7  <-  source row r, slot s at r * P + s
      const int sl = j / D, r0 = j % D;
#pragma unroll
      for (int i = 0; i < 8; ++i) e[i] = t[(r0 + i) * P + sl];
    }
    u32x4 o;
#pragma unroll
    for (int w = 0; w < 4; ++w) o[w] = (uint32_t)e[2 * w] | ((uint32_t)e[2 * w + 1] << 16);
    st16(d + e0, o);
  }
}

template <int D>
int launch(const uint16_t* src, uint16_t* dst, int64_t num_tiles, bool to_dim_major,
           hipStream_t stream) {
  constexpr int TPW = kPoolWgBytes / (2 * SSA_PAGE_SIZE * D);
  const int64_t grid = (num_tiles + TPW - 1) / TPW;
  if (grid > INT32_MAX) return SSA_ERR_PAGES;
  if (to_dim_major)
    v_pool_convert_kernel<D, true><<<dim3((unsigned)grid), dim3(kPoolThreads), 0, stream>>>(
        src, dst, num_tiles);
  else
    v_pool_convert_kernel<D, false><<<dim3((unsigned)grid), dim3(kPoolThreads), 0, stream>>>(
        src, dst, num_tiles);
  return hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

}  // namespace

extern "C" int ssa_v_pool_convert(const ssa_shape* shape, const uint16_t* src, uint16_t* dst,
                                  int32_t to_dim_major, void* stream) {
  if (!shape || !src || !dst) return SSA_ERR_NULL;
  if (shape->num_kv_heads <= 0) return SSA_ERR_SHAPE;
  if (shape->head_dim != 64 && shape->head_dim != 128) return SSA_ERR_HEAD_DIM;
  if (shape->page_size != SSA_PAGE_SIZE) return SSA_ERR_PAGE_SIZE;
  if (shape->num_pages < 1) return SSA_ERR_PAGES;
  if (to_dim_major != 0 && to_dim_major != 1) return SSA_ERR_ARG;
  const uintptr_t a = reinterpret_cast<uintptr_t>(src), b = reinterpret_cast<uintptr_t>(dst);
  if ((a | b) % 16) return SSA_ERR_ARG;
  const int64_t num_tiles = (int64_t)shape->num_pages * shape->num_kv_heads;
  const uint64_t bytes = (uint64_t)num_tiles * SSA_PAGE_SIZE * shape->head_dim * 2;
  if (a < b + bytes && b < a + bytes) return SSA_ERR_ARG;  // the two pools overlap
  hipStream_t s = static_cast<hipStream_t>(stream);
  return shape->head_dim == 128 ? launch<128>(src, dst, num_tiles, to_dim_major, s)
                                : launch<64>(src, dst, num_tiles, to_dim_major, s);
}
