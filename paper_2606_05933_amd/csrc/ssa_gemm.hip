// HIP kernels for gfx950 of the dense steps of a transformer layer
// (include/ssa_layer.h): the linear layers as one MFMA GEMM with fused
// epilogues, and RMSNorm.
//
// ssa_linear: out = x W^T, x [M, K] and W [N, K] bf16, both K-contiguous (the
// torch Linear layout), fp32 accumulation.
//  * One workgroup (4 waves, 2 x 2) per 128 x 128 output tile and K range; each
//    wave owns 64 x 64 = 4 x 4 v_mfma_f32_16x16x32_bf16 tiles, with W as the A
//    operand (MFMA rows = output columns n) and x as the B operand (MFMA columns
//    = tokens), so a lane ends with 4 consecutive n of one token: one 8-byte
//    store per tile.
//  * K blocks of 64 are copied global -> LDS without registers
//    (global_load_lds_dwordx4) into a ring of STAGES stages, STAGES - 1 blocks
//    ahead; one barrier per block.  LDS rows are 128 bytes; the 16-byte chunk c
//    of row r sits at chunk c ^ (r & 7), so the 16 rows one ds_read_b128 reads
//    fall on 8 distinct chunk slots per lane octet (no bank conflict).
//  * Rows of x past M are read from row M - 1 (in bounds) and never stored.
//  * Too few tiles to fill the chip: K is split; each split writes its fp32
//    tile with device-scope stores, takes a ticket, and the last one adds the
//    splits in split order (the result does not depend on arrival order),
//    applies the epilogue and resets the ticket.
//  * Work ids are laid out so that consecutive ids (the M tiles of one N tile,
//    which read the same W panel) run on one XCD and share its L2.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/ssa_layer.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kStageBytes = (BM + BN) * BK * 2;       // 32 KB: x rows, then W rows
constexpr int kLoads = kStageBytes / 1024 / 4;        // 1 KB copies per wave per stage
constexpr int kTileFloats = BM * BN;
constexpr int kXcds = 8;
constexpr float kLog2e = 1.4426950408889634f;

// One wave-wide global -> LDS copy: lane i's 16 bytes from g land at l + 16 i
// (l wave-uniform).  Readers wait for it explicitly (vm_wait, then a barrier).
__device__ __forceinline__ void dma16(const void* g, const char* l) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)l;
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(a) : "memory");
}
// s_waitcnt vmcnt(N): all but this wave's N most recent vector-memory
// operations have completed.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
__device__ __forceinline__ f32x4 mfma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Split partials cross workgroups and XCDs (whose L2s are not coherent with
// each other): device-scope 8-byte stores and loads, a device-scope ticket.
__device__ __forceinline__ void st16_dev(float* p, f32x4 v) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  const uint64_t lo = (uint64_t)__float_as_uint(v[0]) | ((uint64_t)__float_as_uint(v[1]) << 32);
  const uint64_t hi = (uint64_t)__float_as_uint(v[2]) | ((uint64_t)__float_as_uint(v[3]) << 32);
  __hip_atomic_store(q, lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ f32x4 ld16_dev(const float* p) {
  uint64_t* q = reinterpret_cast<uint64_t*>(const_cast<float*>(p));
  const uint64_t lo = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t hi = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return f32x4{__uint_as_float((uint32_t)lo), __uint_as_float((uint32_t)(lo >> 32)),
               __uint_as_float((uint32_t)hi), __uint_as_float((uint32_t)(hi >> 32))};
}

// silu(z) = z / (1 + e^-z), with e^-z as 2^(-z log2 e)
__device__ __forceinline__ float silu(float z) {
  return z * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-z * kLog2e));
}

struct GemmArgs {
  const uint16_t* x;
  const uint16_t* w;
  const uint16_t* res;
  uint16_t* out;
  int* tickets;
  float* part;
  int m, n, k;
  int tiles_m, tiles_n, splits, kbps, kblocks;
};

// Wait until at most `left` K blocks (kLoads copies each) of this wave are in flight.
template <int STAGES>
__device__ __forceinline__ void wait_blocks(int left) {
  if (STAGES >= 4 && left >= 2) vm_wait<2 * kLoads>();
  else if (STAGES >= 3 && left >= 1) vm_wait<kLoads>();
  else vm_wait<0>();
}

template <int STAGES, int EPI>
__global__ __launch_bounds__(kThreads, STAGES <= 2 ? 2 : 1) void linear_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) char lds[STAGES * kStageBytes];
  __shared__ int s_last;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int r16 = lane & 15, g = lane >> 4;

  // work id: consecutive ids on one XCD (dispatch goes round-robin over XCDs)
  const int total = (int)gridDim.x, xcd = (int)blockIdx.x % kXcds, local = (int)blockIdx.x / kXcds;
  const int per = total / kXcds, rem = total % kXcds;
  const int wid = xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
  const int tm = wid % a.tiles_m;
  const int tn = (wid / a.tiles_m) % a.tiles_n;
  const int split = wid / (a.tiles_m * a.tiles_n);
  const int m0 = tm * BM, n0 = tn * BN;
  const int kb0 = split * a.kbps;
  const int nkb = min(a.kbps, a.kblocks - kb0);

  // Copy r of this wave fills 1 KB piece p = 4 r + w of a stage: pieces 0..15
  // hold x rows 8p..8p+7, pieces 16..31 W rows; lane i fetches the chunk that
  // belongs at its LDS slot (row 8p + i / 8, slot i % 8).
  const uint16_t* src[kLoads];
#pragma unroll
  for (int r = 0; r < kLoads; ++r) {
    const int p = r * 4 + w;
    const int row = (p & 15) * 8 + (lane >> 3);
    const int chunk = (lane & 7) ^ (lane >> 3);
    if (p < 16)
      src[r] = a.x + (size_t)min(m0 + row, a.m - 1) * a.k + (size_t)kb0 * BK + chunk * 8;
    else
      src[r] = a.w + (size_t)(n0 + row) * a.k + (size_t)kb0 * BK + chunk * 8;
  }
  auto issue = [&](int i) {
    const char* st = lds + (i % STAGES) * kStageBytes;
#pragma unroll
    for (int r = 0; r < kLoads; ++r) dma16(src[r] + (size_t)i * BK, st + (r * 4 + w) * 1024);
  };

  // fragment reads: row r16 of a 16-row tile, logical chunk 4 ks + g
  const int xoff = (wm * 64 + r16) * 128;
  const int woff = BM * 128 + (wn * 64 + r16) * 128;
  const int c0 = (g ^ (r16 & 7)) << 4, c1 = ((4 + g) ^ (r16 & 7)) << 4;

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int i = 0; i < STAGES - 1; ++i)
    if (i < nkb) issue(i);
  for (int i = 0; i < nkb; ++i) {
    wait_blocks<STAGES>(min(nkb - 1 - i, STAGES - 2));
    __syncthreads();  // block i has landed for every wave; stage (i - 1) % STAGES is free
    if (i + STAGES - 1 < nkb) issue(i + STAGES - 1);
    const char* st = lds + (i % STAGES) * kStageBytes;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c = ks ? c1 : c0;
      bf16x8 xf[4], wf[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        xf[t] = as_bf16x8(ld16(st + xoff + t * 2048 + c));
        wf[t] = as_bf16x8(ld16(st + woff + t * 2048 + c));
      }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) acc[mt][nt] = mfma(wf[nt], xf[mt], acc[mt][nt]);
    }
  }

  // 16-token tiles of this wave that hold rows < M (wave-uniform)
  const int nmt = max(0, min(4, (a.m - (m0 + wm * 64) + 15) / 16));
  if (a.splits > 1) {
    const int tile = tn * a.tiles_m + tm;
    float* mine = a.part + ((size_t)tile * a.splits + split) * kTileFloats + w * 4096 + lane * 4;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
      if (mt < nmt)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) st16_dev(mine + (mt * 4 + nt) * 256, acc[mt][nt]);
    vm_wait<0>();  // this thread's device-scope stores have completed
    __syncthreads();
    if (tid == 0) {
      const int prev =
          __hip_atomic_fetch_add(&a.tickets[tile], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == a.splits - 1);
    }
    __syncthreads();
    if (!s_last) return;
    const float* base = a.part + (size_t)tile * a.splits * kTileFloats + w * 4096 + lane * 4;
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      if (mt >= nmt) continue;
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        f32x4 sum = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < a.splits; ++s)
          sum += (s == split) ? acc[mt][nt] : ld16_dev(base + (size_t)s * kTileFloats + (mt * 4 + nt) * 256);
        acc[mt][nt] = sum;
      }
    }
    if (tid == 0) __hip_atomic_store(&a.tickets[tile], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // epilogue: lane holds n = nbase + 4 g .. + 3 of token m0 + wm 64 + 16 mt + r16
#pragma unroll
  for (int mt = 0; mt < 4; ++mt) {
    if (mt >= nmt) continue;
    const int tok = m0 + wm * 64 + mt * 16 + r16;
    if (tok >= a.m) continue;
    if (EPI == SSA_EPILOGUE_SWIGLU) {
      // W rows in 16-row blocks, gate block then up block of the same 16 outputs
      const int nout = a.n / 2;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const f32x4 gt = acc[mt][2 * j], up = acc[mt][2 * j + 1];
        const int col = (n0 + wn * 64) / 2 + j * 16 + g * 4;
        u32x2 v = {pack2(silu(gt[0]) * up[0], silu(gt[1]) * up[1]),
                   pack2(silu(gt[2]) * up[2], silu(gt[3]) * up[3])};
        *reinterpret_cast<u32x2*>(a.out + (size_t)tok * nout + col) = v;
      }
    } else {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int col = n0 + wn * 64 + nt * 16 + g * 4;
        f32x4 v = acc[mt][nt];
        if (EPI == SSA_EPILOGUE_RESIDUAL) {
          const u32x2 r = *reinterpret_cast<const u32x2*>(a.res + (size_t)tok * a.n + col);
          v[0] += bf16_lo(r[0]);
          v[1] += bf16_hi(r[0]);
          v[2] += bf16_lo(r[1]);
          v[3] += bf16_hi(r[1]);
        }
        *reinterpret_cast<u32x2*>(a.out + (size_t)tok * a.n + col) =
            u32x2{pack2(v[0], v[1]), pack2(v[2], v[3])};
      }
    }
  }
}

// RMSNorm: one workgroup per row, up to 4 16-byte chunks per thread.
constexpr int kNormChunks = 4;
__global__ __launch_bounds__(kThreads) void rms_norm_kernel(const uint16_t* x, const uint16_t* wt,
                                                            uint16_t* out, int n, float eps) {
  __shared__ float s_part[kThreads / 64];
  const int tid = threadIdx.x;
  const uint16_t* row = x + (size_t)blockIdx.x * n;
  u32x4 v[kNormChunks];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < kNormChunks; ++c) {
    const int e = (c * kThreads + tid) * 8;
    v[c] = e < n ? ld16(row + e) : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float lo = bf16_lo(v[c][j]), hi = bf16_hi(v[c][j]);
      ss += lo * lo + hi * hi;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if ((tid & 63) == 0) s_part[tid >> 6] = ss;
  __syncthreads();
  const float tot = s_part[0] + s_part[1] + s_part[2] + s_part[3];
  const float rs = __builtin_amdgcn_rsqf(tot / (float)n + eps);
#pragma unroll
  for (int c = 0; c < kNormChunks; ++c) {
    const int e = (c * kThreads + tid) * 8;
    if (e >= n) continue;
    const u32x4 wv = ld16(wt + e);
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = pack2(bf16_lo(v[c][j]) * rs * bf16_lo(wv[j]), bf16_hi(v[c][j]) * rs * bf16_hi(wv[j]));
    *reinterpret_cast<u32x4*>(out + (size_t)blockIdx.x * n + e) = o;
  }
}

constexpr int kStages = 3;
constexpr int kTargetWgs = 512;

struct GemmCfg {
  int tiles_m, tiles_n, splits, kbps, kblocks;
  size_t ws;
};

GemmCfg gemm_cfg(int m, int n, int k) {
  GemmCfg c;
  c.tiles_m = (m + BM - 1) / BM;
  c.tiles_n = n / BN;
  c.kblocks = k / BK;
  const int tiles = c.tiles_m * c.tiles_n;
  int s = 1;
  if (tiles < kTargetWgs / 2) s = (kTargetWgs + tiles - 1) / tiles;
  s = std::max(1, std::min(s, c.kblocks / 4));  // at least 4 K blocks per split
  c.kbps = (c.kblocks + s - 1) / s;
  c.splits = (c.kblocks + c.kbps - 1) / c.kbps;
  const size_t tickets = ((size_t)tiles * 4 + 255) / 256 * 256;
  c.ws = c.splits > 1 ? tickets + (size_t)tiles * c.splits * kTileFloats * 4 : 0;
  return c;
}

int check_linear(int32_t m, int32_t n, int32_t k, int32_t epilogue) {
  if (m < 0 || n <= 0 || k <= 0 || n % BN || k % BK) return SSA_ERR_ARG;
  if (epilogue < SSA_EPILOGUE_NONE || epilogue > SSA_EPILOGUE_SWIGLU) return SSA_ERR_ARG;
  if ((int64_t)m * k > INT64_C(1) << 40 || (int64_t)n * k > INT64_C(1) << 40) return SSA_ERR_ARG;
  return SSA_OK;
}

}  // namespace

extern "C" {

int ssa_linear_workspace_size(int32_t m, int32_t n, int32_t k, size_t* ws_bytes) {
  if (!ws_bytes) return SSA_ERR_NULL;
  const int rc = check_linear(m, n, k, SSA_EPILOGUE_NONE);
  if (rc) return rc;
  *ws_bytes = m == 0 ? 0 : gemm_cfg(m, n, k).ws;
  return SSA_OK;
}

int ssa_linear(int32_t m, int32_t n, int32_t k, int32_t epilogue, const uint16_t* x,
               const uint16_t* w, const uint16_t* residual, uint16_t* out, void* workspace,
               size_t ws_bytes, void* stream) {
  const int rc = check_linear(m, n, k, epilogue);
  if (rc) return rc;
  if (m == 0) return SSA_OK;
  if (!x || !w || !out || (epilogue == SSA_EPILOGUE_RESIDUAL && !residual)) return SSA_ERR_NULL;
  const GemmCfg c = gemm_cfg(m, n, k);
  if (c.ws > 0 && (!workspace || ws_bytes < c.ws)) return SSA_ERR_WORKSPACE;
  const size_t tickets = ((size_t)c.tiles_m * c.tiles_n * 4 + 255) / 256 * 256;
  GemmArgs a{x, w, residual, out,
             static_cast<int*>(workspace),
             c.ws > 0 ? reinterpret_cast<float*>(static_cast<char*>(workspace) + tickets) : nullptr,
             m, n, k, c.tiles_m, c.tiles_n, c.splits, c.kbps, c.kblocks};
  (void)hipGetLastError();
  const dim3 grid(c.tiles_m * c.tiles_n * c.splits);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (epilogue == SSA_EPILOGUE_NONE)
    hipLaunchKernelGGL((linear_kernel<kStages, SSA_EPILOGUE_NONE>), grid, dim3(kThreads), 0, s, a);
  else if (epilogue == SSA_EPILOGUE_RESIDUAL)
    hipLaunchKernelGGL((linear_kernel<kStages, SSA_EPILOGUE_RESIDUAL>), grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((linear_kernel<kStages, SSA_EPILOGUE_SWIGLU>), grid, dim3(kThreads), 0, s, a);
  return hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

int ssa_rms_norm(int32_t m, int32_t n, const uint16_t* x, const uint16_t* weight, float eps,
                 uint16_t* out, void* stream) {
  if (m < 0 || n <= 0 || n % 8 || n > kThreads * 8 * kNormChunks || !(eps >= 0.f))
    return SSA_ERR_ARG;
  if (m == 0) return SSA_OK;
  if (!x || !weight || !out) return SSA_ERR_NULL;
  (void)hipGetLastError();
  hipLaunchKernelGGL(rms_norm_kernel, dim3(m), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     x, weight, out, n, eps);
  return hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

}  // extern "C"
