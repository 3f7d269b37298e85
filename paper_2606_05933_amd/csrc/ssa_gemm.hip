// HIP kernels for gfx950 of the dense steps of a transformer layer
// (include/ssa_layer.h): the linear layers as one MFMA GEMM with fused
// epilogues, and RMSNorm.
//
// ssa_linear: out = x W^T, x [M, K] and W [N, K] bf16, both K-contiguous (the
// torch Linear layout), fp32 accumulation.
//  * One workgroup per output tile and K range.  A tile configuration
//    (TileCfg) sets the wave grid and each wave's share in
//    v_mfma_f32_16x16x32_bf16 tiles: 128 x 128 on 2 x 2 waves of 64 x 64,
//    256 x 256 on 2 x 4 waves of 128 x 64, 64 x 128 on 2 x 2 waves of 32 x 64,
//    32 x 256 on 1 x 4 waves of 32 x 64.  The host picks one per shape.
//  * W is the MFMA A operand (MFMA rows = output columns n) and x the B operand
//    (MFMA columns = tokens), so a lane ends with 4 consecutive n of one token:
//    one 8-byte store per 16 x 16 tile.
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
#include "ssa_device.h"

namespace {
using namespace ssa_dev;

constexpr int kNormThreads = 256;
constexpr int BK = 64;  // K block: one 128-byte LDS row per operand row
constexpr int kXcds = 8;
constexpr float kLog2e = 1.4426950408889634f;

// Split partials cross workgroups and XCDs (whose L2s are not coherent with
// each other): device-scope 8-byte stores, device-coherent loads (below), a
// device-scope ticket.
__device__ __forceinline__ void st16_dev(float* p, f32x4 v) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  const uint64_t lo = (uint64_t)__float_as_uint(v[0]) | ((uint64_t)__float_as_uint(v[1]) << 32);
  const uint64_t hi = (uint64_t)__float_as_uint(v[2]) | ((uint64_t)__float_as_uint(v[3]) << 32);
  __hip_atomic_store(q, lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Reads of the partials: 16-byte buffer loads with the device-coherent cache
// policy (sc1), the instruction of a device-scope load, so they do not hit a
// stale line of this XCD's L2.  Being plain loads to the compiler, they are
// issued back to back and waited for where a value is used (device-scope
// atomic loads would be serialised).  Offsets are bytes from the tile's first
// partial; a read past num_records would return zeros, never fault.
constexpr int kCachePolicySc1 = 16;
struct PartReader {
  __amdgpu_buffer_rsrc_t rsrc;
  __device__ explicit PartReader(const float* base)
      : rsrc(__builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), (short)0, 0x7fffffff,
                                               0x00020000)) {}
  __device__ f32x4 operator()(int byte_off) const {
    return __builtin_bit_cast(
        f32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, byte_off, 0, kCachePolicySc1));
  }
};

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

// A tile configuration: NWM x NWN waves, each owning TM x TN MFMA tiles of
// 16 x 16 (TM along tokens, TN along output features); STAGES K blocks in the
// LDS ring; OCC workgroups per CU the launch bounds ask for.
template <int NWM_, int NWN_, int TM_, int TN_, int STAGES_, int OCC_>
struct TileCfg {
  static constexpr int NWM = NWM_, NWN = NWN_, TM = TM_, TN = TN_, STAGES = STAGES_, OCC = OCC_;
  static constexpr int kWaves = NWM * NWN, kThreads = kWaves * 64;
  static constexpr int BM = NWM * TM * 16, BN = NWN * TN * 16;
  static constexpr int kStage = (BM + BN) * BK * 2;  // x rows, then W rows
  static constexpr int kPieces = (BM + BN) / 8;      // 1 KB copies (8 rows) per stage
  static constexpr int kLoads = kPieces / kWaves;    // copies per wave per stage
  static constexpr int kTileFloats = BM * BN;
  static_assert(kPieces % kWaves == 0, "copies must split evenly over the waves");
  static_assert(TN % 2 == 0, "the SwiGLU epilogue pairs n tiles");
  static_assert((STAGES - 2) * kLoads < 64, "vmcnt range");
};

// Wait until at most `left` K blocks (LOADS copies each) of this wave are in flight.
template <int STAGES, int LOADS>
__device__ __forceinline__ void wait_blocks(int left) {
  if (STAGES >= 4 && left >= 2) vm_wait<2 * LOADS>();
  else if (STAGES >= 3 && left >= 1) vm_wait<LOADS>();
  else vm_wait<0>();
}

template <class C, int EPI>
__global__ __launch_bounds__(C::kThreads, C::OCC) void linear_kernel(GemmArgs a) {
  constexpr int TM = C::TM, TN = C::TN, STAGES = C::STAGES, LOADS = C::kLoads;
  constexpr int BM = C::BM, BN = C::BN;
  __shared__ __attribute__((aligned(16))) char lds[STAGES * C::kStage];
  // The split reduction's "last arriver" flag shares the ring's first word: it
  // is written after every wave has drained its copies (vmcnt(0)) and passed a
  // barrier behind its last ring read.  (A separate word would take the
  // 192-row tile's two workgroups 8 bytes past the CU's 160 KB.)
  int& s_last = *reinterpret_cast<int*>(lds);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w / C::NWN, wn = w % C::NWN;
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

  // Copy r of this wave fills 1 KB piece p = kWaves r + w of a stage: pieces
  // below BM / 8 hold x rows 8p..8p+7, the rest W rows; lane i fetches the
  // chunk that belongs at its LDS slot (row 8p + i / 8, slot i % 8).
  const uint16_t* src[LOADS];
#pragma unroll
  for (int r = 0; r < LOADS; ++r) {
    const int p = r * C::kWaves + w;
    const int chunk = (lane & 7) ^ (lane >> 3);
    if (p < BM / 8) {
      const int row = p * 8 + (lane >> 3);
      src[r] = a.x + (size_t)min(m0 + row, a.m - 1) * a.k + (size_t)kb0 * BK + chunk * 8;
    } else {
      const int row = (p - BM / 8) * 8 + (lane >> 3);
      src[r] = a.w + (size_t)(n0 + row) * a.k + (size_t)kb0 * BK + chunk * 8;
    }
  }
  auto issue = [&](int i) {
    const char* st = lds + (i % STAGES) * C::kStage;
#pragma unroll
    for (int r = 0; r < LOADS; ++r)
      dma16(src[r] + (size_t)i * BK, st + (r * C::kWaves + w) * 1024);
  };

  // fragment reads: row r16 of a 16-row tile, logical chunk 4 ks + g
  const int xoff = (wm * TM * 16 + r16) * 128;
  const int woff = BM * 128 + (wn * TN * 16 + r16) * 128;
  const int c0 = (g ^ (r16 & 7)) << 4, c1 = ((4 + g) ^ (r16 & 7)) << 4;

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int i = 0; i < STAGES - 1; ++i)
    if (i < nkb) issue(i);
  for (int i = 0; i < nkb; ++i) {
    wait_blocks<STAGES, LOADS>(min(nkb - 1 - i, STAGES - 2));
    __syncthreads();  // block i has landed for every wave; stage (i - 1) % STAGES is free
    if (i + STAGES - 1 < nkb) issue(i + STAGES - 1);
    const char* st = lds + (i % STAGES) * C::kStage;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c = ks ? c1 : c0;
      bf16x8 xf[TM], wf[TN];
#pragma unroll
      for (int t = 0; t < TM; ++t) xf[t] = as_bf16x8(ld16(st + xoff + t * 2048 + c));
#pragma unroll
      for (int t = 0; t < TN; ++t) wf[t] = as_bf16x8(ld16(st + woff + t * 2048 + c));
#pragma unroll
      for (int mt = 0; mt < TM; ++mt)
#pragma unroll
        for (int nt = 0; nt < TN; ++nt) acc[mt][nt] = mfma(wf[nt], xf[mt], acc[mt][nt]);
    }
  }

  // 16-token tiles of this wave that hold rows < M (wave-uniform)
  const int nmt = max(0, min(TM, (a.m - (m0 + wm * TM * 16) + 15) / 16));
  if (a.splits > 1) {
    const int tile = tn * a.tiles_m + tm;
    const size_t wbase = (size_t)w * (TM * TN * 256) + lane * 4;
    float* mine = a.part + ((size_t)tile * a.splits + split) * C::kTileFloats + wbase;
#pragma unroll
    for (int mt = 0; mt < TM; ++mt)
      if (mt < nmt)
#pragma unroll
        for (int nt = 0; nt < TN; ++nt) st16_dev(mine + (mt * TN + nt) * 256, acc[mt][nt]);
    vm_wait<0>();  // this thread's device-scope stores have completed
    __syncthreads();
    if (tid == 0) {
      const int prev =
          __hip_atomic_fetch_add(&a.tickets[tile], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == a.splits - 1);
    }
    __syncthreads();
    if (!s_last) return;
    // sum in split order, own split from registers (the same bits it stored);
    // the partials of four splits are in flight at once
    const PartReader rd(a.part + (size_t)tile * a.splits * C::kTileFloats);
    const int wb = (int)wbase * 4;
#pragma unroll
    for (int mt = 0; mt < TM; ++mt) {
      if (mt >= nmt) continue;
      f32x4 tot[TN];
#pragma unroll
      for (int nt = 0; nt < TN; ++nt) tot[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int s0 = 0; s0 < a.splits; s0 += 4) {
        f32x4 v[4][TN];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int s = s0 + j;
#pragma unroll
          for (int nt = 0; nt < TN; ++nt)
            v[j][nt] = (s < a.splits && s != split)
                           ? rd((s * C::kTileFloats + (mt * TN + nt) * 256) * 4 + wb)
                           : acc[mt][nt];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (s0 + j < a.splits)
#pragma unroll
            for (int nt = 0; nt < TN; ++nt) tot[nt] += v[j][nt];
      }
#pragma unroll
      for (int nt = 0; nt < TN; ++nt) acc[mt][nt] = tot[nt];
    }
    if (tid == 0) __hip_atomic_store(&a.tickets[tile], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }

  // epilogue: lane holds n = nbase + 4 g .. + 3 of token m0 + wm TM 16 + 16 mt + r16
#pragma unroll
  for (int mt = 0; mt < TM; ++mt) {
    if (mt >= nmt) continue;
    const int tok = m0 + wm * TM * 16 + mt * 16 + r16;
    if (tok >= a.m) continue;
    const int nbase = n0 + wn * TN * 16;
    if (EPI == SSA_EPILOGUE_SWIGLU) {
      // W rows in 16-row blocks, gate block then up block of the same 16 outputs
      const int nout = a.n / 2;
#pragma unroll
      for (int j = 0; j < TN / 2; ++j) {
        const f32x4 gt = acc[mt][2 * j], up = acc[mt][2 * j + 1];
        const int col = nbase / 2 + j * 16 + g * 4;
        u32x2 v = {pack2(silu(gt[0]) * up[0], silu(gt[1]) * up[1]),
                   pack2(silu(gt[2]) * up[2], silu(gt[3]) * up[3])};
        *reinterpret_cast<u32x2*>(a.out + (size_t)tok * nout + col) = v;
      }
    } else {
#pragma unroll
      for (int nt = 0; nt < TN; ++nt) {
        const int col = nbase + nt * 16 + g * 4;
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
__global__ __launch_bounds__(kNormThreads) void rms_norm_kernel(const uint16_t* x, const uint16_t* wt,
                                                            uint16_t* out, int n, float eps) {
  __shared__ float s_part[kNormThreads / 64];
  const int tid = threadIdx.x;
  const uint16_t* row = x + (size_t)blockIdx.x * n;
  u32x4 v[kNormChunks];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < kNormChunks; ++c) {
    const int e = (c * kNormThreads + tid) * 8;
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
    const int e = (c * kNormThreads + tid) * 8;
    if (e >= n) continue;
    const u32x4 wv = ld16(wt + e);
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      o[j] = pack2(bf16_lo(v[c][j]) * rs * bf16_lo(wv[j]), bf16_hi(v[c][j]) * rs * bf16_hi(wv[j]));
    *reinterpret_cast<u32x4*>(out + (size_t)blockIdx.x * n + e) = o;
  }
}

// The tile configurations the host chooses from.
using CfgMid2 = TileCfg<2, 2, 4, 4, 2, 2>;   // 128 x 128, 4 waves of 64 x 64, two per CU
using CfgBig = TileCfg<2, 4, 8, 4, 2, 1>;    // 256 x 256, 8 waves of 128 x 64
using CfgM64 = TileCfg<2, 2, 2, 4, 3, 2>;    // 64 x 128, 4 waves of 32 x 64, two per CU
using CfgTiny = TileCfg<1, 4, 2, 4, 4, 1>;   // 32 x 256: few tokens, weight streaming
using CfgM160 = TileCfg<2, 2, 5, 4, 2, 2>;   // 160 x 128, 4 waves of 80 x 64, two per CU
using CfgM192 = TileCfg<2, 2, 6, 4, 2, 2>;   // 192 x 128, 4 waves of 96 x 64, two per CU
enum { kCfgMid2, kCfgBig, kCfgM64, kCfgTiny, kCfgM160, kCfgM192, kNumCfgs };

struct CfgShape {
  int bm, bn, occ;
};
template <class C>
constexpr CfgShape shape_of() {
  return CfgShape{C::BM, C::BN, C::OCC};
}
constexpr CfgShape kCfgShapes[kNumCfgs] = {shape_of<CfgMid2>(), shape_of<CfgBig>(),
                                           shape_of<CfgM64>(),  shape_of<CfgTiny>(),
                                           shape_of<CfgM160>(), shape_of<CfgM192>()};

struct GemmPlan {
  int cfg, tiles_m, tiles_n, splits, kbps, kblocks;
  size_t tickets, ws;
};

constexpr int kCus = 256;

// Split K when the tiles alone leave the chip under target_wgs workgroups
// (at least 4 K blocks per split).  Tiles that overfill the chip by a partial
// round are not split: measured on MI355X, the extra partials cost about what
// the evened rounds save (an even spread needs per-unit scheduling instead).
GemmPlan gemm_plan(int cfg, int m, int n, int k, int target_wgs) {
  const CfgShape& cs = kCfgShapes[cfg];
  GemmPlan c;
  c.cfg = cfg;
  c.tiles_m = (m + cs.bm - 1) / cs.bm;
  c.tiles_n = n / cs.bn;
  c.kblocks = k / BK;
  const int tiles = c.tiles_m * c.tiles_n;
  int s = 1;
  if (tiles < target_wgs / 2) s = (target_wgs + tiles - 1) / tiles;
  s = std::max(1, std::min(s, c.kblocks / 4));
  c.kbps = (c.kblocks + s - 1) / s;
  c.splits = (c.kblocks + c.kbps - 1) / c.kbps;
  c.tickets = ((size_t)tiles * 4 + 255) / 256 * 256;
  c.ws = c.splits > 1 ? c.tickets + (size_t)tiles * c.splits * cs.bm * cs.bn * 4 : 0;
  return c;
}

// The same tiles in (up to) s K splits of at least 4 K blocks.
GemmPlan split_plan(GemmPlan c, int s) {
  const CfgShape& cs = kCfgShapes[c.cfg];
  s = std::max(1, std::min(s, c.kblocks / 4));
  c.kbps = (c.kblocks + s - 1) / s;
  c.splits = (c.kblocks + c.kbps - 1) / c.kbps;
  const size_t tiles = (size_t)c.tiles_m * c.tiles_n;
  c.ws = c.splits > 1 ? c.tickets + tiles * c.splits * cs.bm * cs.bn * 4 : 0;
  return c;
}

// Among the 128 x 128, 160 x 128 and 192 x 128 tiles (two workgroups per CU)
// and 1 or s K splits: the one whose workgroups take the fewest rounds of the
// chip's 512 slots, counted in rows of tile per split (a last partial round
// costs about a whole one); splits pay their partials' write and read, about
// 1.35x on this count (measured on the down projection).  Ties go to the
// smaller tile.
GemmPlan fewest_rounds(int m, int n, int k, int max_splits) {
  GemmPlan best{};
  double best_cost = 1e30;
  for (int cfg : {kCfgMid2, kCfgM160, kCfgM192}) {
    for (int s : {1, max_splits}) {
      const GemmPlan c = split_plan(gemm_plan(cfg, m, n, k, 1), s);
      const CfgShape& cs = kCfgShapes[cfg];
      const int64_t wgs = (int64_t)c.tiles_m * c.tiles_n * c.splits;
      const int64_t slots = (int64_t)kCus * cs.occ;
      double cost = (double)((wgs + slots - 1) / slots) * cs.bm / c.splits;
      if (c.splits > 1) cost *= 1.35;
      if (cost < best_cost - 1e-9) best_cost = cost, best = c;
    }
  }
  return best;
}

// Measured on MI355X against the Llama-3-8B projections (N x K = 6144 x 4096,
// 4096 x 4096, 28672 x 4096, 4096 x 14336) for M = 28 .. 4096, with the
// weights out of the caches as they are inside a layer (T128 = the number of
// 128 x 128 tiles):
//  * M <= 64: weight streaming; 32 x 256 tiles, K split to about 128 (long K
//    and M > 32: 256) workgroups;
//  * M >= 1536 with at least 192 tiles of 256 x 256: those;
//  * under-filled shapes, T128 < 256 (K > 8192: T128 < 96): 64 x 128 tiles, K-split
//    to about 256 workgroups when there are at most 128 of them, and at least
//    in two for K > 8192 (at M = 640: 40 against 60 us for the O projection);
//  * otherwise fewest_rounds over 128-, 160- and 192-row tiles (1 or 3 K splits
//    for K > 8192): gate/up at M = 384 102 against 133 us (192 rows), at
//    M = 640 169 against 194 us (160 rows); the down projection at M = 2176
//    252 against 342 us (160 rows unsplit).
GemmPlan choose_plan(int m, int n, int k) {
  const int64_t t128 = (int64_t)((m + 127) / 128) * (n / 128);
  if (n % 256 == 0) {
    if (m <= 64) return gemm_plan(kCfgTiny, m, n, k, (m > 32 && k > 8192) ? 256 : 128);
    if (m >= 1536 && (int64_t)((m + 255) / 256) * (n / 256) >= 192)
      return gemm_plan(kCfgBig, m, n, k, 256);
  }
  auto m64 = [&](int min_splits) {
    const GemmPlan c = gemm_plan(kCfgM64, m, n, k, 1);
    const int tiles = c.tiles_m * c.tiles_n;
    return split_plan(c, std::max(min_splits, tiles <= 128 ? (256 + tiles - 1) / tiles : 1));
  };
  if (k > 8192) return t128 < 96 ? m64(2) : fewest_rounds(m, n, k, 3);
  if (t128 < 256) return m64(1);
  return fewest_rounds(m, n, k, 1);
}

template <class C>
void launch_cfg(const GemmPlan& c, int epilogue, const GemmArgs& a, hipStream_t s) {
  const dim3 grid(c.tiles_m * c.tiles_n * c.splits), block(C::kThreads);
  if (epilogue == SSA_EPILOGUE_NONE)
    hipLaunchKernelGGL((linear_kernel<C, SSA_EPILOGUE_NONE>), grid, block, 0, s, a);
  else if (epilogue == SSA_EPILOGUE_RESIDUAL)
    hipLaunchKernelGGL((linear_kernel<C, SSA_EPILOGUE_RESIDUAL>), grid, block, 0, s, a);
  else
    hipLaunchKernelGGL((linear_kernel<C, SSA_EPILOGUE_SWIGLU>), grid, block, 0, s, a);
}

// Launch a planned product; the workspace has been checked against c.ws.
int launch_linear(const GemmPlan& c, int m, int n, int k, int epilogue, const uint16_t* x,
                  const uint16_t* w, const uint16_t* residual, uint16_t* out, void* workspace,
                  hipStream_t s) {
  GemmArgs a{x, w, residual, out,
             static_cast<int*>(workspace),
             c.ws > 0 ? reinterpret_cast<float*>(static_cast<char*>(workspace) + c.tickets) : nullptr,
             m, n, k, c.tiles_m, c.tiles_n, c.splits, c.kbps, c.kblocks};
  (void)hipGetLastError();
  switch (c.cfg) {
    case kCfgMid2: launch_cfg<CfgMid2>(c, epilogue, a, s); break;
    case kCfgBig: launch_cfg<CfgBig>(c, epilogue, a, s); break;
    case kCfgM64: launch_cfg<CfgM64>(c, epilogue, a, s); break;
    case kCfgM160: launch_cfg<CfgM160>(c, epilogue, a, s); break;
    case kCfgM192: launch_cfg<CfgM192>(c, epilogue, a, s); break;
    default: launch_cfg<CfgTiny>(c, epilogue, a, s); break;
  }
  return hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

// Sizes whose tile and workgroup counts fit the plan's 32-bit fields (at most
// 2^24 tiles of the smallest tile, 32 x 128, each split at most kblocks / 4
// ways) and whose operands stay below 2^40 elements.
int check_linear(int32_t m, int32_t n, int32_t k, int32_t epilogue) {
  if (m < 0 || n <= 0 || k <= 0 || n % 128 || k % BK) return SSA_ERR_ARG;
  if (epilogue < SSA_EPILOGUE_NONE || epilogue > SSA_EPILOGUE_SWIGLU) return SSA_ERR_ARG;
  if ((int64_t)m * k > INT64_C(1) << 40 || (int64_t)n * k > INT64_C(1) << 40) return SSA_ERR_ARG;
  if ((int64_t)(m / 32 + 1) * (n / 128) > INT64_C(1) << 24) return SSA_ERR_ARG;
  return SSA_OK;
}

}  // namespace

extern "C" {

int ssa_linear_workspace_size(int32_t m, int32_t n, int32_t k, size_t* ws_bytes) {
  if (!ws_bytes) return SSA_ERR_NULL;
  const int rc = check_linear(m, n, k, SSA_EPILOGUE_NONE);
  if (rc) return rc;
  *ws_bytes = m == 0 ? 0 : choose_plan(m, n, k).ws;
  return SSA_OK;
}

int ssa_linear(int32_t m, int32_t n, int32_t k, int32_t epilogue, const uint16_t* x,
               const uint16_t* w, const uint16_t* residual, uint16_t* out, void* workspace,
               size_t ws_bytes, void* stream) {
  const int rc = check_linear(m, n, k, epilogue);
  if (rc) return rc;
  if (m == 0) return SSA_OK;
  if (!x || !w || !out || (epilogue == SSA_EPILOGUE_RESIDUAL && !residual)) return SSA_ERR_NULL;
  const GemmPlan c = choose_plan(m, n, k);
  if (c.ws > 0 && (!workspace || ws_bytes < c.ws)) return SSA_ERR_WORKSPACE;
  return launch_linear(c, m, n, k, epilogue, x, w, residual, out, workspace,
                       static_cast<hipStream_t>(stream));
}

int ssa_rms_norm(int32_t m, int32_t n, const uint16_t* x, const uint16_t* weight, float eps,
                 uint16_t* out, void* stream) {
  if (m < 0 || n <= 0 || n % 8 || n > kNormThreads * 8 * kNormChunks || !(eps >= 0.f))
    return SSA_ERR_ARG;
  if (m == 0) return SSA_OK;
  if (!x || !weight || !out) return SSA_ERR_NULL;
  (void)hipGetLastError();
  hipLaunchKernelGGL(rms_norm_kernel, dim3(m), dim3(kNormThreads), 0, static_cast<hipStream_t>(stream),
                     x, weight, out, n, eps);
  return hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

}  // extern "C"
