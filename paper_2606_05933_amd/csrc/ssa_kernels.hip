// HIP kernels for gfx950 (CDNA4) and the launching entry points of the C ABI:
// ssa_kv_append, ssa_mixed_attention, and ssa_append_attention (both in one
// launch; also without a workspace argument, ssa_append_attention_static).
//
// Attention work is one launch of a flat grid; workgroup b runs work item b of
// the plan (longest first).  Two kinds of item share the launch:
//
//  * chunk tile (prefill rows, c_i > 1; Sec. 2.1 chunked prefill, Tab. 1 x1/x2):
//    128 columns = (token, q head of the kv group) pairs of one request and kv
//    head; each of the 4 waves owns 32 columns as two 16-wide MFMA N tiles, so
//    that a wave fits in 256 registers and two workgroups share a CU.
//    Key blocks of 32 keys (two 16-slot pages) are copied global -> LDS
//    (global_load_lds_dwordx4) into four stages, three blocks ahead, and shared
//    by the 4 waves.  S^T = K Q^T and O^T += V^T P run on
//    v_mfma_f32_16x16x32_bf16 with fp32 accumulation; each wave alternates the
//    two tiles so that a tile's softmax (online, base 2, fp32) sits beside the
//    other tile's MFMAs.  Causal masking is applied only on blocks that cross
//    the diagonal.
//
//  * decode split (c_i == 1; Tab. 1 x4/x5): the G q heads of one kv head are the
//    N columns of the same MFMA formulation, so each K/V byte read from HBM is
//    used by the whole GQA group.  The 4 waves of the workgroup take
//    interleaved 32-key blocks of the split's key range, the next block in
//    flight while one is computed: key rows through two LDS stages per wave
//    (whole-row global -> LDS copies), value rows straight into registers
//    (non-temporal 16-byte loads); the waves merge their (m, l, O) partials
//    through LDS at the end.
//
// Items that cover part of a key range write an fp32 partial record; the last
// item of the group to finish (atomic ticket) merges the records in split
// order and writes bf16 output, then zeroes the ticket for the next launch.
//
// MFMA operand mapping (16x16x32 bf16, wave64, lane l, g = l / 16, r = l % 16):
// A row r and B column r live in lane r of each 16-lane group; lane group g
// holds 8 consecutive K-dim elements.  The output holds rows 4g..4g+3 of
// column r.  Keys are permuted inside a 32-key block so that after the two
// QK^T MFMAs (key halves h = 0, 1) lane group g holds keys 8g..8g+7: A row r of
// half h is key 8*(r/4) + 4h + r%4.  Those 8 probabilities are exactly the B
// operand of the PV MFMA, whose A operand (V^T) is then 8 consecutive slots of
// one value-page row: a single 16-byte load.  That is why value pages are
// stored dim-major ([D][16 slots]).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <type_traits>

#include "../../include/ssa.h"
#include "ssa_device.h"
#include "ssa_plan_format.h"

namespace ssa {
int check_plan(const ssa_shape* s, const void* plan_host, const PlanHeader** out);
}

namespace {
using namespace ssa;
using namespace ssa_dev;

// Block-table and plan reads go through the constant address space: the
// kernels never write them, and wave-uniform reads then become scalar loads,
// which are not ordered with the vector loads of K/V pages.
typedef const __attribute__((address_space(4))) int32_t cint32;

constexpr float kLog2e = 1.4426950408889634f;
// The running maximum of a column is raised only when a block's logit exceeds
// it by more than this (base 2): probabilities then stay below 2^8, and the
// O accumulators are rescaled rarely.  The final normalisation uses the same
// reference, so the result does not depend on it.
constexpr float kRescaleThreshold = 8.0f;
constexpr float kNegInf = -__builtin_inff();
// LDS stages of the chunk pipeline: key block b lives in stage b % kChunkStages
// and is fetched kChunkStages - 1 blocks ahead.
constexpr int kChunkStages = 4;
// LDS operand fragments the chunk steps keep in flight ahead of their MFMAs.
constexpr int kReadAhead = 2;

template <int D>
struct Cfg {
  static constexpr int KK = D / 32;          // MFMA k-steps over the head dim
  static constexpr int MT = D / 16;          // 16-row output tiles over the head dim
  static constexpr int CPR = D / 8;          // 16-byte chunks per key row
  static constexpr int K_ROW = D * 2;        // LDS bytes per key row (chunks XOR-swizzled)
  static constexpr int K_STAGE = 32 * K_ROW; // one 32-key block of K
  static constexpr int V_PAGE = D * 32;      // LDS bytes of one value page: D rows of 16 slots
  static constexpr int V_STAGE = 2 * V_PAGE;
  static constexpr int STAGE = K_STAGE + V_STAGE;
  static constexpr int LDS_CHUNK = kChunkStages * STAGE;          // chunk item: K/V stages
  static constexpr int LDS_DECODE_KEYS = kWaves * 2 * K_STAGE;    // decode item: key stages
  static constexpr int LDS_DECODE_MERGE = kWaves * (32 + 16 * D) * 4;  // decode: waves' m, l, o
  static constexpr int LDS = std::max({LDS_CHUNK, LDS_DECODE_KEYS, LDS_DECODE_MERGE + 16});
  static constexpr int LOADS = D / 64;       // 16-byte K (and V) chunks per thread per block
  static constexpr int KROWS_PER_LOAD = 64 / CPR;  // key rows one wave-wide 1 KB load fills
};

struct AttnArgs {
  const uint8_t* plan;
  uint64_t hash;
  int32_t off_items, off_groups;
  int64_t ws_partials_off;
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  const int32_t* bt;
  uint16_t* out;
  uint8_t* ws;
  float scale_log2;
  int hq, hkv, G, maxp;
  // fused launch (append workgroups first in the grid): their number, and the
  // chunk items in the grid (the only ones that read rows appended in the
  // launch); 0 for a plain attention launch
  int append_wgs, num_chunk_items;
  int wait_polls;  // polls before the wait for appended rows gives up
  // two-stream launch: the chunk launch's last workgroup sets the dispatch
  // flag when it starts (every workgroup of the launch has then been placed)
  int signal_dispatched;
  // fused launch: this iteration's new key / value rows ([T, Hkv, D])
  const uint16_t* k_new;
  const uint16_t* v_new;
};


// 16-byte load / store at device scope (bypassing stale copies in another
// die's L2): two 8-byte device-scope atomics.  Used where one launch both
// writes and reads the same pool slots.
__device__ __forceinline__ u32x4 ld16_dev(const void* p) {
  uint64_t* q = reinterpret_cast<uint64_t*>(const_cast<void*>(p));
  const uint64_t lo = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t hi = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return u32x4{(uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32)};
}
__device__ __forceinline__ void st16_dev(void* p, u32x4 v) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  const uint32_t v0 = v[0], v1 = v[1], v2 = v[2], v3 = v[3];
  __hip_atomic_store(q, (uint64_t)v0 | ((uint64_t)v1 << 32), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, (uint64_t)v2 | ((uint64_t)v3 << 32), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

// Workspace words of a fused launch (ahead of the merge tickets): appending
// workgroups that have finished, chunk items that have finished.  Both are
// zero at rest; the last chunk item to finish takes the launch's counts back
// off them.  Then the status word: sticky error bits (SSA_STATUS_* in ssa.h).
constexpr int kCounterAppended = 0, kCounterAttended = 1;

__device__ __forceinline__ void report(uint8_t* ws, int bits) {
  __hip_atomic_fetch_or(reinterpret_cast<int*>(ws) + kWsStatusWord, bits, __ATOMIC_RELAXED,
                        __HIP_MEMORY_SCOPE_AGENT);
}

// Wait (a fused launch) until every appending workgroup has published its
// rows.  They come first in the grid and never wait, and workgroups are
// dispatched in index order, so the wait ends.  The bound (about half a second
// by default) is a safety exit: on it the wait reports SSA_STATUS_WAIT_TIMEOUT
// and the launch runs on (no hang, possibly stale rows).  One lane per wave
// polls: hundreds of waiting workgroups polling the one counter word with
// every lane would slow the very stores they wait for.
__device__ __forceinline__ void wait_appended(const AttnArgs& a) {
  if (a.append_wgs == 0) return;
  int* counters = reinterpret_cast<int*>(a.ws);
  const int me = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const int poller = __builtin_amdgcn_readfirstlane(me);
  for (int spin = 0;; ++spin) {
    int done = 0;
    if (me == poller)
      done = __hip_atomic_load(&counters[kCounterAppended], __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    if (__builtin_amdgcn_readfirstlane(done) >= a.append_wgs) break;
    if (spin >= a.wait_polls) {
      if (me == poller) report(a.ws, SSA_STATUS_WAIT_TIMEOUT);
      break;
    }
    __builtin_amdgcn_s_sleep(8);
  }
}



__device__ __forceinline__ bf16x8 pack8(const float (&p)[8]) {
  u32x4 r = {pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
  return as_bf16x8(r);
}

// Keep the first `keep` (0..8) bf16 elements of a 16-byte chunk, zero the rest.
__device__ __forceinline__ u32x4 keep_first(u32x4 v, int keep) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int e = 2 * i;
    uint32_t m = (e < keep ? 0x0000FFFFu : 0u) | (e + 1 < keep ? 0xFFFF0000u : 0u);
    r[i] = v[i] & m;
  }
  return r;
}

// 16-byte streaming load into registers issued as inline assembly: the
// compiler does not track it, and the caller waits for it with an exact
// count (wait_loads) before any use.  Non-temporal (nt): a decode reads each
// value row once, so its lines should not displace what the caches hold for
// others (measured: the decode segment 8% faster than with normal loads).
__device__ __forceinline__ u32x4 ld16_stream(const void* p) {
  u32x4 r;
  asm volatile("global_load_dwordx4 %0, %1, off nt" : "=v"(r) : "v"(p) : "memory");
  return r;
}
// s_waitcnt vmcnt(N) that also makes the registers of the loads it waits for
// valid for their uses (which the compiler may not schedule above it).
template <int N, int M>
__device__ __forceinline__ void wait_loads(u32x4 (&v)[M]) {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  if constexpr (M == 8)
    asm volatile("s_waitcnt vmcnt(%8)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]),
                   "+v"(v[6]), "+v"(v[7])
                 : "n"(N)
                 : "memory");
  else if constexpr (M == 4)
    asm volatile("s_waitcnt vmcnt(%4)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3])
                 : "n"(N)
                 : "memory");
  else
    static_assert(M == 4 || M == 8, "value fragments per block");
}

// XOR swizzle of the 16-byte chunk index of key row `key` in the LDS K block.
// One ds_read_b128 of a K operand reads the same chunk of 16 rows, keys
// 8*(r/4) + r%4 (+4 for the second half), r = 0..15; the swizzle sends them to
// 16 distinct 16-byte bank slots (D = 128: 256-byte rows), and in particular
// to 8 distinct ones within each lane octet.  It ignores key bit 2, so both key
// halves share it.  For D = 64 (128-byte rows) it separates each octet.
template <int D>
__device__ __forceinline__ int kswz(int key) {
  if (D == 128) return (key & 3) | ((key >> 1) & 12);
  return (key & 3) | ((key & 8) >> 1);
}

// Bit casts go through named scalars: applied directly to an element of a
// vector value, __builtin_bit_cast has been seen to read element 0.
__device__ __forceinline__ float as_f32(unsigned u) { return __builtin_bit_cast(float, u); }
__device__ __forceinline__ unsigned as_u32(float f) { return __builtin_bit_cast(unsigned, f); }

// Reductions over the four 16-lane groups of a wave (the lanes that hold one
// column of an MFMA output tile), with the gfx950 row-swap permutes.  With
// both operands holding x, a 16-lane swap returns rows {0,0,2,2} and {1,1,3,3}
// of x, a 32-lane swap halves {0,0} and {1,1}; combining the two results
// reduces over row pairs.
__device__ __forceinline__ float wave_max_cols(float x) {
  const unsigned u = as_u32(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const unsigned a0 = a[0], a1 = a[1];
  const unsigned v = as_u32(__builtin_elementwise_maximum(as_f32(a0), as_f32(a1)));
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  const unsigned b0 = b[0], b1 = b[1];
  return __builtin_elementwise_maximum(as_f32(b0), as_f32(b1));
}
__device__ __forceinline__ float wave_sum_cols(float x) {
  const unsigned u = as_u32(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const unsigned a0 = a[0], a1 = a[1];
  const unsigned v = as_u32(as_f32(a0) + as_f32(a1));
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  const unsigned b0 = b[0], b1 = b[1];
  return as_f32(b0) + as_f32(b1);
}

// Online-softmax step for one 16-column tile and one 32-key block.
//   s      the lane's 8 raw logits <q, k> (keys 8g .. 8g+7 of the block)
//   c      softmax_scale * log2(e) >= 0: probabilities are exp2(c*s - m)
//   MASKED whether some keys of the block are invisible to some column; then
//          bit e of `valid` says whether key e is visible to this lane's column
// m_run is the running reference in base-2 units.  It moves only when the
// block's maximum exceeds it by more than kRescaleThreshold (or while it is
// still -inf); the O accumulators and l_run are rescaled only then, in a
// wave-uniform branch.  Returns P in bf16 (the PV operand); l_run accumulates
// the same rounded values, so the normalisation matches the product.
template <int MT, bool MASKED>
__device__ __forceinline__ bf16x8 softmax_step(const float (&s)[8], unsigned valid, float c,
                                               float& m_run, float& l_run, f32x4 (&o)[MT]) {
  float mr;
  if (MASKED) {
    mr = kNegInf;
#pragma unroll
    for (int e = 0; e < 8; ++e) mr = fmaxf(mr, ((valid >> e) & 1) ? s[e] : kNegInf);
  } else {
    mr = fmaxf(fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3])), fmaxf(fmaxf(s[4], s[5]), fmaxf(s[6], s[7])));
  }
  mr = wave_max_cols(mr);
  const float mx = (mr == kNegInf) ? kNegInf : mr * c;
  const bool raise = mx > m_run + kRescaleThreshold;  // false while mx is -inf
  if (__builtin_amdgcn_ballot_w64(raise)) {
    const float m_new = raise ? mx : m_run;
    const float alpha = (m_run == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(m_run - m_new);
    l_run *= alpha;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) o[mt] *= alpha;
    m_run = m_new;
  }
  const float nm = (m_run == kNegInf) ? 0.f : -m_run;
  float p[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], c, nm));
    if (MASKED) p[e] = ((valid >> e) & 1) ? p[e] : 0.f;
  }
  // l accumulates the bf16-rounded probabilities, the values the PV product uses
  const bf16x8 pk = pack8(p);
  const u32x4 w = __builtin_bit_cast(u32x4, pk);
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t pair = w[i];
    l_run = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pair), one, l_run, false);
  }
  return pk;
}

__device__ __forceinline__ void store_bf16x4(uint16_t* dst, float a, float b, float c, float d) {
  u32x2 v = {pack2(a, b), pack2(c, d)};
  *reinterpret_cast<u32x2*>(dst) = v;
}

// Output row and q head of column `col` (local to the item) of an item.
__device__ __forceinline__ void col_target(const WorkItem& it, const ReqEntry& rq, int G, int col,
                                           int& row, int& head) {
  if (it.kind == kItemDecode) {
    row = rq.q_start;
    head = it.kvh * G + col;
  } else {
    const int cc = it.col0 + col;
    const int j = cc / G;
    row = rq.q_start + j;
    head = it.kvh * G + (cc - j * G);
  }
}

// Partial records cross workgroups (and XCDs, whose L2s are not coherent with
// each other).  They are written with device-scope stores, which write through
// to the device coherence point, and read back with device-coherent loads
// (RecordReader below), which do not hit a stale L2 copy; the ticket is a
// device-scope atomic.  This needs no L2 write-back or invalidation.
__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// s_waitcnt vmcnt(0): this wave's stores have completed at their scope.
__device__ __forceinline__ void wait_vm_stores() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Reads of the partial records by the merging workgroup: 4-byte buffer loads
// with the device-coherent cache policy (sc1), the instruction of a
// device-scope load, so they do not hit a stale L2 line.  Being plain loads to
// the compiler, many are issued before the first wait (device-scope atomic
// loads are issued one split at a time).  Offsets are bytes from the group's
// first record.
constexpr int kCachePolicySc1 = 16;
struct RecordReader {
  __amdgpu_buffer_rsrc_t rsrc;
  __device__ explicit RecordReader(const float* base)
      : rsrc(__builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), (short)0, 0x7fffffff,
                                               0x00020000)) {}
  __device__ float operator()(int64_t float_off) const {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_raw_buffer_load_b32(rsrc, (int)(float_off * 4), 0, kCachePolicySc1));
  }
  // four floats at a 16-byte aligned float offset
  __device__ f32x4 quad(int64_t float_off) const {
    return __builtin_bit_cast(
        f32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)(float_off * 4), 0, kCachePolicySc1));
  }
};

// Last arriver of a merge group: combine the split records in split order.
// Thread t takes the (column, four dims) units t, t + 256, ...: U of them per
// pass, consecutive lanes on consecutive 16-byte pieces of o.  The merge is
// latency bound (the records come from the device coherence point), so each
// round issues the loads of F splits for all U units before it uses any:
// first the maxima, then the weighted sums in split order.
template <int D, int U, int F1, int F2>
__device__ void merge_pass(const AttnArgs& a, const WorkItem& it, const ReqEntry& rq,
                           const RecordReader& rd, int C, int S, int u0) {
  constexpr int UPC = D / 4;  // units per column
  const int units = C * UPC;
  const int64_t rec = rec_floats(C, D), o_off = rec_o_off(C);
  int col[U], d0[U];
#pragma unroll
  for (int j = 0; j < U; ++j) {
    const int idx = min(u0 + j * kThreads + (int)threadIdx.x, units - 1);
    col[j] = idx / UPC;
    d0[j] = (idx % UPC) * 4;
  }
  float M[U];
#pragma unroll
  for (int j = 0; j < U; ++j) M[j] = kNegInf;
  for (int s0 = 0; s0 < S; s0 += F1) {
    float ms[F1][U];
#pragma unroll
    for (int f = 0; f < F1; ++f)
#pragma unroll
      for (int j = 0; j < U; ++j) ms[f][j] = s0 + f < S ? rd((s0 + f) * rec + col[j]) : kNegInf;
#pragma unroll
    for (int f = 0; f < F1; ++f)
#pragma unroll
      for (int j = 0; j < U; ++j) M[j] = fmaxf(M[j], ms[f][j]);
  }
  float L[U];
  f32x4 acc[U];
#pragma unroll
  for (int j = 0; j < U; ++j) {
    L[j] = 0.f;
    acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int s0 = 0; s0 < S; s0 += F2) {
    float ms[F2][U], ls[F2][U];
    f32x4 os[F2][U];
#pragma unroll
    for (int f = 0; f < F2; ++f) {
      const int64_t r = (int64_t)(s0 + f) * rec;
      const bool in = s0 + f < S;
#pragma unroll
      for (int j = 0; j < U; ++j) {
        ms[f][j] = in ? rd(r + col[j]) : kNegInf;
        ls[f][j] = in ? rd(r + C + col[j]) : 0.f;
        os[f][j] = in ? rd.quad(r + o_off + (int64_t)col[j] * D + d0[j]) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
#pragma unroll
    for (int f = 0; f < F2; ++f) {
      if (s0 + f >= S) break;
#pragma unroll
      for (int j = 0; j < U; ++j) {
        const float w = (ms[f][j] == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(ms[f][j] - M[j]);
        L[j] += w * ls[f][j];
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[j][k] += w * os[f][j][k];
      }
    }
  }
#pragma unroll
  for (int j = 0; j < U; ++j) {
    if (u0 + j * kThreads + (int)threadIdx.x >= units) break;
    const float inv = 1.f / L[j];
    int row, head;
    col_target(it, rq, a.G, col[j], row, head);
    store_bf16x4(a.out + ((size_t)row * a.hq + head) * D + d0[j], acc[j][0] * inv,
                 acc[j][1] * inv, acc[j][2] * inv, acc[j][3] * inv);
  }
}

template <int D>
__device__ void merge_group(const AttnArgs& a, const WorkItem& it, const ReqEntry& rq,
                            const MergeGroup& grp) {
  const RecordReader rd(reinterpret_cast<const float*>(a.ws + a.ws_partials_off) + grp.ws_off);
  const int C = grp.ncols, S = grp.nsplit;
  const int units = C * (D / 4);
  if (units >= 4 * kThreads) {
    // chunk tiles: few splits, many units
    for (int u0 = 0; u0 < units; u0 += 4 * kThreads) merge_pass<D, 4, 4, 2>(a, it, rq, rd, C, S, u0);
  } else {
    // decode splits and narrow tiles: many splits, few units
    for (int u0 = 0; u0 < units; u0 += kThreads) merge_pass<D, 1, 8, 8>(a, it, rq, rd, C, S, u0);
  }
}

// After this workgroup wrote its partial record (device-scope stores): wait for
// the stores, take a ticket; the last of the group's items merges and resets
// the ticket for the next launch.
template <int D>
__device__ void finish_split(const AttnArgs& a, const WorkItem& it, const ReqEntry& rq,
                             char* lds) {
  // the last word of the kernel's LDS buffer: past the decode merge area, and
  // in staging that is dead once every wave has passed the barrier below
  // (each wave waited for its own copies before leaving its loop)
  int& s_last = *reinterpret_cast<int*>(lds + Cfg<D>::LDS - 16);
  const MergeGroup grp = reinterpret_cast<const MergeGroup*>(a.plan + a.off_groups)[it.group];
  int* tickets = reinterpret_cast<int*>(a.ws) + kLaunchCounters;
  wait_vm_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int prev = __hip_atomic_fetch_add(&tickets[it.group], 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    s_last = (prev == grp.nsplit - 1);
  }
  __syncthreads();
  if (!s_last) return;
  merge_group<D>(a, it, rq, grp);
  if (threadIdx.x == 0)
    __hip_atomic_store(&tickets[it.group], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------- chunk tiles

// Per-column online-softmax state of one 16-column tile (one lane's column).
//   m    reference in base-2 units (probabilities are exp2(c*s - m))
//   thr  raw logit above which a block raises the reference:
//        (m + kRescaleThreshold) / c, -inf while nothing was seen
//   l    sum of the bf16-rounded probabilities
struct ColState {
  float m, thr, l;
};

// One 32-key block of a 16-column tile, in compute-then-correct form: the
// probabilities are formed against the current reference right away (no
// cross-lane step; softmax_begin), and only if some lane sees a logit above
// `thr` does a wave-uniform branch (softmax_end) take the column maxima, raise
// the reference of those columns, rescale their O and l, and form the block
// again.  After the first block of a column that branch is rare, so the common
// path is the 8-way maximum, 8 FMA + 8 exp2, packing and the l sum, none of
// which depends on the MFMAs of the other tile: the caller interleaves them.
//   s0, s1 the QK^T outputs of the block's two key halves (this lane: keys
//          8g .. 8g+7 of the block for column r16)
//   lim    (MASKED) key e of the lane is visible iff e <= lim
//   c      softmax_scale * log2(e) >= 0, inv_c = 1 / c (inf for c = 0)
// Maximum of 8 logits with the NaN-propagating maximum (v_maximum3_f32 on
// gfx950): unlike fmaxf it needs no quieting of its MFMA-produced operands.
// Every operand is a finite logit or -inf (masked), never NaN.
__device__ __forceinline__ float max8(const float (&s)[8]) {
  auto mx = [](float a, float b) { return __builtin_elementwise_maximum(a, b); };
  return mx(mx(mx(s[0], s[1]), mx(s[2], s[3])), mx(mx(s[4], s[5]), mx(s[6], s[7])));
}

struct SmBlock {
  float s[8];
  float lb;
  u32x4 pk;
};

template <bool MASKED>
__device__ __forceinline__ u32x4 sm_form(const float (&s)[8], int lim, float c, float m,
                                         float& lb) {
  float p[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e], c, -m));
    if (MASKED) p[e] = (e <= lim) ? p[e] : 0.f;
  }
  const u32x4 w = {pack2(p[0], p[1]), pack2(p[2], p[3]), pack2(p[4], p[5]), pack2(p[6], p[7])};
  const uint32_t w0 = w[0], w1 = w[1], w2 = w[2], w3 = w[3];
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
  float acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w0), one, 0.f, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w1), one, acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w2), one, acc, false);
  lb = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w3), one, acc, false);
  return w;
}

template <bool MASKED>
__device__ __forceinline__ SmBlock softmax_begin(f32x4 s0, f32x4 s1, int lim, float c,
                                                 const ColState& st) {
  SmBlock b;
  b.s[0] = s0[0]; b.s[1] = s0[1]; b.s[2] = s0[2]; b.s[3] = s0[3];
  b.s[4] = s1[0]; b.s[5] = s1[1]; b.s[6] = s1[2]; b.s[7] = s1[3];
  if (MASKED) {
#pragma unroll
    for (int e = 0; e < 8; ++e) b.s[e] = (e <= lim) ? b.s[e] : kNegInf;
  }
  b.pk = sm_form<MASKED>(b.s, lim, c, st.m, b.lb);
  return b;
}

template <int MT, bool MASKED>
__device__ __forceinline__ bf16x8 softmax_end(SmBlock& b, int lim, float c, float inv_c,
                                              ColState& st, f32x4 (&o)[MT]) {
  // A logit above thr gives a probability above 2^kRescaleThreshold = 256, and
  // then the lane's sum of its rounded probabilities is at least 256 (bf16
  // rounding is monotone): the cheap test on the sum, which is formed anyway,
  // admits every block that may raise a reference (and, rarely, some that do
  // not: those leave every column as it was).  While a reference is still
  // -inf its probabilities are +inf, so a column's first visible block always
  // enters.
  if (__builtin_amdgcn_ballot_w64(b.lb >= 256.f)) {
    const float cmax = wave_max_cols(max8(b.s));
    const bool raise = cmax > st.thr;  // the same for every lane of a column
    const float m_new = raise ? cmax * c : st.m;
    const float alpha = raise ? __builtin_amdgcn_exp2f(st.m - m_new) : 1.f;
    st.l *= alpha;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) o[mt] *= alpha;
    st.m = m_new;
    st.thr = raise ? (m_new + kRescaleThreshold) * inv_c : st.thr;
    float lb2;
    const u32x4 pk2 = sm_form<MASKED>(b.s, lim, c, m_new, lb2);
    // columns that did not raise keep the block as first formed (the same values)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t x = pk2[i], y = b.pk[i];
      b.pk[i] = raise ? x : y;
    }
    b.lb = raise ? lb2 : b.lb;
  }
  st.l += b.lb;
  return as_bf16x8(b.pk);
}

// Scheduling hints for one pipeline step (one basic block) of READS operand
// fragments, each feeding two MFMAs: two reads ahead, then per fragment its
// two MFMAs with VALU instructions (the softmax of the other tile) between
// them and the next read, so the matrix core and the vector ALU both stay busy
// while few fragments are live.
constexpr int kMaskMfma = 0x008, kMaskValu = 0x002 | 0x400, kMaskDsRead = 0x100;

template <int READS, int VALU_PER_MFMA, int AHEAD = 2>
__device__ __forceinline__ void interleave_stream() {
  __builtin_amdgcn_sched_group_barrier(kMaskDsRead, AHEAD, 0);
  __builtin_amdgcn_sched_group_barrier(kMaskValu, 2, 0);
#pragma unroll
  for (int i = 0; i < READS; ++i) {
    __builtin_amdgcn_sched_group_barrier(kMaskMfma, 1, 0);
    __builtin_amdgcn_sched_group_barrier(kMaskValu, VALU_PER_MFMA, 0);
    if (i + AHEAD < READS) __builtin_amdgcn_sched_group_barrier(kMaskDsRead, 1, 0);
    __builtin_amdgcn_sched_group_barrier(kMaskMfma, 1, 0);
    __builtin_amdgcn_sched_group_barrier(kMaskValu, VALU_PER_MFMA, 0);
  }
}

template <int S>
using Stage = std::integral_constant<int, S>;

template <int D, bool FUSED>
__device__ void chunk_item(const AttnArgs& a, const WorkItem& it, const ReqEntry& rq,
                           char* lds) {
  using C = Cfg<D>;
  constexpr int KK = C::KK, MT = C::MT, NT = kChunkWaveCols / 16;
  static_assert(NT == 2, "the chunk pipeline alternates two 16-column tiles");
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int g = lane >> 4, r16 = lane & 15;
  const int G = a.G;
  const int u = rq.ctx_len;
  const int nvalid = rq.ctx_len + rq.q_len;
  cint32* bt = (cint32*)a.bt + (size_t)it.req * a.maxp;
  const size_t page_stride = (size_t)a.hkv * 16 * D;
  const uint16_t* kbase = a.kc + (size_t)it.kvh * 16 * D;
  const uint16_t* vbase = a.vc + (size_t)it.kvh * 16 * D;
  const float c = a.scale_log2;
  const float inv_c = 1.f / c;

  // this wave's columns start at wc0; the tile's end is colend
  const int colend = it.col0 + it.ncols;
  const int wc0 = it.col0 + w * kChunkWaveCols;
  const int nb = (it.key1 - it.key0 + 31) / 32;  // blocks of the item
  // Blocks [0, b_vis) are visible to every column of the tile (their last key
  // is at most the tile's smallest position): they need no causal mask.
  const int vis = u + it.col0 / G + 1 - it.key0;
  const int b_vis = vis <= 0 ? 0 : min(nb, vis >> 5);

  bf16x8 qop[NT][KK];
  int pos[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int col = wc0 + nt * 16 + r16;
    if (col < colend) {
      const int j = col / G;
      const int hg = col - j * G;
      // the last key this column may see in this item: its own position, or
      // the item's last key when the item is a piece of the key range
      pos[nt] = min(u + j, it.key1 - 1);
      const uint16_t* qrow = a.q + ((size_t)(rq.q_start + j) * a.hq + it.kvh * G + hg) * D;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) qop[nt][kk] = as_bf16x8(ld16(qrow + kk * 32 + g * 8));
    } else {
      pos[nt] = -1;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) qop[nt][kk] = as_bf16x8(u32x4{0, 0, 0, 0});
    }
  }

  ColState cs[NT];
  f32x4 o[NT][MT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    cs[nt] = ColState{kNegInf, kNegInf, 0.f};
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) o[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // LDS read addresses (bytes from a stage's base).  A row r16 of key half h
  // is key 8*(r16/4) + 4h + r16%4; the XOR swizzle of its 16-byte chunks does
  // not depend on h, so half 1 sits 4 rows after half 0.
  const int key0 = 8 * (r16 >> 2) + (r16 & 3);
  const int sw = kswz<D>(key0);
  int kaddr[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) kaddr[kk] = key0 * C::K_ROW + (((kk * 4 + g) ^ sw) << 4);
  // Value pages sit in LDS page-major, as in HBM: page half h of the block,
  // row d, 16 slots (32 bytes), unswizzled.  A lane reads 16 bytes of row r16:
  // measured with the LDS bank-conflict counter, this pattern (rows 32 bytes
  // apart, halves by lane group) is conflict-free on gfx950, while swapping
  // the halves of some rows costs a second pass on every read.
  const int vaddr = C::K_STAGE + (g >> 1) * C::V_PAGE + r16 * 32 + ((g & 1) << 4);

  // Staging of one 32-key block, global -> LDS without registers
  // (global_load_lds_dwordx4): load r of wave w fills 1 KB of the stage,
  // 16 bytes per lane in lane order, so each lane fetches the global chunk
  // that belongs at its LDS slot.  Load r of every wave reads one page of the
  // block (page r for D = 128; page w / 2 for D = 64), whose index is a
  // wave-uniform scalar load.  A page past the request's last one is read
  // from the first page instead (in bounds): its keys are beyond every
  // position, and the values of unwritten slots are zeroed in LDS before use
  // (a zero probability times a NaN would not be zero).
  int kgo[C::LOADS], vgo[C::LOADS];
#pragma unroll
  for (int r = 0; r < C::LOADS; ++r) {
    const int m = r * kWaves + w;  // which 1 KB of the stage
    const int key = m * C::KROWS_PER_LOAD + lane / C::CPR;
    const int ch = (lane % C::CPR) ^ kswz<D>(key);
    kgo[r] = (key & 15) * D + ch * 8;
    const int d = (m * 32) % D + (lane >> 1);
    vgo[r] = d * 16 + ((lane & 1) << 3);
  }
  // In a fused launch the blocks from the first one holding keys >= u on are
  // copied at device scope (COH), after one wait for the appending workgroups
  // (outside the loops).
  auto dma = [&](auto coh_t, int kb, char* stage) {
    const int lp0 = kb >> 4;
    const int pg0 = bt[lp0];
    const int pg1 = (lp0 + 1 < rq.n_pages) ? bt[lp0 + 1] : pg0;
    auto issue = [&](auto coherent_t) {
      constexpr bool COH = decltype(coherent_t)::value;
#pragma unroll
      for (int r = 0; r < C::LOADS; ++r) {
        const int m = r * kWaves + w;
        const bool second = (D == 128) ? (r != 0) : (w >= 2);
        const size_t pb = (size_t)(second ? pg1 : pg0) * page_stride;
        dma16<COH>(kbase + pb + kgo[r], stage + m * 1024);
        dma16<COH>(vbase + pb + vgo[r], stage + C::K_STAGE + m * 1024);
      }
    };
    issue(coh_t);
  };
  // Zero the values of key slots >= nvalid of the block at kb (the block that
  // holds the request's end), in a stage whose loads have completed.
  auto zero_tail = [&](int kb, char* stage) {
    const int nv = nvalid - kb;
#pragma unroll
    for (int k = 0; k < D / 64; ++k) {
      const int idx = tid + k * kThreads;  // (page half, row, 16-byte half)
      const int h = idx / (2 * D), d = (idx >> 1) % D, j = idx & 1;
      const int keep = nv - (h * 16 + (j << 3));
      char* p = stage + C::K_STAGE + h * C::V_PAGE + d * 32 + j * 16;
      if (keep < 8) st16(p, keep <= 0 ? u32x4{0, 0, 0, 0} : keep_first(ld16(p), keep));
    }
  };

  // Software pipeline over (block, tile) steps.  QK(b,t) is S^T of key
  // block b for tile t, SM(b,t) its softmax and PV(b,t) its O update.
  // Iteration b of a wave runs two steps, each 16 MFMAs next to the softmax
  // of one tile that they do not depend on:
  //   step A: K(b+1) from LDS; MFMA QK(b+1,0), QK(b+1,1) | VALU SM(b,1)
  //   step B: V(b) from LDS;   MFMA PV(b,0), PV(b,1)     | VALU SM(b+1,0)
  // Operands stream: each 16-byte K or V fragment read from LDS feeds the
  // MFMAs of both tiles and is dropped, so few are live at a time.  Blocks
  // live in kChunkStages LDS stages (block b in stage b % S): iteration b
  // reads stages b%S and (b+1)%S, and fetches block b+S-1 into the stage of
  // block b-1, which every wave finished reading before the barrier that
  // ended iteration b-1; one barrier per block suffices.
  f32x4 s0[2], s1[2];  // QK outputs of tile 0 and tile 1 (two key halves each)
  bf16x8 p0, p1;

  // QK(b+1, 0..1) from stage stk into n0, n1
  auto qk2 = [&](const char* stk, f32x4 (&n0)[2], f32x4 (&n1)[2]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      n0[h] = f32x4{0.f, 0.f, 0.f, 0.f};
      n1[h] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bf16x8 k = as_bf16x8(ld16(stk + kaddr[kk] + h * 4 * C::K_ROW));
        n0[h] = mfma(k, qop[0][kk], n0[h]);
        n1[h] = mfma(k, qop[1][kk], n1[h]);
      }
  };
  // PV(b, 0..1) from stage stv
  auto pv2 = [&](const char* stv) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const bf16x8 v = as_bf16x8(ld16(stv + vaddr + mt * 16 * 32));
      o[0][mt] = mfma(v, p0, o[0][mt]);
      o[1][mt] = mfma(v, p1, o[1][mt]);
    }
  };
  auto lim_of = [&](int nt, int kb) { return pos[nt] - (kb + 8 * g); };
  // SM(b,0) as one unit (prologue)
  auto softmax_tile0 = [&](auto masked_t, int kb) {
    constexpr bool M = decltype(masked_t)::value;
    const int lim = lim_of(0, kb);
    SmBlock sb = softmax_begin<M>(s0[0], s0[1], lim, c, cs[0]);
    return softmax_end<MT, M>(sb, lim, c, inv_c, cs[0], o[0]);
  };
  auto step_a = [&](auto masked_t, const char* stk, int kb) {
    constexpr bool M = decltype(masked_t)::value;
    const int lim = lim_of(1, kb);
    f32x4 n0[2], n1[2];
    qk2(stk, n0, n1);
    SmBlock sb = softmax_begin<M>(s1[0], s1[1], lim, c, cs[1]);
    interleave_stream<2 * KK, 1, kReadAhead>();
    p1 = softmax_end<MT, M>(sb, lim, c, inv_c, cs[1], o[1]);
    s0[0] = n0[0]; s0[1] = n0[1];
    s1[0] = n1[0]; s1[1] = n1[1];
  };
  auto step_b = [&](auto masked_t, const char* stv, int kb_next) {
    constexpr bool M = decltype(masked_t)::value;
    const int lim = lim_of(0, kb_next);
    pv2(stv);
    SmBlock sb = softmax_begin<M>(s0[0], s0[1], lim, c, cs[0]);
    interleave_stream<MT, 1, kReadAhead>();
    p0 = softmax_end<MT, M>(sb, lim, c, inv_c, cs[0], o[0]);
  };
  // Every iteration issues the same number of LDS copies per thread (the
  // fetch is clamped to the last block), so the copies still allowed in
  // flight at a barrier are an exact count: the barrier ending iteration b
  // needs blocks up to b+2 (read by iteration b+1) and leaves the fetches of
  // the S-3 most recent iterations outstanding.
  constexpr int S = kChunkStages;
  constexpr int kInFlight = (S - 3) * 2 * C::LOADS;
  // Iteration b (stage SV = b % S): fetch block b+S-1 (clamped to the last
  // block) into the stage of block b-1, zero the value tail of the block read
  // next once it has landed, then step A (QK of block b+1, softmax of block b
  // for tile 1) and step B (PV of block b, softmax of block b+1 for tile 0).
  // Every wave runs every iteration, with no data-dependent branch around the
  // MFMAs: an accumulator then has exactly one use, its next MFMA, and each
  // MFMA accumulates in place.  Blocks past the item's last one are masked for
  // every column (their stages hold copies of the last block, value tails
  // zeroed: a zero probability times a zero value adds nothing).
  auto block = [&](auto masked_t, auto coh_t, auto sv_t, int b) {
    constexpr int SV = decltype(sv_t)::value;
    const int bf = min(b + S - 1, nb - 1);
    char* fst = lds + ((SV + S - 1) % S) * C::STAGE;
    dma(coh_t, it.key0 + bf * 32, fst);
    const int kn = it.key0 + min(b + 1, nb - 1) * 32;
    if (kn + 32 > nvalid) zero_tail(kn, lds + ((SV + 1) % S) * C::STAGE);
    const int kb = it.key0 + b * 32;
    step_a(masked_t, lds + ((SV + 1) % S) * C::STAGE, kb);
    step_b(masked_t, lds + SV * C::STAGE, kb + 32);
    vm_wait<kInFlight>();
    __syncthreads();
  };

  // The query fragments have landed before the first copy is issued: the
  // compiler's own waits for them would otherwise count the copies (which it
  // does not see) and stall on them inside the loop.
  lds_dma_wait();
  // Block index of the first block holding keys >= u, and the first loop
  // step (a multiple of the stage count) from which the copies are
  // device-scope: at or before the step that fetches that block.
  const int first_new = u > it.key0 ? (u - it.key0) / 32 : 0;
  const int b_coh = FUSED ? min(nb, max(0, first_new - (S - 1)) / S * S) : nb;
  const bool coh_prologue = FUSED && first_new <= S - 2;
  if (coh_prologue) wait_appended(a);
  if (coh_prologue) {
#pragma unroll
    for (int k = 0; k < S - 1; ++k)
      dma(std::true_type{}, it.key0 + min(k, nb - 1) * 32, lds + k * C::STAGE);
  } else {
#pragma unroll
    for (int k = 0; k < S - 1; ++k)
      dma(std::false_type{}, it.key0 + min(k, nb - 1) * 32, lds + k * C::STAGE);
  }
  vm_wait<kInFlight>();  // blocks 0 and 1 have landed
  __syncthreads();
  if (it.key0 + 32 > nvalid) {
    zero_tail(it.key0, lds);
    __syncthreads();
  }
  // QK(0,0), QK(0,1), SM(0,0)
  qk2(lds, s0, s1);
  if (b_vis >= 1)
    p0 = softmax_tile0(std::false_type{}, it.key0);
  else
    p0 = softmax_tile0(std::true_type{}, it.key0);
  static_assert(kChunkStages == 4, "the loop runs trips of four stages");
  // Trips of S iterations: unmasked while both blocks an iteration softmaxes
  // (b and b+1) are visible to every column, then masked up to the item's
  // block count rounded up to a trip.  One exit per loop, after whole trips.
  // In a fused launch the trips from b_coh on (when it lies inside the item)
  // copy at device scope, after one wait; each (masked, coherent) kind of trip
  // has a loop of its own, so no trip branches on either.
  const int n_um = b_vis >= 1 ? (b_vis - 1) / S * S : 0;
  const int nb_pad = (nb + S - 1) / S * S;
  const int nc_end = (FUSED && b_coh < nb) ? b_coh : nb_pad;  // end of the plain trips
  auto trip = [&](auto masked_t, auto coh_t, int b0) {
    block(masked_t, coh_t, Stage<0>{}, b0);
    block(masked_t, coh_t, Stage<1>{}, b0 + 1);
    block(masked_t, coh_t, Stage<2>{}, b0 + 2);
    block(masked_t, coh_t, Stage<3>{}, b0 + 3);
  };
  using No = std::false_type;
  using Yes = std::true_type;  // trip(masked?, coherent?, first block)
  bool waited = coh_prologue;
  int b = 0;
  for (const int e = min(n_um, nc_end); b < e; b += S) trip(No{}, No{}, b);
  if constexpr (FUSED) {
    if (b < n_um) {
      if (!waited) wait_appended(a);
      waited = true;
      for (; b < n_um; b += S) trip(No{}, Yes{}, b);
    }
  }
  for (; b < nc_end; b += S) trip(Yes{}, No{}, b);
  if constexpr (FUSED) {
    if (b < nb_pad) {
      if (!waited) wait_appended(a);
      for (; b < nb_pad; b += S) trip(Yes{}, Yes{}, b);
    }
  }
  lds_dma_wait();  // no copy may land after this workgroup has left

  // epilogue
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) cs[nt].l = wave_sum_cols(cs[nt].l);
  if (it.group < 0) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int col = wc0 + nt * 16 + r16;
      if (col >= colend) continue;
      const int j = col / G;
      const int hg = col - j * G;
      uint16_t* orow = a.out + ((size_t)(rq.q_start + j) * a.hq + it.kvh * G + hg) * D;
      const float inv = 1.f / cs[nt].l;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        store_bf16x4(orow + mt * 16 + 4 * g, o[nt][mt][0] * inv, o[nt][mt][1] * inv,
                     o[nt][mt][2] * inv, o[nt][mt][3] * inv);
    }
  } else {
    const MergeGroup grp = reinterpret_cast<const MergeGroup*>(a.plan + a.off_groups)[it.group];
    const int Cn = grp.ncols;
    float* rec = reinterpret_cast<float*>(a.ws + a.ws_partials_off) + grp.ws_off +
                 (int64_t)it.split * rec_floats(Cn, D);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int col = wc0 + nt * 16 + r16;
      if (col >= colend) continue;
      const int cl = col - it.col0;
      if (g == 0) {
        st_dev(rec + cl, cs[nt].m);
        st_dev(rec + Cn + cl, cs[nt].l);
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)  // 16-byte aligned, as records and o rows are
        st16_dev(rec + rec_o_off(Cn) + (int64_t)cl * D + mt * 16 + 4 * g,
                 __builtin_bit_cast(u32x4, o[nt][mt]));
    }
    finish_split<D>(a, it, rq, lds);
  }
}

// --------------------------------------------------------------- decode splits

template <int D, bool FUSED>
__device__ void decode_item(const AttnArgs& a, const WorkItem& it, const ReqEntry& rq,
                            char* lds) {
  using C = Cfg<D>;
  constexpr int KK = C::KK, MT = C::MT;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 4, r16 = lane & 15;
  const int G = a.G;
  cint32* bt = (cint32*)a.bt + (size_t)it.req * a.maxp;
  const size_t page_stride = (size_t)a.hkv * 16 * D;
  const size_t head_off = (size_t)it.kvh * 16 * D;
  const int key1 = it.key1;

  bf16x8 qop[KK];
  if (r16 < G) {
    const uint16_t* qrow = a.q + ((size_t)rq.q_start * a.hq + it.kvh * G + r16) * D;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qop[kk] = as_bf16x8(ld16(qrow + kk * 32 + g * 8));
  } else {
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) qop[kk] = as_bf16x8(u32x4{0, 0, 0, 0});
  }
  float m_run = kNegInf, l_run = 0.f;
  f32x4 o[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) o[mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // The two page indices of a block are wave-uniform scalar loads (no
  // vector-memory wait before the K/V loads).  A page past the request's last
  // one is read from the first page instead (in bounds); keys from it are at or
  // beyond key1, so their logits are masked and their values zeroed in compute.
  //
  // In a fused launch the item that holds key u (its last key: u + 1 = key1)
  // appends the request's new row to the pool itself, before its loop: the
  // wave that owns the item's last block stores the key row and the value
  // column of slot u and waits for the stores, so its own later reads of that
  // block see them (the waves of a workgroup share one CU and its L1).  No
  // other workgroup reads the slot in the launch, and other waves of this one
  // read it only as masked padding, so the decode never waits on another
  // workgroup and computes exactly what it computes after a separate append.
  const int nb = (key1 - it.key0 + 31) / 32;
  const int wave = __builtin_amdgcn_readfirstlane(w);
  if constexpr (FUSED) {
    const bool has_new = rq.q_len > 0 && it.key0 <= rq.ctx_len && rq.ctx_len < key1;
    if (has_new && wave == (nb - 1) % kWaves) {
      const size_t new_off = ((size_t)rq.q_start * a.hkv + it.kvh) * D;
      const size_t pg = (size_t)bt[rq.ctx_len >> 4] * page_stride + head_off;
      const int slot = rq.ctx_len & 15;
      uint16_t* kp = const_cast<uint16_t*>(a.kc) + pg;
      uint16_t* vp = const_cast<uint16_t*>(a.vc) + pg;
      if (lane < C::CPR) st16(kp + slot * D + lane * 8, ld16(a.k_new + new_off + lane * 8));
      uint16_t vn[D / 64];
#pragma unroll
      for (int k = 0; k < D / 64; ++k) vn[k] = a.v_new[new_off + k * 64 + lane];
#pragma unroll
      for (int k = 0; k < D / 64; ++k) vp[(k * 64 + lane) * 16 + slot] = vn[k];
      asm volatile("" ::: "memory");  // the stores are issued before the wait
      vm_wait<0>();
    }
  }
  // Key rows pass through LDS: each wave owns two stages of one 32-key block
  // (the chunk path's swizzled row layout), filled with global_load_lds so
  // that every load instruction reads whole key rows (non-temporal, like the
  // value loads: a decode reads each row once, while chunk tiles beside it
  // reread theirs from the caches); the MFMA operands are
  // then read from LDS in the permuted-key layout.  Value rows (dim-major
  // pages) load straight into registers, 16 bytes of 8 slots of one dim per
  // lane.  Both are issued as inline assembly and waited for with exact
  // counts: one block's KLOADS copies and MT loads stay in flight while the
  // block before it is computed.
  constexpr int KLOADS = C::K_STAGE / 1024;
  static_assert(kWaves * 2 * C::K_STAGE <= C::LDS, "key stages fit the kernel's LDS");
  char* kst = lds + w * 2 * C::K_STAGE;
  int kgo[KLOADS], kch[KLOADS];
#pragma unroll
  for (int r = 0; r < KLOADS; ++r) {
    const int key = r * C::KROWS_PER_LOAD + lane / C::CPR;
    kch[r] = (lane % C::CPR) ^ kswz<D>(key);
    kgo[r] = (key & 15) * D + kch[r] * 8;
  }
  const int key0p = 8 * (r16 >> 2) + (r16 & 3);
  const int swz = kswz<D>(key0p);
  int kaddr[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) kaddr[kk] = key0p * C::K_ROW + (((kk * 4 + g) ^ swz) << 4);

  auto issue = [&](int stage, int kb, u32x4 (&v)[MT]) {
    const int lp0 = kb >> 4;
    const int pg0 = bt[lp0];
    const int pg1 = (lp0 + 1 < rq.n_pages) ? bt[lp0 + 1] : pg0;
#pragma unroll
    for (int r = 0; r < KLOADS; ++r) {
      const int key = r * C::KROWS_PER_LOAD + lane / C::CPR;
      dma16_stream(a.kc + (size_t)((key >> 4) ? pg1 : pg0) * page_stride + head_off + kgo[r],
                   kst + stage * C::K_STAGE + r * 1024);
    }
    const uint16_t* vs = a.vc + (size_t)((g >> 1) ? pg1 : pg0) * page_stride + head_off +
                         r16 * 16 + (g & 1) * 8;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) v[mt] = ld16_stream(vs + mt * 16 * 16);
  };
  // kb: the block's first key (past the item's keys for a padding block,
  // whose stage and registers hold a copy of the last block: all masked)
  auto compute = [&](int stage, int kb, u32x4 (&v)[MT]) {
    const char* stk = kst + stage * C::K_STAGE;
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      s0 = mfma(as_bf16x8(ld16(stk + kaddr[kk])), qop[kk], s0);
      s1 = mfma(as_bf16x8(ld16(stk + kaddr[kk] + 4 * C::K_ROW)), qop[kk], s1);
    }
    const float sv[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
    bf16x8 pop;
    if (kb + 32 > key1) {
      const int lim = key1 - (kb + 8 * g);  // key e of the lane group valid iff e < lim
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) v[mt] = keep_first(v[mt], lim);
      const unsigned valid = lim <= 0 ? 0u : (lim >= 8 ? 0xFFu : (1u << lim) - 1u);
      pop = softmax_step<MT, true>(sv, valid, a.scale_log2, m_run, l_run, o);
    } else {
      pop = softmax_step<MT, false>(sv, 0xFFu, a.scale_log2, m_run, l_run, o);
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) o[mt] = mfma(as_bf16x8(v[mt]), pop, o[mt]);
  };

  // Wave w takes blocks w, w+4, ..., in pairs: every wave runs at least one
  // pair, padded with masked blocks (loads clamped to the item's last block),
  // so the loop has one exit and its accumulators one use each.  The next
  // block's loads are issued before the current one is computed.
  const int nbw = nb > wave ? (nb - wave + kWaves - 1) / kWaves : 0;
  const int n2 = nbw <= 2 ? 2 : (nbw + 1) / 2 * 2;
  auto kb_load = [&](int i) { return it.key0 + min(wave + i * kWaves, nb - 1) * 32; };
  auto kb_of = [&](int i) { return it.key0 + (wave + i * kWaves) * 32; };
  constexpr int kIssue = KLOADS + MT;
  vm_wait<0>();  // q has landed: the waits below count exactly
  u32x4 v0[MT], v1[MT];
  issue(0, kb_load(0), v0);
  for (int i = 0; i < n2; i += 2) {
    issue(1, kb_load(i + 1), v1);
    wait_loads<kIssue>(v0);
    compute(0, kb_of(i), v0);
    issue(0, kb_load(i + 2), v0);
    wait_loads<kIssue>(v1);
    compute(1, kb_of(i + 1), v1);
  }
  vm_wait<0>();  // the last (unused) copies have landed before LDS is reused
  l_run = wave_sum_cols(l_run);
  // merge the 4 waves through LDS: per wave m[16], l[16], o[D][16] (over the
  // staging area: every wave has left its loop)
  __syncthreads();
  float* sm = reinterpret_cast<float*>(lds);
  float* wm = sm + w * (32 + 16 * D);
  if (g == 0) {
    wm[r16] = m_run;
    wm[16 + r16] = l_run;
  }
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) wm[32 + (mt * 16 + 4 * g + jj) * 16 + r16] = o[mt][jj];
  __syncthreads();

  float* rec = nullptr;
  if (it.group >= 0) {
    const MergeGroup grp = reinterpret_cast<const MergeGroup*>(a.plan + a.off_groups)[it.group];
    rec = reinterpret_cast<float*>(a.ws + a.ws_partials_off) + grp.ws_off +
          (int64_t)it.split * rec_floats(G, D);
  }
  for (int idx = tid; idx < G * (D / 4); idx += kThreads) {
    const int col = idx % G;
    const int d0 = (idx / G) * 4;
    float M = kNegInf;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) M = fmaxf(M, sm[ww * (32 + 16 * D) + col]);
    float L = 0.f;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) {
      const float* pw = sm + ww * (32 + 16 * D);
      const float wt = (pw[col] == kNegInf) ? 0.f : __builtin_amdgcn_exp2f(pw[col] - M);
      L += wt * pw[16 + col];
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[k] += wt * pw[32 + (d0 + k) * 16 + col];
    }
    if (rec) {
      if (d0 == 0) {
        st_dev(rec + col, M);
        st_dev(rec + G + col, L);
      }
      st16_dev(rec + rec_o_off(G) + (int64_t)col * D + d0,  // 16-byte aligned
               u32x4{__builtin_bit_cast(uint32_t, acc[0]), __builtin_bit_cast(uint32_t, acc[1]),
                     __builtin_bit_cast(uint32_t, acc[2]), __builtin_bit_cast(uint32_t, acc[3])});
    } else {
      const float inv = 1.f / L;
      store_bf16x4(a.out + ((size_t)rq.q_start * a.hq + it.kvh * G + col) * D + d0,
                   acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
    }
  }
  if (rec) finish_split<D>(a, it, rq, lds);
}

// One attention work item of the plan.
template <int D, bool FUSED>
__device__ void attention_wg(const AttnArgs& a, const WorkItem& it, char* lds) {
  ReqEntry rq;
  rq.q_start = it.q_start;
  rq.ctx_len = it.ctx_len;
  rq.q_len = it.nvalid - it.ctx_len;
  rq.n_pages = (it.nvalid + 15) >> 4;
  if (it.kind == kItemChunk)
    chunk_item<D, FUSED>(a, it, rq, lds);
  else
    decode_item<D, FUSED>(a, it, rq, lds);
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void mixed_attention_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) char lds[Cfg<D>::LDS];
  // The plan may live in device-mapped host memory: the header check and this
  // workgroup's item are independent loads.
  const PlanHeader* hdr = reinterpret_cast<const PlanHeader*>(a.plan);
  const WorkItem it = reinterpret_cast<const WorkItem*>(a.plan + a.off_items)[blockIdx.x];
  if (hdr->magic != kPlanMagic || hdr->hash != a.hash) {
    if (threadIdx.x == 0) report(a.ws, SSA_STATUS_PLAN_MISMATCH);
    return;
  }
  attention_wg<D, false>(a, it, lds);
}

// ---------------------------------------------- decode rows on a second stream
//
// The decode items of ssa_append_attention_streams, in a kernel of their own
// that runs beside the chunk rows' launch.  A CU holds two chunk workgroups
// (two waves of 216 registers per SIMD, 64 KB of LDS each); this kernel is
// built to fit in what they leave, 80 registers per lane and 32 KB, so that one
// of its workgroups runs on every CU as a third resident workgroup and streams
// the decode rows' K/V while the chunk tiles compute.
//
// The 4 waves split the head dim (wave w owns dims 32w .. 32w+31) and walk the
// same 32-key blocks of the item.  QK tile p of a block holds the 16 keys of
// its page p (A row r = slot r; this wave's 32 dims), so the output gives lane
// group g keys 4g..4g+3 of each page: element e of the lane's 8 probabilities
// is key 16*(e/4) + 4g + e%4, and the V operand takes the same keys (8 bytes of
// 4 slots of one dim from each dim-major page).  Each wave's partial logits
// (over its dims) are summed through LDS: G <= 8, so only columns 0..7 hold
// logits and lanes 8..15 of each row carry those of the second tile; one
// 16-byte record per lane, double-buffered, one barrier per block.  Every wave
// then forms the same probabilities and accumulates O for its own dims.
// Every load reads one page through a buffer resource of that page's head (16
// slots x D, range-checked), non-temporal, with a loop-invariant lane offset;
// the loads of two blocks are in flight (K of block i+2 issued once block i's
// QK MFMAs have read their operands, V once its PV MFMAs have).
constexpr int kStreamMaxG = 8;
constexpr int kWaitDispatchedPolls = 2048;  // about 1 ms
constexpr int kStreamD = 128;
constexpr int kCachePolicyNt = 2;  // buffer-load cache policy: non-temporal

// value of lane (l & ~15) | ((l + 8) & 15): rotate each row of 16 lanes by 8
__device__ __forceinline__ float row_ror8(float x) {
  return as_f32((unsigned)__builtin_amdgcn_update_dpp(0, (int)as_u32(x), 0x128, 0xF, 0xF, false));
}

// Keep the bf16 elements whose bit is set in `valid`, zero the others.
__device__ __forceinline__ u32x4 keep_valid(u32x4 v, unsigned valid) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t m = (((valid >> (2 * i)) & 1) ? 0x0000FFFFu : 0u) |
                       (((valid >> (2 * i + 1)) & 1) ? 0xFFFF0000u : 0u);
    r[i] = v[i] & m;
  }
  return r;
}

// One decode item.  xs: each wave's partial logits of the current block,
// [buffer][wave][lane]; s_last: the merge ticket's verdict (both in LDS).
__device__ __forceinline__ void decode_stream_item(const AttnArgs& a, const WorkItem& it,
                                                   f32x4 (&xs)[2][kWaves][64], int& s_last) {
  constexpr int D = kStreamD;
  ReqEntry rq;
  rq.q_start = it.q_start;
  rq.ctx_len = it.ctx_len;
  rq.q_len = it.nvalid - it.ctx_len;
  rq.n_pages = (it.nvalid + 15) >> 4;
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, r16 = lane & 15;
  const int G = a.G;
  cint32* bt = (cint32*)a.bt + (size_t)it.req * a.maxp;
  const size_t page_stride = (size_t)a.hkv * 16 * D;
  const size_t head_off = (size_t)it.kvh * 16 * D;
  const int key0 = it.key0, key1 = it.key1;
  const int nb = (key1 - key0 + 31) / 32;

  // The item that holds key u appends the request's new row first: each wave
  // stores its own 32 dims of the key row and of the value column of slot u
  // and waits for them; those are the only bytes of the slot that wave reads
  // back, and no other workgroup reads the slot in this launch.
  if (rq.q_len > 0 && key0 <= rq.ctx_len && rq.ctx_len < key1) {
    const size_t new_off = ((size_t)rq.q_start * a.hkv + it.kvh) * D + 32 * w;
    const size_t pg = (size_t)bt[rq.ctx_len >> 4] * page_stride + head_off;
    const int slot = rq.ctx_len & 15;
    uint16_t* kp = const_cast<uint16_t*>(a.kc) + pg + slot * D + 32 * w;
    uint16_t* vp = const_cast<uint16_t*>(a.vc) + pg + (size_t)(32 * w) * 16 + slot;
    if (lane < 4) st16(kp + lane * 8, ld16(a.k_new + new_off + lane * 8));
    if (lane < 32) vp[lane * 16] = a.v_new[new_off + lane];
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  bf16x8 qop = as_bf16x8(u32x4{0, 0, 0, 0});
  if (r16 < G)
    qop = as_bf16x8(ld16(a.q + ((size_t)rq.q_start * a.hq + it.kvh * G + r16) * D + 32 * w + 8 * g));

  const int voffK = r16 * (2 * D) + 2 * (32 * w + 8 * g);  // bytes: slot r16, 8 dims
  const int voffV = (32 * w + r16) * 32 + 8 * g;           // bytes: dim row, slots 4g..4g+3
  const uint16_t* kbase = a.kc + head_off;
  const uint16_t* vbase = a.vc + head_off;
  auto rsrc = [&](const uint16_t* base, int pg) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base) + (size_t)pg * page_stride,
                                             (short)0, 16 * D * 2, 0x00020000);
  };
  // the block's two pages; a page past the request's last one is read from the
  // first (in range; its keys are at or past key1 and masked)
  auto pages = [&](int i, int& pg0, int& pg1) {
    const int lp0 = (key0 + min(i, nb - 1) * 32) >> 4;
    pg0 = bt[lp0];
    pg1 = (lp0 + 1 < rq.n_pages) ? bt[lp0 + 1] : pg0;
  };
  auto issue_k = [&](int i, u32x4 (&r)[4]) {
    int pg0, pg1;
    pages(i, pg0, pg1);
    r[0] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc(kbase, pg0), voffK, 0, kCachePolicyNt));
    r[1] = __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc(kbase, pg1), voffK, 0, kCachePolicyNt));
  };
  auto issue_v = [&](int i, u32x4 (&r)[4]) {
    int pg0, pg1;
    pages(i, pg0, pg1);
    const auto v0 = rsrc(vbase, pg0), v1 = rsrc(vbase, pg1);
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const u32x2 lo = __builtin_bit_cast(
          u32x2, __builtin_amdgcn_raw_buffer_load_b64(v0, voffV, mt * 512, kCachePolicyNt));
      const u32x2 hi = __builtin_bit_cast(
          u32x2, __builtin_amdgcn_raw_buffer_load_b64(v1, voffV, mt * 512, kCachePolicyNt));
      r[2 + mt] = u32x4{lo[0], lo[1], hi[0], hi[1]};
    }
  };

  float m_run = kNegInf, l_run = 0.f;
  f32x4 o[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  const bool lo8 = r16 < 8;
  // block i (keys key0 + 32 i ..) from r; then r takes block nxt's loads
  auto step = [&](int i, u32x4 (&r)[4], int nxt) {
    const int kb = key0 + i * 32;
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    const f32x4 s0 = mfma(as_bf16x8(r[0]), qop, z);
    const f32x4 s1 = mfma(as_bf16x8(r[1]), qop, z);
    issue_k(nxt, r);
    const int buf = i & 1;
    f32x4 x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // the rotate reads other lanes: it runs in every lane, never under a
      // branch on lo8 (where the lanes it reads would be inactive)
      float rr = row_ror8(s1[j]);
      asm volatile("" : "+v"(rr));
      x[j] = lo8 ? s0[j] : rr;
    }
    xs[buf][w][lane] = x;
    __syncthreads();
    // the four partials in a fixed order (the same sum in every wave), one
    // read in flight at a time
    f32x4 t = xs[buf][0][lane];
#pragma unroll
    for (int ww = 1; ww < kWaves; ++ww) {
      asm volatile("" : "+v"(t)::"memory");
      t += xs[buf][ww][lane];
    }
    float sv[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float rr = row_ror8(t[j]);
      asm volatile("" : "+v"(rr));
      sv[j] = t[j];
      sv[4 + j] = rr;
    }
    // element e of the lane: key kb + 16*(e/4) + 4g + e%4, valid below key1
    unsigned valid = 0xFFu;
    if (kb + 32 > key1) {
      const int l0 = key1 - (kb + 4 * g), l1 = key1 - (kb + 16 + 4 * g);
      const unsigned m0 = l0 <= 0 ? 0u : (l0 >= 4 ? 0xFu : (1u << l0) - 1u);
      const unsigned m1 = l1 <= 0 ? 0u : (l1 >= 4 ? 0xFu : (1u << l1) - 1u);
      valid = m0 | (m1 << 4);
      r[2] = keep_valid(r[2], valid);
      r[3] = keep_valid(r[3], valid);
    }
    const bf16x8 pop = softmax_step<2, true>(sv, valid, a.scale_log2, m_run, l_run, o);
    o[0] = mfma(as_bf16x8(r[2]), pop, o[0]);
    o[1] = mfma(as_bf16x8(r[3]), pop, o[1]);
    issue_v(nxt, r);
  };

  // Every wave runs every block, in pairs (a padding block past the item's
  // last one is masked for every key: its loads repeat the last block), so the
  // waits and barriers match across waves.
  vm_wait<0>();
  u32x4 ra[4], rb[4];
  issue_k(0, ra);
  issue_v(0, ra);
  issue_k(1, rb);
  issue_v(1, rb);
  const int n2 = (nb + 1) / 2 * 2;
  for (int i = 0; i < n2; i += 2) {
    step(i, ra, i + 2);
    step(i + 1, rb, i + 3);
  }
  const float l = wave_sum_cols(l_run);

  float* rec = nullptr;
  MergeGroup grp{};
  if (it.group >= 0) {
    grp = reinterpret_cast<const MergeGroup*>(a.plan + a.off_groups)[it.group];
    rec = reinterpret_cast<float*>(a.ws + a.ws_partials_off) + grp.ws_off +
          (int64_t)it.split * rec_floats(G, D);
  }
  // lane (g, r16) holds dims 32w + 16mt + 4g .. +3 of column r16
  if (r16 < G) {
    if (rec) {
      if (w == 0 && g == 0) {
        st_dev(rec + r16, m_run);
        st_dev(rec + G + r16, l);
      }
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
        st16_dev(rec + rec_o_off(G) + (int64_t)r16 * D + 32 * w + 16 * mt + 4 * g,
                 __builtin_bit_cast(u32x4, o[mt]));
    } else {
      const float inv = 1.f / l;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
        store_bf16x4(a.out + ((size_t)rq.q_start * a.hq + it.kvh * G + r16) * D + 32 * w + 16 * mt +
                         4 * g,
                     o[mt][0] * inv, o[mt][1] * inv, o[mt][2] * inv, o[mt][3] * inv);
    }
  }
  if (!rec) return;
  // the last of the group's items merges the records (as finish_split)
  int* tickets = reinterpret_cast<int*>(a.ws) + kLaunchCounters;
  wait_vm_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int prev = __hip_atomic_fetch_add(&tickets[it.group], 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    s_last = (prev == grp.nsplit - 1);
  }
  __syncthreads();
  if (!s_last) return;
  // G * D / 4 <= kThreads units: one pass of the decode merge
  static_assert(kStreamMaxG * (D / 4) <= kThreads, "one merge pass");
  const RecordReader rd(reinterpret_cast<const float*>(a.ws + a.ws_partials_off) + grp.ws_off);
  merge_pass<D, 1, 4, 4>(a, it, rq, rd, grp.ncols, grp.nsplit, 0);
  if (threadIdx.x == 0)
    __hip_atomic_store(&tickets[it.group], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// On the decode stream of a two-stream launch, ahead of the decode launch: wait
// until the chunk launch has placed all its workgroups (its last one sets the
// flag when it starts), so that decode workgroups only take the slots the
// chunk tiles leave, then clear the flag (zero at rest).  Where the two streams
// share a hardware queue this kernel runs after the chunk launch and finds the
// flag set.  Bounded: after `polls` polls (about half a microsecond each) the
// decode launch goes ahead anyway.
__global__ __launch_bounds__(64) void wait_dispatched_kernel(int* flag, int polls) {
  for (int i = 0; i < polls; ++i) {
    if (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) break;
    __builtin_amdgcn_s_sleep(16);
  }
  if (threadIdx.x == 0) __hip_atomic_store(flag, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One decode item per workgroup: item item0 + blockIdx.x of the plan.
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(6, 8)))
void decode_stream_kernel(AttnArgs a, int item0) {
  __shared__ __attribute__((aligned(16))) f32x4 xs[2][kWaves][64];
  __shared__ int s_last;
  const PlanHeader* hdr = reinterpret_cast<const PlanHeader*>(a.plan);
  const WorkItem it = reinterpret_cast<const WorkItem*>(a.plan + a.off_items)[item0 + (int)blockIdx.x];
  if (hdr->magic != kPlanMagic || hdr->hash != a.hash) {
    if (threadIdx.x == 0) report(a.ws, SSA_STATUS_PLAN_MISMATCH);
    return;
  }
  decode_stream_item(a, it, xs, s_last);
}

// ------------------------------------------------------------------ kv_append

struct AppendArgs {
  const uint16_t* k_new;
  const uint16_t* v_new;
  uint16_t* kc;
  uint16_t* vc;
  int32_t off_segments;
};

// The rows of one append segment (consecutive new tokens of one request that
// land in one page) for kv head h: key rows are copied as they are; value
// rows are transposed into the dim-major page ([D][16 slots]), as whole
// 16-byte half rows where a segment covers them, else slot by slot.  At most
// 16 rows: one key chunk and one value half row per thread.
template <int D>
__device__ void append_rows(const AppendArgs& ap, const AppendSeg& sg, const int32_t* bt, int h,
                            int hkv, int maxp) {
  constexpr int CPR = D / 8;
  static_assert(16 * CPR <= kThreads && 2 * D <= kThreads, "one unit per thread");
  const int slot0 = sg.pos0 % 16;
  const size_t pb = (size_t)bt[(size_t)sg.req * maxp + sg.pos0 / 16] * hkv * 16 * D +
                    (size_t)h * 16 * D;
  const int t = threadIdx.x;
  // key rows: (row, 16-byte chunk)
  if (t < sg.n * CPR) {
    const int r = t / CPR, c = t % CPR;
    st16(ap.kc + pb + (size_t)(slot0 + r) * D + c * 8,
         ld16(ap.k_new + ((size_t)(sg.row0 + r) * hkv + h) * D + c * 8));
  }
  // value rows: (dim, half page row of 8 slots), slots [lo, hi) of the half
  if (t < 2 * D) {
    const int d = t >> 1, half = t & 1;
    const int lo = max(half * 8, slot0), hi = min(half * 8 + 8, slot0 + sg.n);
    if (lo < hi) {
      uint16_t* dst = ap.vc + pb + (size_t)d * 16;
      auto src = [&](int sl) {
        return (uint32_t)ap.v_new[((size_t)(sg.row0 + sl - slot0) * hkv + h) * D + d];
      };
      if (lo == half * 8 && hi == half * 8 + 8) {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = src(lo + 2 * i) | (src(lo + 2 * i + 1) << 16);
        st16(dst + lo, u32x4{w[0], w[1], w[2], w[3]});
      } else {
        for (int sl = lo; sl < hi; ++sl) dst[sl] = (uint16_t)src(sl);
      }
    }
  }
}

// One append segment for every kv head, in a fused launch (device-scope
// stores).  Latency matters more than issue here (the launch's decode traffic
// fills the memory queues), so each pass makes one round of 16-byte loads of
// whole key and value rows for HG heads, stores the key rows, and transposes
// the value rows through LDS into the dim-major page.
template <int D>
__device__ void append_segment_staged(const AppendArgs& ap, const AppendSeg& sg,
                                      const int32_t* bt, int hkv, int maxp, char* lds) {
  constexpr int CPR = D / 8;
  constexpr int HG = 128 / CPR;                    // heads per pass
  constexpr int UK = HG * 16 * CPR / kThreads;     // 16-byte units per thread per pass and kind
  static_assert(UK * kThreads == HG * 16 * CPR, "whole units per thread");
  static_assert(HG * 16 * D * 2 <= Cfg<D>::LDS, "staging fits the kernel's LDS");
  const int n = sg.n, slot0 = sg.pos0 % 16;
  const size_t pb = (size_t)bt[(size_t)sg.req * maxp + sg.pos0 / 16] * hkv * 16 * D;
  uint16_t* vt = reinterpret_cast<uint16_t*>(lds);  // [HG][16 rows][D], token-major
  for (int h0 = 0; h0 < hkv; h0 += HG) {
    u32x4 kr[UK], vr[UK];
#pragma unroll
    for (int k = 0; k < UK; ++k) {
      const int idx = threadIdx.x + k * kThreads;  // (head, row, 16-byte chunk)
      const int hl = idx / (16 * CPR), r = (idx / CPR) & 15, c = idx % CPR;
      if (h0 + hl < hkv && r < n) {
        const size_t off = ((size_t)(sg.row0 + r) * hkv + h0 + hl) * D + c * 8;
        kr[k] = ld16(ap.k_new + off);
        vr[k] = ld16(ap.v_new + off);
      }
    }
    // All rows have landed before the first store: the compiler's own waits
    // (the loads sit in masked branches) would otherwise also wait for the
    // write-through stores issued in between, one round trip per unit.
    vm_wait<0>();
#pragma unroll
    for (int k = 0; k < UK; ++k) {
      const int idx = threadIdx.x + k * kThreads;
      const int hl = idx / (16 * CPR), r = (idx / CPR) & 15, c = idx % CPR;
      if (h0 + hl < hkv && r < n) {
        st16_dev(ap.kc + pb + (size_t)(h0 + hl) * 16 * D + (size_t)(slot0 + r) * D + c * 8, kr[k]);
        st16(vt + ((size_t)hl * 16 + r) * D + c * 8, vr[k]);
      }
    }
    __syncthreads();
    // value pages: units (head, dim, half page row of 8 slots)
    for (int idx = threadIdx.x; idx < HG * 2 * D; idx += kThreads) {
      const int hl = idx / (2 * D), d = (idx >> 1) % D, half = idx & 1;
      const int lo = max(half * 8, slot0), hi = min(half * 8 + 8, slot0 + n);
      if (h0 + hl >= hkv || lo >= hi) continue;
      const uint16_t* col = vt + (size_t)hl * 16 * D + d;  // row s - slot0 at col[(s - slot0) * D]
      uint16_t* dst = ap.vc + pb + (size_t)(h0 + hl) * 16 * D + (size_t)d * 16;
      if (lo == half * 8 && hi == half * 8 + 8) {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int s0 = half * 8 + 2 * i - slot0;
          w[i] = (uint32_t)col[s0 * D] | ((uint32_t)col[(s0 + 1) * D] << 16);
        }
        st16_dev(dst + half * 8, u32x4{w[0], w[1], w[2], w[3]});
      } else {
        for (int sl = lo; sl < hi; ++sl)
          __hip_atomic_store(dst + sl, col[(sl - slot0) * D], __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    __syncthreads();  // the next pass reuses the staging area
  }
}

// kv_append: workgroup (segment, kv head).
template <int D>
__global__ __launch_bounds__(kThreads) void kv_append_kernel(const uint8_t* plan, uint64_t hash,
                                                             AppendArgs ap, const int32_t* bt,
                                                             int hkv, int maxp) {
  const PlanHeader* hdr = reinterpret_cast<const PlanHeader*>(plan);
  const AppendSeg sg = reinterpret_cast<const AppendSeg*>(plan + ap.off_segments)[blockIdx.x];
  if (hdr->magic != kPlanMagic || hdr->hash != hash) return;
  append_rows<D>(ap, sg, bt, blockIdx.y, hkv, maxp);
}

// kv_append and mixed attention in one launch.  Workgroups 0 .. append_wgs-1
// append one segment of a chunk request each (every kv head) with
// device-scope stores, then count themselves done.  The others run the
// attention work items: a chunk block that holds keys appended in this launch
// is read, at device scope, only after every appending workgroup has counted
// (they never wait, and workgroups are dispatched in index order, so they all
// run); a decode item appends its request's one new row itself.  The last
// chunk item to finish resets both counters for the next launch.
template <int D>
__global__ __launch_bounds__(kThreads, 2) void append_attention_kernel(AttnArgs a, AppendArgs ap) {
  __shared__ __attribute__((aligned(16))) char lds[Cfg<D>::LDS];
  const PlanHeader* hdr = reinterpret_cast<const PlanHeader*>(a.plan);
  int* counters = reinterpret_cast<int*>(a.ws);
  if (a.signal_dispatched && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0)
    __hip_atomic_store(&counters[kWsDispatched], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if ((int)blockIdx.x < a.append_wgs) {
    const AppendSeg sg = reinterpret_cast<const AppendSeg*>(a.plan + ap.off_segments)[blockIdx.x];
    if (hdr->magic != kPlanMagic || hdr->hash != a.hash) {
      if (threadIdx.x == 0) report(a.ws, SSA_STATUS_PLAN_MISMATCH);
      return;
    }
    append_segment_staged<D>(ap, sg, a.bt, a.hkv, a.maxp, lds);
    vm_wait<0>();  // this thread's device-scope stores have completed
    __syncthreads();
    if (threadIdx.x == 0)
      __hip_atomic_fetch_add(&counters[kCounterAppended], 1, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  const WorkItem it =
      reinterpret_cast<const WorkItem*>(a.plan + a.off_items)[(int)blockIdx.x - a.append_wgs];
  if (hdr->magic != kPlanMagic || hdr->hash != a.hash) {
    if (threadIdx.x == 0) report(a.ws, SSA_STATUS_PLAN_MISMATCH);
    return;
  }
  attention_wg<D, true>(a, it, lds);
  // Decode items never read the appended rows: only chunk items count, so the
  // many decode workgroups of a batch end without a device-scope atomic.
  if (it.kind != kItemChunk) return;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int prev = __hip_atomic_fetch_add(&counters[kCounterAttended], 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT);
    if (prev == a.num_chunk_items - 1) {
      // Take this launch's counts back off the counters: subtraction (not a
      // store of zero) returns them to their values at launch whatever the
      // timing, even if an appending workgroup counts after a timed-out wait.
      wait_appended(a);
      __hip_atomic_fetch_sub(&counters[kCounterAppended], a.append_wgs, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_fetch_sub(&counters[kCounterAttended], a.num_chunk_items, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

hipError_t clear_and_check() { return hipGetLastError(); }

}  // namespace

extern "C" {

int ssa_kv_append_timed(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                        const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache,
                        uint16_t* v_cache, const int32_t* block_table, void* stream,
                        void* start_event, void* stop_event) {
  const PlanHeader* h = nullptr;
  int rc = check_plan(shape, plan_host, &h);
  if (rc) return rc;
  if (!plan_dev) return SSA_ERR_NULL;
  if (h->num_segments == 0) return SSA_OK;
  if (!k_new || !v_new || !k_cache || !v_cache || !block_table) return SSA_ERR_NULL;
  (void)clear_and_check();
  const uint8_t* p = static_cast<const uint8_t*>(plan_dev);
  uint64_t hash = h->hash;
  AppendArgs ap{k_new, v_new, k_cache, v_cache, h->off_segments};
  int32_t hkv = h->hkv, maxp = h->max_pages_per_req;
  void* args[] = {&p, &hash, &ap, &block_table, &hkv, &maxp};
  const void* fn = h->head_dim == 128 ? reinterpret_cast<const void*>(&kv_append_kernel<128>)
                                      : reinterpret_cast<const void*>(&kv_append_kernel<64>);
  hipError_t e = hipExtLaunchKernel(fn, dim3(h->num_segments, h->hkv), dim3(kThreads), args, 0,
                                    static_cast<hipStream_t>(stream),
                                    static_cast<hipEvent_t>(start_event),
                                    static_cast<hipEvent_t>(stop_event), 0);
  return e == hipSuccess && hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

int ssa_kv_append(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                  const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache,
                  uint16_t* v_cache, const int32_t* block_table, void* stream) {
  return ssa_kv_append_timed(shape, plan_host, plan_dev, k_new, v_new, k_cache, v_cache,
                             block_table, stream, nullptr, nullptr);
}

}  // extern "C"

namespace {
// Validated attention arguments of a plan (SSA_OK, or the error to return).
int attention_args(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                   const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                   const int32_t* block_table, uint16_t* out, void* workspace,
                   size_t workspace_bytes, const PlanHeader** hp, AttnArgs* a) {
  const PlanHeader* h = nullptr;
  int rc = check_plan(shape, plan_host, &h);
  if (rc) return rc;
  if (!plan_dev) return SSA_ERR_NULL;
  *hp = h;
  if (h->num_items == 0) return SSA_OK;
  if (!q || !k_cache || !v_cache || !block_table || !out) return SSA_ERR_NULL;
  if (!workspace || workspace_bytes < (size_t)h->ws_bytes) return SSA_ERR_WORKSPACE;
  a->plan = static_cast<const uint8_t*>(plan_dev);
  a->hash = h->hash;
  a->off_items = h->off_items;
  a->off_groups = h->off_groups;
  a->ws_partials_off = h->ws_partials_off;
  a->q = q;
  a->kc = k_cache;
  a->vc = v_cache;
  a->bt = block_table;
  a->out = out;
  a->ws = static_cast<uint8_t*>(workspace);
  a->scale_log2 = h->softmax_scale * kLog2e;
  a->hq = h->hq;
  a->hkv = h->hkv;
  a->G = h->hq / h->hkv;
  a->maxp = h->max_pages_per_req;
  a->append_wgs = 0;
  a->num_chunk_items = h->num_chunk_items;
  a->wait_polls = h->wait_polls;
  a->signal_dispatched = 0;
  a->k_new = nullptr;
  a->v_new = nullptr;
  return SSA_OK;
}

// Validated arguments of a fused launch (SSA_OK, or the error to return).
int append_attention_args(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                          const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
                          uint16_t* k_cache, uint16_t* v_cache, const int32_t* block_table,
                          uint16_t* out, void* workspace, size_t workspace_bytes,
                          const PlanHeader** hp, AttnArgs* a, AppendArgs* ap) {
  int rc = attention_args(shape, plan_host, plan_dev, q, k_cache, v_cache, block_table, out,
                          workspace, workspace_bytes, hp, a);
  if (rc || (*hp)->num_items == 0) return rc;
  const PlanHeader* h = *hp;
  if (h->num_segments > 0 && (!k_new || !v_new)) return SSA_ERR_NULL;
  // the last chunk item resets the counters: appending workgroups need one
  if (h->num_chunk_segments > 0 && h->num_chunk_items == 0) return SSA_ERR_PLAN_MISMATCH;
  a->append_wgs = h->num_chunk_segments;
  a->k_new = k_new;
  a->v_new = v_new;
  *ap = AppendArgs{k_new, v_new, k_cache, v_cache, h->off_segments};
  return SSA_OK;
}

int launch_append_attention(const PlanHeader* h, AttnArgs& a, AppendArgs& ap, void* stream,
                            void* start_event, void* stop_event) {
  (void)clear_and_check();
  void* args[] = {&a, &ap};
  const void* fn = h->head_dim == 128
                       ? reinterpret_cast<const void*>(&append_attention_kernel<128>)
                       : reinterpret_cast<const void*>(&append_attention_kernel<64>);
  hipError_t e = hipExtLaunchKernel(fn, dim3(a.append_wgs + h->num_items), dim3(kThreads), args,
                                    0, static_cast<hipStream_t>(stream),
                                    static_cast<hipEvent_t>(start_event),
                                    static_cast<hipEvent_t>(stop_event), 0);
  return e == hipSuccess && hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

}  // namespace

// ------------------------------------------- the allocation-free entry point

// Scratch of ssa_append_attention_static: the fused launch's counters, status
// word, merge tickets and split records, in place of a caller's workspace.
// One copy per GPU (held until the process ends); every call on a GPU shares
// it.  In host code the name is a stand-in, not a device address: the
// per-device address comes from hipGetSymbolAddress.
constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
struct ScratchState {
  void* ptr = nullptr;    // device address of `scratch` on this device
  int64_t clean = 0;      // leading bytes that are zero at rest
};
std::mutex g_scratch_mutex;
ScratchState g_scratch[kMaxScratchDevices];

__global__ __launch_bounds__(kThreads) void clear_words_kernel(uint32_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kThreads)
    p[i] = 0u;
}

// The current device's scratch address, its first zero_bytes bytes zero when
// the launch that follows on `stream` starts.  Set-up happens on a device's
// first call (with that device current).  A call's split records start at
// its zero_bytes, so after it exactly that prefix is zero at rest (the kernel
// resets its counters and tickets); a later call with a larger prefix first
// clears the difference with a fill kernel on the same stream (no memset: a
// caller may capture the calls in a graph).
int scratch_for_launch(int64_t zero_bytes, hipStream_t stream, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return SSA_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  ScratchState& st = g_scratch[dev];
  if (!st.ptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return SSA_ERR_HIP;
    }
    st.ptr = p;
    st.clean = 0;
  }
  if (zero_bytes > st.clean) {
    const int64_t words = (zero_bytes + 3) / 4;
    const int64_t grid = std::min<int64_t>((words + kThreads - 1) / kThreads, 1024);
    (void)clear_and_check();
    hipLaunchKernelGGL(clear_words_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream,
                       static_cast<uint32_t*>(st.ptr), words);
    if (hipGetLastError() != hipSuccess) return SSA_ERR_HIP;
  }
  st.clean = zero_bytes;
  *out = st.ptr;
  return SSA_OK;
}
}  // namespace

extern "C" {

int ssa_mixed_attention_timed(const ssa_shape* shape, const void* plan_host,
                              const void* plan_dev, const uint16_t* q, const uint16_t* k_cache,
                              const uint16_t* v_cache, const int32_t* block_table, uint16_t* out,
                              void* workspace, size_t workspace_bytes, void* stream,
                              void* start_event, void* stop_event) {
  const PlanHeader* h = nullptr;
  AttnArgs a;
  int rc = attention_args(shape, plan_host, plan_dev, q, k_cache, v_cache, block_table, out,
                          workspace, workspace_bytes, &h, &a);
  if (rc || h->num_items == 0) return rc;
  (void)clear_and_check();
  void* args[] = {&a};
  const void* fn = h->head_dim == 128
                       ? reinterpret_cast<const void*>(&mixed_attention_kernel<128>)
                       : reinterpret_cast<const void*>(&mixed_attention_kernel<64>);
  hipError_t e = hipExtLaunchKernel(fn, dim3(h->num_items), dim3(kThreads), args, 0,
                                    static_cast<hipStream_t>(stream),
                                    static_cast<hipEvent_t>(start_event),
                                    static_cast<hipEvent_t>(stop_event), 0);
  return e == hipSuccess && hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

int ssa_mixed_attention(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                        const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                        const int32_t* block_table, uint16_t* out, void* workspace,
                        size_t workspace_bytes, void* stream) {
  return ssa_mixed_attention_timed(shape, plan_host, plan_dev, q, k_cache, v_cache, block_table,
                                   out, workspace, workspace_bytes, stream, nullptr, nullptr);
}

int ssa_append_attention(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                         const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
                         uint16_t* k_cache, uint16_t* v_cache, const int32_t* block_table,
                         uint16_t* out, void* workspace, size_t workspace_bytes, void* stream,
                         void* start_event, void* stop_event) {
  const PlanHeader* h = nullptr;
  AttnArgs a;
  AppendArgs ap;
  int rc = append_attention_args(shape, plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache,
                                 block_table, out, workspace, workspace_bytes, &h, &a, &ap);
  if (rc || h->num_items == 0) return rc;
  return launch_append_attention(h, a, ap, stream, start_event, stop_event);
}

int ssa_append_attention_static(const ssa_shape* shape, const void* plan_host,
                                const void* plan_dev, const uint16_t* q, const uint16_t* k_new,
                                const uint16_t* v_new, uint16_t* k_cache, uint16_t* v_cache,
                                const int32_t* block_table, uint16_t* out, void* stream,
                                void* start_event, void* stop_event) {
  const PlanHeader* h = nullptr;
  AttnArgs a;
  AppendArgs ap;
  // every argument is checked before any HIP call: the scratch stands in as a
  // workspace of its size at a placeholder address until it is resolved
  int rc = check_plan(shape, plan_host, &h);
  if (rc) return rc;
  if (h->ws_bytes > (int64_t)kScratchBytes) return SSA_ERR_WORKSPACE;
  rc = append_attention_args(shape, plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache,
                             block_table, out, reinterpret_cast<void*>(kScratchBytes),
                             kScratchBytes, &h, &a, &ap);
  if (rc || h->num_items == 0) return rc;
  void* ws = nullptr;
  rc = scratch_for_launch(h->ws_partials_off, static_cast<hipStream_t>(stream), &ws);
  if (rc) return rc;
  a.ws = static_cast<uint8_t*>(ws);
  return launch_append_attention(h, a, ap, stream, start_event, stop_event);
}

}  // extern "C"

// ------------------------------------------------ the two-stream launch pair

namespace {
// Fork and join events of ssa_append_attention_streams, per host thread and
// device (created on first use, kept until the thread ends): two threads never
// record the same event.
struct ForkJoin {
  hipEvent_t fork = nullptr, join = nullptr;
};
thread_local ForkJoin t_fork_join[kMaxScratchDevices];

int fork_join_events(ForkJoin** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return SSA_ERR_HIP;
  ForkJoin& fj = t_fork_join[dev];
  for (hipEvent_t* e : {&fj.fork, &fj.join}) {
    if (*e) continue;
    if (hipEventCreateWithFlags(e, hipEventDisableTiming) != hipSuccess) {
      *e = nullptr;
      (void)hipGetLastError();
      return SSA_ERR_HIP;
    }
  }
  *out = &fj;
  return SSA_OK;
}

// The plan puts every chunk item before every decode item, and decode items
// start on 32-key block boundaries (both as the planner writes them with
// mix_order 1).
bool chunk_items_first(const PlanHeader* h, const void* plan_host) {
  const WorkItem* items =
      reinterpret_cast<const WorkItem*>(static_cast<const uint8_t*>(plan_host) + h->off_items);
  for (int i = 0; i < h->num_items; ++i) {
    const bool chunk = i < h->num_chunk_items;
    if ((items[i].kind == kItemChunk) != chunk) return false;
    if (!chunk && (items[i].key0 & 31)) return false;
  }
  return true;
}
}  // namespace

extern "C" {

int ssa_append_attention_streams(const ssa_shape* shape, const void* plan_host,
                                 const void* plan_dev, const uint16_t* q, const uint16_t* k_new,
                                 const uint16_t* v_new, uint16_t* k_cache, uint16_t* v_cache,
                                 const int32_t* block_table, uint16_t* out, void* workspace,
                                 size_t workspace_bytes, void* stream, void* decode_stream,
                                 void* start_event, void* stop_event) {
  const PlanHeader* h = nullptr;
  AttnArgs a;
  AppendArgs ap;
  int rc = append_attention_args(shape, plan_host, plan_dev, q, k_new, v_new, k_cache, v_cache,
                                 block_table, out, workspace, workspace_bytes, &h, &a, &ap);
  if (rc || h->num_items == 0) return rc;
  // the one-launch path on `stream`: a plan that does not ask for the split,
  // shapes the decode kernel does not take, batches without decode rows
  const int nd = h->num_decode_items;
  if (h->streams_beside < 0 || h->head_dim != kStreamD || a.G > kStreamMaxG || nd == 0 ||
      !chunk_items_first(h, plan_host))
    return launch_append_attention(h, a, ap, stream, start_event, stop_event);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipStream_t sd = static_cast<hipStream_t>(decode_stream);
  ForkJoin* fj = nullptr;
  rc = fork_join_events(&fj);
  if (rc) return rc;
  (void)clear_and_check();
  bool ok = true;
  hipEvent_t e0 = static_cast<hipEvent_t>(start_event), e1 = static_cast<hipEvent_t>(stop_event);
  const bool two = h->num_chunk_items > 0;
  if (two) {
    ok = ok && hipEventRecord(fj->fork, s) == hipSuccess;
    ok = ok && hipStreamWaitEvent(sd, fj->fork, 0) == hipSuccess;
    // the chunk rows (two workgroups per CU); the last workgroup to be placed
    // releases the decode launch
    AttnArgs ca = a;
    ca.signal_dispatched = 1;
    void* cargs[] = {&ca, &ap};
    ok = ok && hipExtLaunchKernel(reinterpret_cast<const void*>(&append_attention_kernel<kStreamD>),
                                  dim3(a.append_wgs + h->num_chunk_items), dim3(kThreads), cargs, 0,
                                  s, e0, e1, 0) == hipSuccess;
  }
  // decode items: the first `beside` of them (longest first) on the decode
  // stream once the chunk launch has placed its workgroups, the rest in one
  // launch on the chunk stream after the chunk rows
  const int beside = two ? std::min(h->streams_beside, nd) : 0;
  const void* dfn = reinterpret_cast<const void*>(&decode_stream_kernel);
  if (beside > 0) {
    int* flag = reinterpret_cast<int*>(a.ws) + kWsDispatched;
    int polls = kWaitDispatchedPolls;
    void* wargs[] = {&flag, &polls};
    ok = ok && hipExtLaunchKernel(reinterpret_cast<const void*>(&wait_dispatched_kernel), dim3(1),
                                  dim3(64), wargs, 0, sd, nullptr, nullptr, 0) == hipSuccess;
    int item0 = h->num_chunk_items;
    void* dargs[] = {&a, &item0};
    ok = ok && hipExtLaunchKernel(dfn, dim3(beside), dim3(kThreads), dargs, 0, sd, nullptr, nullptr,
                                  0) == hipSuccess;
  }
  if (beside < nd) {
    int item0 = h->num_chunk_items + beside;
    void* dargs[] = {&a, &item0};
    ok = ok && hipExtLaunchKernel(dfn, dim3(nd - beside), dim3(kThreads), dargs, 0, s,
                                  two ? nullptr : e0, two ? nullptr : e1, 0) == hipSuccess;
  }
  if (two) {
    ok = ok && hipEventRecord(fj->join, sd) == hipSuccess;
    ok = ok && hipStreamWaitEvent(s, fj->join, 0) == hipSuccess;
  }
  return ok && hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

}  // extern "C"
