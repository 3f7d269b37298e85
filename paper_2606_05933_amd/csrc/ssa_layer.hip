// HIP kernels for gfx950 of the layer steps around attention (include/ssa_layer.h).
//
// ssa_rope_append: for each append segment of the plan (consecutive new
// tokens of one request inside one page, at most 16), workgroups of 8 heads
// each.  A rotating workgroup rotates 8 of the segment's query and key heads
// (rotate-half pairs (i, i + D/2), cos/sin from the position's row of the
// table) and writes the queries to q_out and the keys to their slots of the
// key page (slot-major rows); a value workgroup stages 8 value heads' rows in
// LDS and writes them to the dim-major value page as 16-byte half rows (8
// slots of one dim), the layout ssa_mixed_attention reads.  Each thread issues
// all its loads before its first store.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ssa_layer.h"
#include "ssa_device.h"
#include "ssa_plan_format.h"

namespace ssa {
int check_plan(const ssa_shape* s, const void* plan_host, const PlanHeader** out);
}

namespace {
using namespace ssa;
using namespace ssa_dev;

constexpr int kLayerThreads = 256;

// Rotate 8 pairs: x1 = dims i..i+7, x2 = dims i+D/2..i+D/2+7 of one head.
__device__ __forceinline__ void rotate8(u32x4 x1, u32x4 x2, const float* cs, int half, int i,
                                        u32x4* o1, u32x4* o2) {
  const f32x4 c0 = *reinterpret_cast<const f32x4*>(cs + i);
  const f32x4 c1 = *reinterpret_cast<const f32x4*>(cs + i + 4);
  const f32x4 s0 = *reinterpret_cast<const f32x4*>(cs + half + i);
  const f32x4 s1 = *reinterpret_cast<const f32x4*>(cs + half + i + 4);
  const float c[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
  const float s[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float a0 = bf16_lo(x1[w]), a1 = bf16_hi(x1[w]);
    const float b0 = bf16_lo(x2[w]), b1 = bf16_hi(x2[w]);
    const int k = 2 * w;
    (*o1)[w] = pack2(a0 * c[k] - b0 * s[k], a1 * c[k + 1] - b1 * s[k + 1]);
    (*o2)[w] = pack2(b0 * c[k] + a0 * s[k], b1 * c[k + 1] + a1 * s[k + 1]);
  }
}

struct RopeArgs {
  const uint8_t* plan;
  uint64_t hash;
  int32_t off_segments;
  const uint16_t* qkv;
  const float* cos_sin;
  uint16_t* q_out;
  uint16_t* kc;
  uint16_t* vc;
  const int32_t* bt;
  int hq, hkv, maxp;
};

// Heads per workgroup: blockIdx.y < rot_groups rotates query/key heads
// 8 y .. 8 y + 7 (of the Hq + Hkv rotated ones); the others copy value heads.
constexpr int kHeadGroup = 8;

template <int D>
__global__ __launch_bounds__(kLayerThreads) void rope_append_kernel(RopeArgs a) {
  constexpr int HALF = D / 2, UPH = HALF / 8;     // 8-pair units per head
  constexpr int HG = kHeadGroup;
  constexpr int RU = 16 * HG * UPH / kLayerThreads;  // rotation units per thread
  constexpr int VU = 16 * HG * (D / 8) / kLayerThreads;  // value chunks per thread
  constexpr int TU = HG * 2 * D / kLayerThreads;     // value half rows per thread
  __shared__ __attribute__((aligned(16))) uint16_t vt[HG * 16 * D];  // [head][row][D]
  const PlanHeader* hdr = reinterpret_cast<const PlanHeader*>(a.plan);
  const AppendSeg sg = reinterpret_cast<const AppendSeg*>(a.plan + a.off_segments)[blockIdx.x];
  if (hdr->magic != kPlanMagic || hdr->hash != a.hash) return;
  const int n = sg.n, slot0 = sg.pos0 % 16, tid = threadIdx.x;
  const size_t stride = (size_t)(a.hq + 2 * a.hkv) * D;
  const size_t pb = (size_t)a.bt[(size_t)sg.req * a.maxp + sg.pos0 / 16] * a.hkv * 16 * D;
  const int nrot = a.hq + a.hkv, rot_groups = (nrot + HG - 1) / HG;
  if ((int)blockIdx.y < rot_groups) {
    // query and key heads h0 .. h0 + nh - 1: units (row, head, 8 pairs); all
    // loads first, then the rotations and stores
    const int h0 = blockIdx.y * HG, nh = min(HG, nrot - h0);
    const int nu = n * nh * UPH;
    u32x4 x1[RU], x2[RU];
#pragma unroll
    for (int j = 0; j < RU; ++j) {
      const int idx = tid + j * kLayerThreads;
      if (idx >= nu) continue;
      const int r = idx / (nh * UPH), rem = idx % (nh * UPH);
      const int h = h0 + rem / UPH, i = (rem % UPH) * 8;
      const uint16_t* src = a.qkv + (size_t)(sg.row0 + r) * stride + (size_t)h * D;
      x1[j] = ld16(src + i);
      x2[j] = ld16(src + HALF + i);
    }
#pragma unroll
    for (int j = 0; j < RU; ++j) {
      const int idx = tid + j * kLayerThreads;
      if (idx >= nu) continue;
      const int r = idx / (nh * UPH), rem = idx % (nh * UPH);
      const int h = h0 + rem / UPH, i = (rem % UPH) * 8;
      u32x4 o1, o2;
      rotate8(x1[j], x2[j], a.cos_sin + (size_t)(sg.pos0 + r) * D, HALF, i, &o1, &o2);
      uint16_t* dst = h < a.hq ? a.q_out + ((size_t)(sg.row0 + r) * a.hq + h) * D
                               : a.kc + pb + (size_t)(h - a.hq) * 16 * D + (size_t)(slot0 + r) * D;
      st16(dst + i, o1);
      st16(dst + HALF + i, o2);
    }
    return;
  }
  // value heads h0 .. h0 + nh - 1: rows to LDS, then 8-slot half rows of one dim
  const int h0 = ((int)blockIdx.y - rot_groups) * HG, nh = min(HG, a.hkv - h0);
  const int nv = n * nh * (D / 8);
  u32x4 v[VU];
#pragma unroll
  for (int j = 0; j < VU; ++j) {
    const int idx = tid + j * kLayerThreads;
    if (idx >= nv) continue;
    const int r = idx / (nh * (D / 8)), rem = idx % (nh * (D / 8));
    const int hl = rem / (D / 8), c = rem % (D / 8);
    v[j] = ld16(a.qkv + (size_t)(sg.row0 + r) * stride + (size_t)(a.hq + a.hkv + h0 + hl) * D + c * 8);
  }
#pragma unroll
  for (int j = 0; j < VU; ++j) {
    const int idx = tid + j * kLayerThreads;
    if (idx >= nv) continue;
    const int r = idx / (nh * (D / 8)), rem = idx % (nh * (D / 8));
    const int hl = rem / (D / 8), c = rem % (D / 8);
    st16(vt + ((size_t)hl * 16 + r) * D + c * 8, v[j]);
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < TU; ++j) {
    const int idx = tid + j * kLayerThreads;
    if (idx >= nh * 2 * D) continue;
    const int hl = idx / (2 * D), d = (idx >> 1) % D, half = idx & 1;
    const int lo = max(half * 8, slot0), hi = min(half * 8 + 8, slot0 + n);
    if (lo >= hi) continue;
    const uint16_t* col = vt + (size_t)hl * 16 * D + d;  // slot s at col[(s - slot0) * D]
    uint16_t* dst = a.vc + pb + (size_t)(h0 + hl) * 16 * D + (size_t)d * 16;
    if (lo == half * 8 && hi == half * 8 + 8) {
      uint32_t w[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int s0 = half * 8 + 2 * k - slot0;
        w[k] = (uint32_t)col[s0 * D] | ((uint32_t)col[(s0 + 1) * D] << 16);
      }
      st16(dst + half * 8, u32x4{w[0], w[1], w[2], w[3]});
    } else {
      for (int s = lo; s < hi; ++s) dst[s] = col[(s - slot0) * D];
    }
  }
}

}  // namespace

extern "C" {

int ssa_rope_append(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                    const uint16_t* qkv, const float* cos_sin, int32_t max_position,
                    uint16_t* q_out, uint16_t* k_cache, uint16_t* v_cache,
                    const int32_t* block_table, void* stream) {
  const PlanHeader* h = nullptr;
  int rc = check_plan(shape, plan_host, &h);
  if (rc) return rc;
  if (!plan_dev) return SSA_ERR_NULL;
  const ReqEntry* reqs = reinterpret_cast<const ReqEntry*>(
      static_cast<const uint8_t*>(plan_host) + h->off_reqs);
  for (int32_t i = 0; i < h->num_reqs; ++i)
    if (reqs[i].q_len > 0 && (int64_t)reqs[i].ctx_len + reqs[i].q_len > max_position)
      return SSA_ERR_ARG;
  if (h->num_segments == 0) return SSA_OK;
  if (!qkv || !cos_sin || !q_out || !k_cache || !v_cache || !block_table) return SSA_ERR_NULL;
  (void)hipGetLastError();
  RopeArgs a{static_cast<const uint8_t*>(plan_dev), h->hash, h->off_segments, qkv, cos_sin,
             q_out, k_cache, v_cache, block_table, h->hq, h->hkv, h->max_pages_per_req};
  const dim3 grid(h->num_segments, (h->hq + h->hkv + kHeadGroup - 1) / kHeadGroup +
                                       (h->hkv + kHeadGroup - 1) / kHeadGroup);
  if (h->head_dim == 128)
    hipLaunchKernelGGL(rope_append_kernel<128>, grid, dim3(kLayerThreads), 0,
                       static_cast<hipStream_t>(stream), a);
  else
    hipLaunchKernelGGL(rope_append_kernel<64>, grid, dim3(kLayerThreads), 0,
                       static_cast<hipStream_t>(stream), a);
  return hipGetLastError() == hipSuccess ? SSA_OK : SSA_ERR_HIP;
}

}  // extern "C"
