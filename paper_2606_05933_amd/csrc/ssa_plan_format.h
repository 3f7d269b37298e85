// Plan blob of one iteration: written by the host planner, read unchanged by
// the kernels after a byte copy to device memory.  Every field is a fixed-size
// integer or float at a fixed offset, so host and device agree byte for byte.
//
//   [PlanHeader 128 B][ReqEntry x num_reqs][WorkItem x num_items]
//   [MergeGroup x num_groups][AppendSeg x num_segments]
//
// The workspace holds kLaunchCounters int32 words (a fused launch's two
// counters, the sticky status word of ssa.h, the two-stream launch's dispatch
// flag) and one int32 ticket
// per merge group (counters and tickets zero at rest), padded to 256 bytes, then,
// at ws_partials_off, fp32 partial results:
// for merge group g and split s, a record of rec_floats(ncols, D) floats at
// float offset ws_off + s * rec_floats(ncols, D): m[ncols], l[ncols], padding
// to a multiple of four floats, o[ncols][D] (so that every o row, like every
// record, starts 16-byte aligned).
#pragma once
#include <stdint.h>

namespace ssa {

constexpr uint32_t kPlanMagic = 0x31415353u;  // "SSA1"
constexpr uint32_t kPlanVersion = 5;
constexpr int kBlockKeys = 32;  // keys per attention block: two 16-slot pages
constexpr int kWaves = 4;       // waves per workgroup
constexpr int kThreads = 256;   // threads per workgroup
constexpr int kChunkWaveCols = 32;  // columns a wave owns in a chunk tile
constexpr int kLaunchCounters = 4;  // workspace words ahead of the merge tickets
constexpr int kWsStatusWord = 2;    // the status word among them (ssa.h)
constexpr int kWsDispatched = 3;    // set once a chunk launch has started all its workgroups
constexpr int kDefaultWaitPolls = 1 << 21;

// Float offset of o in a partial record of ncols columns, and the record's size.
constexpr int64_t rec_o_off(int ncols) { return ((int64_t)2 * ncols + 3) / 4 * 4; }
constexpr int64_t rec_floats(int ncols, int d) { return rec_o_off(ncols) + (int64_t)ncols * d; }

enum ItemKind : int32_t { kItemChunk = 0, kItemDecode = 1 };

struct PlanHeader {
  uint32_t magic;
  uint32_t version;
  uint64_t hash;  // FNV-1a of the shape, the tuning and the length arrays
  int32_t num_reqs, num_tokens;
  int32_t num_items, num_chunk_items, num_decode_items, num_groups, num_segments;
  int32_t hq, hkv, head_dim, page_size, max_pages_per_req, num_pages;
  int32_t chunk_tile_cols;
  int32_t off_reqs, off_items, off_groups, off_segments;  // byte offsets in the blob
  int64_t ws_partials_off;  // byte offset of the partial records in the workspace
  int64_t ws_bytes;         // workspace bytes the plan needs (at least 256)
  int64_t plan_bytes;       // total blob size
  float softmax_scale;
  int32_t num_chunk_segments;  // segments of chunk requests (c > 1): the first ones
  int32_t wait_polls;          // polls before a fused launch's wait for appended rows gives up
  // ssa_append_attention_streams: decode items (the first ones after the chunk
  // items) that run beside the chunk rows on the decode stream, the others
  // after them; -1: the call runs as one launch
  int32_t streams_beside;
};
static_assert(sizeof(PlanHeader) == 128, "plan header size");

struct ReqEntry {
  int32_t q_start;  // first token row of the request in q / out / k_new / v_new
  int32_t q_len;    // c_i
  int32_t ctx_len;  // u_i
  int32_t n_pages;  // ceil((u_i + c_i) / P): block-table entries that may be read
};

// One workgroup of the attention launch.
//   chunk tile: columns [col0, col0 + ncols) of the request's column space, where
//     column n is (token j = n / G, q head kvh * G + n % G); keys [key0, key1).
//   decode split: the request's single new token, q heads kvh*G .. kvh*G+G-1
//     (ncols = G), keys [key0, key1).
// group < 0: the item writes the final output; otherwise it writes partial
// record `split` of merge group `group`, and the last of the group's items to
// finish merges them.  The request fields a workgroup needs are copied into the
// item, so that a workgroup reads one record of the plan before it starts.
struct WorkItem {
  int32_t kind;
  int32_t req;
  int32_t kvh;
  int32_t col0;
  int32_t ncols;
  int32_t key0;
  int32_t key1;
  int32_t group;
  int32_t split;
  int32_t q_start;  // the request's first token row (copied from its ReqEntry)
  int32_t ctx_len;  // u_i
  int32_t nvalid;   // u_i + c_i: keys that hold data after the append
};
static_assert(sizeof(WorkItem) == 48, "work item size");

struct MergeGroup {
  int32_t nsplit;
  int32_t ncols;
  int64_t ws_off;  // float offset of split 0's record from ws_partials_off
};

// kv_append: n consecutive new tokens of one request that land in one page.
struct AppendSeg {
  int32_t req;
  int32_t row0;  // token row of the first of them
  int32_t pos0;  // its position u_i + j
  int32_t n;
};

}  // namespace ssa
