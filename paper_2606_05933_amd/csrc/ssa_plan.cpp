// Host side of the library: argument validation, the iteration plan, status
// strings.  Pure host code (no HIP call), so it is testable without a GPU.
//
// The plan turns the batch B = {(c_i, u_i)} (SlidingServe Sec. 3.2) into the
// work of one attention launch:
//   - request starts: q_start_i = c_0 + ... + c_{i-1};
//   - routing by Eq. 2: c_i == 1 -> decode split items, c_i > 1 -> chunk tile
//     items, c_i == 0 -> nothing (it belongs to the decode set but has no row);
//   - merge groups for items that cover only part of a key range;
//   - append segments for kv_append (new tokens cut at page boundaries);
//   - the scene of Eq. 3 and the batch features x1..x7 of Tab. 1.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <functional>
#include <new>
#include <vector>

#include "../../include/ssa.h"
#include "ssa_plan_format.h"

namespace ssa {
namespace {

constexpr int kDefaultTileCols = 128;
constexpr int kDefaultCus = 256;
constexpr int kMaxLen = 1 << 30;
// Nominal rates for balancing only (fractions of MI355X peaks): bf16 MFMA per
// CU at half of peak, HBM at 70% of 8 TB/s shared by all CUs.
constexpr double kMfmaRatePerCu = 2.5e15 / 256.0 * 0.5;
constexpr double kHbmRate = 8.0e12 * 0.7;
// A chunk tile's key range is cut only into pieces of at least this many keys:
// each piece costs a partial record of ncols*(D+2) floats written and read back.
constexpr int kMinChunkSplitKeys = 1024;
constexpr int kMaxChunkSplits = 16;
// What one extra piece of a split chunk tile costs, in keys of the tile's work
// (its prologue, partial record and share of the merge; measured: three
// pieces of a 33k-key tile about 6% slower than one).
constexpr double kSplitCostKeys = 768.0;
// Decode key ranges are cut into equal pieces of about this many keys: long
// enough that the load latency at the start of an item is amortised over 32
// blocks per wave, short enough that long and short contexts balance over the
// compute units; partial records cost G*(D+2) floats per piece.
constexpr int kDefaultDecodeSplitKeys = 3072;

// Work items of one launch: their blob section must stay within the int32
// offsets of the plan header (and the grid within 2^31 workgroups).
constexpr int64_t kMaxItems = (INT32_MAX - (1 << 20)) / (int64_t)sizeof(WorkItem);

constexpr int kDefaultXcds = 1;
constexpr int kOrderChunkFirst = 1;
constexpr int kOrderInterleave = 2;
constexpr int kOrderPaired = 3;
constexpr int kOrderPairedDecodeFirst = 4;
// automatic order: paired once decode time / chunk time (both estimated) reaches this
constexpr double kPairedMinRatio = 0.85;
// automatic order: paired, then the other decode items first, from this ratio up
constexpr double kPairedDecodeFirstRatio = 0.25;
// mix_order values for ssa_append_attention_streams: automatic, and the split
// forced (half of the decode items beside the chunk rows, half after them)
constexpr int kOrderStreamsAuto = 5;
constexpr int kOrderStreamsForced = 6;
// The two-stream split (ssa_append_attention_streams) pays where the chunk
// items fill both slots of (nearly) every compute unit in one round, so that
// decode work can only take a third slot beside them and no chunk tile waits
// for a slot that decode work holds, and where the decode rows nearly all fit in
// the time the chunk rows take: decode bytes streamed at the rate that one
// decode workgroup per CU reaches beside two chunk tiles, for the chunk rows'
// flops at their rate with that company (both measured on MI355X, on the
// 70B-shaped batch).  The decode items that fit run beside, the rest after.
constexpr double kBesideChunkFlops = 0.95e15;  // chunk rows, flop/s
constexpr double kBesideDecodeBytes = 2.5e12;  // decode rows, bytes/s
constexpr double kBesideMinCover = 0.9;        // share of the decode bytes that must fit
constexpr double kBesideMinFill = 1.5;         // chunk items per compute unit, at least

struct Tuning {
  int tile_cols, chunk_split_keys, decode_split_keys, num_cus, num_xcds, mix_order, wait_polls;
  int auto_order;  // the caller left mix_order at 0: the planner picks it (int: no padding)
  int streams;     // 0: one-launch plan; 1: split when it pays (mix_order 5); 2: forced (6)
};

int check_shape(const ssa_shape* s) {
  if (!s) return SSA_ERR_NULL;
  if (s->num_q_heads <= 0 || s->num_kv_heads <= 0 || s->num_q_heads % s->num_kv_heads != 0 ||
      s->num_q_heads / s->num_kv_heads > 16)
    return SSA_ERR_SHAPE;
  if (s->head_dim != 64 && s->head_dim != 128) return SSA_ERR_HEAD_DIM;
  if (s->page_size != SSA_PAGE_SIZE) return SSA_ERR_PAGE_SIZE;
  if (!std::isfinite(s->softmax_scale) || s->softmax_scale < 0.f) return SSA_ERR_SCALE;
  if (s->num_pages < 1 || s->max_pages_per_req < 1) return SSA_ERR_PAGES;
  return SSA_OK;
}

int resolve_tuning(const ssa_tuning* t, Tuning* out) {
  Tuning r{kDefaultTileCols, 0,    0, kDefaultCus, kDefaultXcds, kOrderChunkFirst, kDefaultWaitPolls,
           1,                0};
  if (t) {
    if (t->chunk_tile_cols) {
      if (t->chunk_tile_cols != 32 && t->chunk_tile_cols != 64 && t->chunk_tile_cols != 128)
        return SSA_ERR_TUNING;
      r.tile_cols = t->chunk_tile_cols;
    }
    if (t->chunk_split_keys < 0 || t->chunk_split_keys % kBlockKeys) return SSA_ERR_TUNING;
    if (t->decode_split_keys < 0 || t->decode_split_keys % kBlockKeys) return SSA_ERR_TUNING;
    if (t->num_cus < 0 || t->num_cus > 4096) return SSA_ERR_TUNING;
    if (t->num_xcds < 0 || t->num_xcds > 64) return SSA_ERR_TUNING;
    if (t->mix_order < 0 || t->mix_order > kOrderStreamsForced) return SSA_ERR_TUNING;
    if (t->append_wait_polls < 0) return SSA_ERR_TUNING;
    if (t->append_wait_polls) r.wait_polls = t->append_wait_polls;
    r.chunk_split_keys = t->chunk_split_keys;
    r.decode_split_keys = t->decode_split_keys;
    if (t->num_cus) r.num_cus = t->num_cus;
    if (t->num_xcds) r.num_xcds = t->num_xcds;
    if (t->mix_order == kOrderStreamsAuto) {
      r.streams = 1;  // the automatic order, or chunk items first where the split pays
    } else if (t->mix_order == kOrderStreamsForced) {
      r.streams = 2;
      r.mix_order = kOrderChunkFirst;
      r.auto_order = 0;
    } else if (t->mix_order) {
      r.mix_order = t->mix_order;
      r.auto_order = 0;
    }
  }
  *out = r;
  return SSA_OK;
}

uint64_t fnv1a(uint64_t h, const void* p, size_t n) {
  const unsigned char* b = static_cast<const unsigned char*>(p);
  for (size_t i = 0; i < n; ++i) {
    h ^= b[i];
    h *= 1099511628211ull;
  }
  return h;
}

struct Plan {
  std::vector<ReqEntry> reqs;
  std::vector<WorkItem> items;
  std::vector<MergeGroup> groups;
  std::vector<AppendSeg> segs;
  int32_t num_chunk_segs = 0;
  PlanHeader hdr;
  ssa_plan_info info;
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Coarse log-scale bucket of an item's estimated duration (16 buckets per
// factor of two): ordering only needs to be approximate.
constexpr int kTimeBuckets = 1024;
int time_bucket(double t) {
  // t in units of 1/1024 ns, as an integer: 16 * floor(log2) + the next 4 bits
  const double x = t * 1.024e12;
  const uint64_t v = x < 1.0 ? 1 : (x > 9.0e18 ? (uint64_t)9.0e18 : (uint64_t)x);
  const int msb = 63 - __builtin_clzll(v);
  const int frac = msb >= 4 ? (int)((v >> (msb - 4)) & 15) : (int)((v << (4 - msb)) & 15);
  return std::min(kTimeBuckets - 1, msb * 16 + frac);
}

// Indices of the items of one kind (kind < 0: all), longest first: a counting
// sort on the time bucket, stable, hence deterministic.
void longest_first(const std::vector<WorkItem>& items, const std::vector<uint16_t>& bucket,
                   int kind, std::vector<uint32_t>* out) {
  static thread_local std::vector<int> count;
  count.assign(kTimeBuckets + 1, 0);
  size_t n = 0;
  for (size_t k = 0; k < items.size(); ++k)
    if (kind < 0 || items[k].kind == kind) {
      count[kTimeBuckets - 1 - bucket[k]]++;
      ++n;
    }
  int acc = 0;
  for (int b = 0; b <= kTimeBuckets; ++b) {
    const int c = count[b];
    count[b] = acc;
    acc += c;
  }
  const size_t base = out->size();
  out->resize(base + n);
  for (size_t k = 0; k < items.size(); ++k)
    if (kind < 0 || items[k].kind == kind) (*out)[base + count[kTimeBuckets - 1 - bucket[k]]++] = (uint32_t)k;
}

// Chunk and decode index lists of one queue: all chunk items then the decode
// items, the two merged in proportion, or paired: the dispatcher gives the
// first `cus` workgroups one compute unit each and the next `cus` the second
// slot of the same units, so the first min(cus, chunk items) chunk items are
// followed by enough decode items to fill the second slots (every unit then
// runs one MFMA-bound and one HBM-bound item side by side), and the rest
// follows merged in proportion or, for order 4, the rest of the decode items
// before the rest of the chunk items (units go back to two chunk tiles each
// once the decode work is gone).
void mix(const std::vector<uint32_t>& a, const std::vector<uint32_t>& b, int order, int cus,
         std::vector<uint32_t>* out) {
  if (order == kOrderChunkFirst) {
    out->insert(out->end(), a.begin(), a.end());
    out->insert(out->end(), b.begin(), b.end());
    return;
  }
  size_t i = 0, j = 0;
  if (order == kOrderPaired || order == kOrderPairedDecodeFirst) {
    i = std::min(a.size(), (size_t)cus);
    j = std::min(b.size(), 2 * (size_t)cus - i);
    out->insert(out->end(), a.begin(), a.begin() + i);
    out->insert(out->end(), b.begin(), b.begin() + j);
    if (order == kOrderPairedDecodeFirst) {  // then the other decode items, then the chunk items
      out->insert(out->end(), b.begin() + j, b.end());
      out->insert(out->end(), a.begin() + i, a.end());
      return;
    }
  }
  const size_t i0 = i, j0 = j;
  while (i < a.size() || j < b.size()) {
    // take from the list that is behind in the fraction of its items emitted
    const bool take_a = j >= b.size() || (i < a.size() && (double)(i - i0) * (b.size() - j0) <=
                                                                (double)(j - j0) * (a.size() - i0));
    out->push_back(take_a ? a[i++] : b[j++]);
  }
}

// Launch order of the work items (indices into `items`).  The dispatcher hands
// out workgroups in index order, so long items go first: by default all chunk
// items, longest first, then the decode items, longest first.  With die-aware
// placement (num_xcds > 1; workgroup b is taken to run on die b mod X), chunk
// items that read the same K/V (one request and kv head) go to one die, dies
// get equal item counts (decode items balance the estimated time), and the
// dies' queues are interleaved so that position b belongs to die b mod X.
void order_items(const std::vector<WorkItem>& items, const std::vector<double>& t,
                 const std::vector<uint16_t>& bucket, const Tuning& tu, int Hkv,
                 std::vector<uint32_t>* seq) {
  const size_t N = items.size();
  seq->clear();
  seq->reserve(N);
  std::vector<uint32_t> ch, de;
  longest_first(items, bucket, kItemChunk, &ch);
  longest_first(items, bucket, kItemDecode, &de);
  const int X = tu.num_xcds;
  if (X > 1 && N > 0) {
    std::vector<std::vector<uint32_t>> sch(X), sde(X);
    std::vector<double> load(X, 0.0);
    std::vector<size_t> cap(X);
    for (int x = 0; x < X; ++x) cap[x] = N / X + ((size_t)x < N % X ? 1 : 0);
    // chunk streams (request, kv head) to dies, largest first onto the least loaded
    std::vector<int64_t> ids;
    std::vector<double> stime;
    std::vector<size_t> sid_of(N, 0);
    for (uint32_t k : ch) {
      const int64_t sid = (int64_t)items[k].req * Hkv + items[k].kvh;
      size_t q = 0;
      while (q < ids.size() && ids[q] != sid) ++q;
      if (q == ids.size()) {
        ids.push_back(sid);
        stime.push_back(0.0);
      }
      stime[q] += t[k];
      sid_of[k] = q;
    }
    std::vector<size_t> sorder(ids.size());
    for (size_t q = 0; q < sorder.size(); ++q) sorder[q] = q;
    std::stable_sort(sorder.begin(), sorder.end(),
                     [&](size_t a, size_t b) { return stime[a] > stime[b]; });
    std::vector<int> sx(ids.size(), 0);
    for (size_t q : sorder) {
      int best = 0;
      for (int x = 1; x < X; ++x)
        if (load[x] < load[best]) best = x;
      sx[q] = best;
      load[best] += stime[q];
    }
    for (uint32_t k : ch) sch[sx[sid_of[k]]].push_back(k);
    bool fits = true;
    for (int x = 0; x < X; ++x) fits = fits && sch[x].size() <= cap[x];
    if (fits) {
      for (uint32_t k : de) {  // longest first onto the least loaded die with room
        int best = -1;
        for (int x = 0; x < X; ++x)
          if (sch[x].size() + sde[x].size() < cap[x] && (best < 0 || load[x] < load[best]))
            best = x;
        sde[best].push_back(k);
        load[best] += t[k];
      }
      std::vector<std::vector<uint32_t>> q(X);
      for (int x = 0; x < X; ++x) mix(sch[x], sde[x], tu.mix_order, tu.num_cus / X, &q[x]);
      for (size_t r = 0; seq->size() < N; ++r)
        for (int x = 0; x < X; ++x)
          if (r < q[x].size()) seq->push_back(q[x][r]);
      return;
    }
  }
  mix(ch, de, tu.mix_order, tu.num_cus, seq);
}

int build(const ssa_shape* s, const int32_t* q_len, const int32_t* ctx_len, int32_t n,
          const ssa_tuning* tuning, Plan* p) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (n < 0) return SSA_ERR_LENGTH;
  if (n > 0 && (!q_len || !ctx_len)) return SSA_ERR_NULL;
  Tuning tu;
  rc = resolve_tuning(tuning, &tu);
  if (rc) return rc;

  const int Hq = s->num_q_heads, Hkv = s->num_kv_heads, D = s->head_dim, P = s->page_size;
  const int G = Hq / Hkv;
  int64_t T = 0;
  for (int i = 0; i < n; ++i) {
    if (q_len[i] < 0 || ctx_len[i] < 0) return SSA_ERR_LENGTH;
    if ((int64_t)q_len[i] + ctx_len[i] > kMaxLen) return SSA_ERR_LENGTH;
    if (ceil_div((int64_t)q_len[i] + ctx_len[i], P) > s->max_pages_per_req) return SSA_ERR_PAGES;
    T += q_len[i];
    if (T > kMaxLen) return SSA_ERR_LENGTH;
  }

  ssa_plan_info& in = p->info;
  std::memset(&in, 0, sizeof in);
  in.num_reqs = n;
  in.num_tokens = (int32_t)T;

  // requests, routing (Eq. 2), features (Tab. 1)
  p->reqs.resize(n);
  int64_t qs = 0;
  double x7 = 0;
  for (int i = 0; i < n; ++i) {
    const int64_t c = q_len[i], u = ctx_len[i];
    p->reqs[i] = ReqEntry{(int32_t)qs, (int32_t)c, (int32_t)u, (int32_t)ceil_div(c + u, P)};
    qs += c;
    // A request with no new token runs nothing this iteration: it is in no
    // feature and does not decide the scene (the scheduler's batch forming
    // leaves it out the same way).
    if (c == 0) continue;
    in.x[2] += (double)u;
    if (c == 1) {
      in.num_decode_reqs++;
      in.x[3] += 1;
      in.x[4] += (double)u;
    } else {
      in.num_chunk_reqs++;
      in.x[0] += (double)c * (double)(u + c);
      in.x[1] += (double)c * (double)c;
      in.x[5] += (double)c;
      x7 = std::max(x7, (double)c);
    }
    if (c == 1) {
      in.decode_bytes += (double)(u + 1) * Hkv * D * 4.0 + 2.0 * Hq * D * 2.0;
      in.decode_flops += 4.0 * Hq * D * (double)(u + 1);
    } else if (c > 1) {
      in.chunk_bytes += (double)(u + c) * Hkv * D * 4.0 + (double)c * 2.0 * Hq * D * 2.0;
      in.chunk_flops += 4.0 * Hq * D * ((double)c * u + (double)c * (c + 1) / 2.0);
    }
  }
  in.x[6] = x7;
  in.append_bytes = (double)T * Hkv * D * 8.0;
  if (T == 0) in.scene = SSA_SCENE_EMPTY;
  else if (in.num_chunk_reqs == 0) in.scene = SSA_SCENE_PURE_DECODE;
  else if (in.num_decode_reqs == 0) in.scene = SSA_SCENE_PURE_PREFILL;
  else in.scene = SSA_SCENE_MIXED;

  // append segments: runs of new tokens inside one page; those of chunk
  // requests first (a fused launch appends only them in workgroups of their
  // own: a decode item writes its request's single new row itself)
  p->segs.clear();
  p->segs.reserve((size_t)n + (size_t)(T / P) + 1);
  for (int pass = 0; pass < 2; ++pass) {
    for (int i = 0; i < n; ++i) {
      if ((q_len[i] > 1) != (pass == 0)) continue;
      int64_t pos = ctx_len[i], end = (int64_t)ctx_len[i] + q_len[i], row = p->reqs[i].q_start;
      while (pos < end) {
        int64_t m = std::min<int64_t>(P - pos % P, end - pos);
        p->segs.push_back(AppendSeg{i, (int32_t)row, (int32_t)pos, (int32_t)m});
        pos += m;
        row += m;
      }
    }
    if (pass == 0) p->num_chunk_segs = (int32_t)p->segs.size();
  }

  // balancing estimates (seconds): chunk work per CU at the nominal MFMA rate,
  // decode bytes at the nominal HBM rate shared by num_cus CUs
  const int ncu = tu.num_cus;
  double decode_blocks = 0, chunk_time_total = 0;
  for (int i = 0; i < n; ++i) {
    if (q_len[i] == 1) decode_blocks += (double)Hkv * ceil_div((int64_t)ctx_len[i] + 1, kBlockKeys);
    if (q_len[i] > 1)
      chunk_time_total += 4.0 * Hq * D * ((double)q_len[i] * ctx_len[i] + (double)q_len[i] * q_len[i]) /
                          kMfmaRatePerCu;
  }
  const double makespan =
      chunk_time_total / ncu + decode_blocks * kBlockKeys * D * 4.0 / kHbmRate;

  const int dec_split = tu.decode_split_keys > 0 ? tu.decode_split_keys : kDefaultDecodeSplitKeys;

  std::vector<WorkItem> raw;
  std::vector<double> est_t;
  raw.reserve(1024);
  est_t.reserve(1024);
  p->groups.clear();
  p->groups.reserve(256);
  int64_t ws_floats = 0;
  auto add_group = [&](int nsplit, int ncols) {
    MergeGroup g{nsplit, ncols, ws_floats};
    ws_floats += (int64_t)nsplit * rec_floats(ncols, D);
    p->groups.push_back(g);
    return (int32_t)p->groups.size() - 1;
  };

  // Key splits of a chunk tile (automatic): pieces of at most half the
  // estimated makespan, times `mult`, within [1, kMaxChunkSplits] and pieces of
  // at least kMinChunkSplitKeys keys.
  auto auto_nsplit = [&](int kend, int mult) {
    const double t_tile = 4.0 * D * (double)tu.tile_cols * kend / kMfmaRatePerCu;
    int ns = makespan > 0 ? (int)std::ceil(t_tile / (0.5 * makespan)) : 1;
    ns = std::max(1, ns) * mult;
    ns = std::min(ns, std::max(1, kend / kMinChunkSplitKeys));
    return std::max(1, std::min(ns, kMaxChunkSplits));
  };
  // The multiplier: chunk items are long, and when their number is not close
  // to a multiple of the workgroup slots (two per CU) the last round runs part
  // empty (768 equal tiles on 512 slots take two tile times; cut in two, three
  // half times).  The chunk items' greedy longest-first schedule on the slots
  // (decode items left out) is simulated for multipliers 1..3, each extra
  // piece charged kSplitCostKeys keys; a larger multiplier must win by 3%.
  int split_mult = 1;
  if (tu.chunk_split_keys == 0 && makespan > 0) {
    std::vector<double> best_pieces;
    double best = 0.0;
    for (int mult = 1; mult <= 3; ++mult) {
      std::vector<double> pieces;
      bool too_many = false;  // left to the item loop below (which reports it)
      for (int i = 0; i < n && !too_many; ++i) {
        const int c = q_len[i], u = ctx_len[i];
        if (c <= 1) continue;
        const int64_t total_cols = (int64_t)c * G;
        for (int64_t col0 = 0; col0 < total_cols && !too_many; col0 += tu.tile_cols) {
          const int64_t ncols = std::min<int64_t>(tu.tile_cols, total_cols - col0);
          const int kend = u + (int)((col0 + ncols - 1) / G) + 1;
          const int ns = auto_nsplit(kend, mult);
          const int piece = (int)ceil_div(ceil_div(kend, ns), kBlockKeys) * kBlockKeys;
          for (int k0 = 0; k0 < kend; k0 += piece)
            pieces.push_back((double)std::min(piece, kend - k0) + (ns > 1 ? kSplitCostKeys : 0));
          too_many = (int64_t)pieces.size() * Hkv > kMaxItems;
        }
      }
      if (pieces.empty() || too_many) break;
      // beyond four rounds of the slots the last round's loss is small
      const size_t slots = 2 * (size_t)tu.num_cus;
      if (mult == 1 && pieces.size() * Hkv > 4 * slots) break;
      std::sort(pieces.begin(), pieces.end(), std::greater<double>());
      // every kv head has the same pieces, launched next to each other: the
      // schedule of one head's pieces on slots / Hkv slots stands for it
      std::vector<double> slot(std::max<size_t>(1, slots / Hkv), 0.0);
      double end = 0.0;
      for (double t : pieces) {
        std::pop_heap(slot.begin(), slot.end(), std::greater<double>());
        slot.back() += t;
        end = std::max(end, slot.back());
        std::push_heap(slot.begin(), slot.end(), std::greater<double>());
      }
      if (mult == 1 || end < 0.97 * best) {
        if (mult > 1) split_mult = mult;
        best = end;
      }
      // no split can beat a schedule within 3% of the larger of the longest
      // piece and the work per slot
      double total = 0.0;
      for (double t : pieces) total += t;
      if (mult == 1 && end <= 1.03 * std::max(pieces.front(), total / slot.size())) break;
    }
  }

  for (int i = 0; i < n; ++i) {
    const int c = q_len[i], u = ctx_len[i];
    if (c > 1) {
      // column n of the request is (token n / G, head n % G); columns and the
      // item fields that hold them are int32
      const int64_t total_cols64 = (int64_t)c * G;
      if (total_cols64 > INT32_MAX) return SSA_ERR_LENGTH;
      const int total_cols = (int)total_cols64;
      // at least one item per tile and kv head (splits are checked as they are made)
      if ((int64_t)raw.size() + ceil_div(total_cols, tu.tile_cols) * Hkv > kMaxItems)
        return SSA_ERR_LENGTH;
      for (int col0 = 0; col0 < total_cols; col0 += tu.tile_cols) {
        const int ncols = std::min(tu.tile_cols, total_cols - col0);
        const int j_last = (col0 + ncols - 1) / G;
        const int kend = u + j_last + 1;
        for (int h = 0; h < Hkv; ++h) {
          int nsplit = 1;
          if (tu.chunk_split_keys > 0)
            nsplit = (int)ceil_div(kend, tu.chunk_split_keys);
          else if (makespan > 0)
            nsplit = auto_nsplit(kend, split_mult);
          int piece = (int)ceil_div(ceil_div(kend, nsplit), kBlockKeys) * kBlockKeys;
          nsplit = (int)ceil_div(kend, piece);
          const int32_t grp = nsplit > 1 ? add_group(nsplit, ncols) : -1;
          for (int sp = 0; sp < nsplit; ++sp) {
            WorkItem it{};
            it.kind = kItemChunk;
            it.req = i;
            it.kvh = h;
            it.col0 = col0;
            it.ncols = ncols;
            it.key0 = sp * piece;
            it.key1 = std::min(kend, (sp + 1) * piece);
            it.group = grp;
            it.split = sp;
            if ((int64_t)raw.size() >= kMaxItems) return SSA_ERR_LENGTH;
            raw.push_back(it);
            est_t.push_back(4.0 * D * (double)tu.tile_cols * (it.key1 - it.key0) / kMfmaRatePerCu);
          }
        }
      }
    } else if (c == 1) {
      const int keys = u + 1;
      // round(keys / dec_split) equal pieces (at least one), block aligned
      int nsplit = std::max(1, (int)(((int64_t)keys + dec_split / 2) / dec_split));
      const int piece = (int)ceil_div(ceil_div(keys, nsplit), kBlockKeys) * kBlockKeys;
      nsplit = (int)ceil_div(keys, piece);
      if ((int64_t)raw.size() + (int64_t)nsplit * Hkv > kMaxItems) return SSA_ERR_LENGTH;
      for (int h = 0; h < Hkv; ++h) {
        const int32_t grp = nsplit > 1 ? add_group(nsplit, G) : -1;
        for (int sp = 0; sp < nsplit; ++sp) {
          WorkItem it{};
          it.kind = kItemDecode;
          it.req = i;
          it.kvh = h;
          it.col0 = 0;
          it.ncols = G;
          it.key0 = sp * piece;
          it.key1 = std::min(keys, (sp + 1) * piece);
          it.group = grp;
          it.split = sp;
          raw.push_back(it);
          est_t.push_back((double)(it.key1 - it.key0) * D * 4.0 * ncu / kHbmRate);
        }
      }
    }
  }
  std::vector<uint16_t> bucket(raw.size());
  for (size_t k = 0; k < raw.size(); ++k) bucket[k] = (uint16_t)time_bucket(est_t[k]);
  std::vector<uint32_t> seq;
  // Automatic launch order, for batches whose chunk items alone fill both
  // slots of every compute unit (otherwise all chunk items first):
  //  * the decode part comparable to the chunk part (estimated decode time, at
  //    0.7 of the HBM peak, at least 0.85 of the chunk time at half the MFMA
  //    peak): one chunk and one decode item on every unit, the rest
  //    interleaved (measured about 10% faster on such batches);
  //  * a smaller but still sizeable decode part (ratio 0.25 .. 0.85): one
  //    chunk item on every unit beside the decode items, then the other chunk
  //    items, which take the slots the decode items free (measured 5-10%
  //    faster than all chunk items first on the 70B-shaped layer, ratio 0.56,
  //    where interleaving the rest is 20% slower: a long chunk tile that
  //    starts late is the launch's tail).
  //
  // mix_order 5 (for ssa_append_attention_streams): where the two-stream split
  // pays, all chunk items first and the split recorded in the plan; otherwise
  // the automatic order and one launch.
  size_t nchunk = 0;
  double decode_kv_bytes = 0;
  for (const WorkItem& it : raw) {
    if (it.kind == kItemChunk) nchunk++;
    else decode_kv_bytes += (double)(it.key1 - it.key0) * 4.0 * D;
  }
  const double beside_budget = in.chunk_flops / kBesideChunkFlops * kBesideDecodeBytes;
  const bool split = tu.streams == 2 ||
                     (tu.streams == 1 && D == 128 && Hq / Hkv <= 8 &&
                      nchunk >= kBesideMinFill * tu.num_cus && nchunk <= 2 * (size_t)tu.num_cus &&
                      decode_kv_bytes > 0 &&
                      beside_budget >= kBesideMinCover * decode_kv_bytes);
  if (split) tu.mix_order = kOrderChunkFirst;
  if (tu.auto_order && !split) {
    const double t_dec = in.decode_bytes / kHbmRate;
    const double t_chk = in.chunk_flops / (kMfmaRatePerCu * tu.num_cus);
    if (nchunk >= 2 * (size_t)tu.num_cus && t_dec >= kPairedMinRatio * t_chk)
      tu.mix_order = kOrderPaired;
    else if (nchunk >= 2 * (size_t)tu.num_cus && t_dec >= kPairedDecodeFirstRatio * t_chk)
      tu.mix_order = kOrderPairedDecodeFirst;
  }
  order_items(raw, est_t, bucket, tu, Hkv, &seq);
  p->items.resize(raw.size());
  for (size_t k = 0; k < seq.size(); ++k) {
    WorkItem it = raw[seq[k]];
    const ReqEntry& r = p->reqs[it.req];
    it.q_start = r.q_start;
    it.ctx_len = r.ctx_len;
    it.nvalid = r.ctx_len + r.q_len;
    p->items[k] = it;
  }
  for (const WorkItem& it : p->items) {
    if (it.kind == kItemChunk) in.num_chunk_items++;
    else in.num_decode_items++;
  }
  in.num_items = (int32_t)p->items.size();
  in.num_merge_groups = (int32_t)p->groups.size();
  in.num_append_segments = (int32_t)p->segs.size();

  PlanHeader& h = p->hdr;
  std::memset(&h, 0, sizeof h);
  h.magic = kPlanMagic;
  h.version = kPlanVersion;
  h.num_reqs = n;
  h.num_tokens = (int32_t)T;
  h.num_items = in.num_items;
  h.num_chunk_items = in.num_chunk_items;
  h.num_decode_items = in.num_decode_items;
  h.num_groups = in.num_merge_groups;
  h.num_segments = in.num_append_segments;
  h.num_chunk_segments = p->num_chunk_segs;
  h.hq = Hq;
  h.hkv = Hkv;
  h.head_dim = D;
  h.page_size = P;
  h.max_pages_per_req = s->max_pages_per_req;
  h.num_pages = s->num_pages;
  h.chunk_tile_cols = tu.tile_cols;
  h.softmax_scale = s->softmax_scale;
  h.wait_polls = tu.wait_polls;
  h.streams_beside = -1;
  if (split) {
    // the decode items follow the chunk items, longest first
    const int nd = in.num_decode_items;
    int beside = (nd + 1) / 2;
    if (tu.streams == 1) {
      double bytes = 0;
      for (beside = 0; beside < nd; ++beside) {
        const WorkItem& it = p->items[in.num_chunk_items + beside];
        bytes += (double)(it.key1 - it.key0) * 4.0 * D;
        if (bytes > beside_budget) break;
      }
    }
    h.streams_beside = beside;
  }
  // the blob's section offsets are int32 fields: a plan beyond 2 GiB (or a
  // grid beyond 2^31 workgroups) is refused
  int64_t off = sizeof(PlanHeader);
  const int64_t off_reqs = off;
  off += (int64_t)sizeof(ReqEntry) * n;
  const int64_t off_items = off;
  off += (int64_t)sizeof(WorkItem) * (int64_t)p->items.size();
  const int64_t off_groups = off;
  off += (int64_t)sizeof(MergeGroup) * (int64_t)p->groups.size();
  const int64_t off_segments = off;
  off += (int64_t)sizeof(AppendSeg) * (int64_t)p->segs.size();
  if (off > INT32_MAX || (int64_t)p->items.size() + (int64_t)p->segs.size() > INT32_MAX)
    return SSA_ERR_LENGTH;
  h.off_reqs = (int32_t)off_reqs;
  h.off_items = (int32_t)off_items;
  h.off_groups = (int32_t)off_groups;
  h.off_segments = (int32_t)off_segments;
  h.plan_bytes = off;
  const int64_t tickets = ceil_div(((int64_t)kLaunchCounters + p->groups.size()) * 4, 256) * 256;
  h.ws_partials_off = tickets;
  h.ws_bytes = tickets + ws_floats * 4;
  in.ws_zero_bytes = tickets;

  uint64_t hv = 1469598103934665603ull;
  int32_t fields[8] = {Hq, Hkv, D, P, s->num_pages, s->max_pages_per_req, n, 0};
  hv = fnv1a(hv, fields, sizeof fields);
  hv = fnv1a(hv, &s->softmax_scale, sizeof(float));
  hv = fnv1a(hv, &tu, sizeof tu);
  if (n > 0) {
    hv = fnv1a(hv, q_len, sizeof(int32_t) * n);
    hv = fnv1a(hv, ctx_len, sizeof(int32_t) * n);
  }
  h.hash = hv;
  return SSA_OK;
}

}  // namespace

// Check that plan_host is a plan built for this shape; used by the launchers.
int check_plan(const ssa_shape* s, const void* plan_host, const PlanHeader** out) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (!plan_host) return SSA_ERR_NULL;
  const PlanHeader* h = static_cast<const PlanHeader*>(plan_host);
  if (h->magic != kPlanMagic || h->version != kPlanVersion || h->hq != s->num_q_heads ||
      h->hkv != s->num_kv_heads || h->head_dim != s->head_dim || h->page_size != s->page_size ||
      h->num_pages != s->num_pages || h->max_pages_per_req != s->max_pages_per_req ||
      std::memcmp(&h->softmax_scale, &s->softmax_scale, sizeof(float)) != 0)
    return SSA_ERR_PLAN_MISMATCH;
  *out = h;
  return SSA_OK;
}

}  // namespace ssa

extern "C" {

const char* ssa_status_string(int code) {
  switch (code) {
    case SSA_OK: return "ok";
    case SSA_ERR_NULL: return "a required pointer is NULL";
    case SSA_ERR_SHAPE: return "invalid head counts (Hq, Hkv > 0, Hq % Hkv == 0, Hq/Hkv <= 16)";
    case SSA_ERR_HEAD_DIM: return "head_dim must be 64 or 128";
    case SSA_ERR_PAGE_SIZE: return "page_size must be 16";
    case SSA_ERR_LENGTH: return "negative or too large q_len / ctx_len";
    case SSA_ERR_PAGES: return "a request needs more pages than max_pages_per_req, or no pages";
    case SSA_ERR_PLAN_SIZE: return "plan buffer too small";
    case SSA_ERR_WORKSPACE: return "workspace missing or too small";
    case SSA_ERR_PLAN_MISMATCH: return "plan does not belong to this shape";
    case SSA_ERR_HIP: return "HIP launch failed";
    case SSA_ERR_SCALE: return "softmax_scale is negative or not finite";
    case SSA_ERR_TUNING: return "tuning field out of range";
    case SSA_ERR_ARG: return "an argument out of range";
    default: return "unknown";
  }
}

int ssa_plan_size(const ssa_shape* shape, const int32_t* q_len_host, const int32_t* ctx_len_host,
                  int32_t num_reqs, const ssa_tuning* tuning, size_t* plan_bytes,
                  size_t* workspace_bytes) {
  if (!plan_bytes || !workspace_bytes) return SSA_ERR_NULL;
  try {
    ssa::Plan p;
    int rc = ssa::build(shape, q_len_host, ctx_len_host, num_reqs, tuning, &p);
    if (rc) return rc;
    *plan_bytes = (size_t)p.hdr.plan_bytes;
    *workspace_bytes = (size_t)p.hdr.ws_bytes;
    return SSA_OK;
  } catch (const std::bad_alloc&) {
    return SSA_ERR_LENGTH;
  }
}

int ssa_check_block_table(const ssa_shape* shape, const void* plan_host,
                          const int32_t* block_table_host) {
  const ssa::PlanHeader* h = nullptr;
  int rc = ssa::check_plan(shape, plan_host, &h);
  if (rc) return rc;
  if (h->num_reqs > 0 && !block_table_host) return SSA_ERR_NULL;
  const ssa::ReqEntry* reqs = reinterpret_cast<const ssa::ReqEntry*>(
      static_cast<const char*>(plan_host) + h->off_reqs);
  for (int32_t i = 0; i < h->num_reqs; ++i) {
    if (reqs[i].q_len == 0) continue;  // no work item or append segment reads this row
    const int32_t* row = block_table_host + (size_t)i * h->max_pages_per_req;
    for (int32_t k = 0; k < reqs[i].n_pages; ++k)
      if (row[k] < 0 || row[k] >= h->num_pages) return SSA_ERR_PAGES;
  }
  return SSA_OK;
}

int ssa_plan(const ssa_shape* shape, const int32_t* q_len_host, const int32_t* ctx_len_host,
             int32_t num_reqs, const ssa_tuning* tuning, void* plan_host, size_t plan_bytes,
             ssa_plan_info* info) {
  if (!plan_host) return SSA_ERR_NULL;
  try {
    ssa::Plan p;
    int rc = ssa::build(shape, q_len_host, ctx_len_host, num_reqs, tuning, &p);
    if (rc) return rc;
    if (plan_bytes < (size_t)p.hdr.plan_bytes) return SSA_ERR_PLAN_SIZE;
    char* b = static_cast<char*>(plan_host);
    std::memcpy(b, &p.hdr, sizeof p.hdr);
    if (!p.reqs.empty())
      std::memcpy(b + p.hdr.off_reqs, p.reqs.data(), sizeof(ssa::ReqEntry) * p.reqs.size());
    if (!p.items.empty())
      std::memcpy(b + p.hdr.off_items, p.items.data(), sizeof(ssa::WorkItem) * p.items.size());
    if (!p.groups.empty())
      std::memcpy(b + p.hdr.off_groups, p.groups.data(), sizeof(ssa::MergeGroup) * p.groups.size());
    if (!p.segs.empty())
      std::memcpy(b + p.hdr.off_segments, p.segs.data(), sizeof(ssa::AppendSeg) * p.segs.size());
    if (info) *info = p.info;
    return SSA_OK;
  } catch (const std::bad_alloc&) {
    return SSA_ERR_LENGTH;
  }
}

}  // extern "C"
