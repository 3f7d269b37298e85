/*
 * ssa.h - mixed chunked-prefill + decode attention over a paged KV cache, for
 * AMD Instinct MI355X (gfx950).
 *
 * One serving iteration executes a batch B = {(c_i, u_i)}: request i computes
 * c_i new tokens on top of u_i tokens already in its KV cache (SlidingServe,
 * Sec. 3.2).  Requests with c_i <= 1 form the decode set, the others the
 * prefill (chunk) set (Sec. 3.2, Eq. 2); a batch is pure decode, pure prefill
 * or mixed (Eq. 3).  A chunk's new token j, at absolute position u_i + j,
 * attends causally to keys 0 .. u_i + j of its own request (chunked prefill,
 * Sec. 1 and Sec. 2.1); a decode token is the case c_i = 1, j = 0.  Query head
 * h reads kv head floor(h / G), G = Hq / Hkv.
 *
 * Call sequence for one iteration (all on one stream):
 *   ssa_plan_size   -> sizes of the plan blob and the workspace      (host)
 *   ssa_plan        -> fills the plan blob from (q_len, ctx_len)      (host)
 *   ssa_kv_append   -> writes the new K/V rows into their pages      (1 kernel)
 *   ssa_mixed_attention -> outputs of every new token                (1 kernel)
 *
 * The kernels read the plan blob through plan_dev: either a device copy of
 * it, or the host buffer itself when that buffer is pinned, device-mapped host
 * memory (hipHostMalloc); the blob is small and each workgroup reads one record
 * of it.  Either way the caller must not change those bytes until the launches
 * that use them have completed (alternate two buffers between iterations).
 *
 * Conventions shared by every call:
 *   - Every function returns SSA_OK (0) or a negative SSA_ERR_* code.  All
 *     arguments are validated before any HIP call; on an error nothing is
 *     written and nothing is launched.  No C++ exception crosses this ABI and
 *     nothing is printed.
 *   - The library allocates no memory and keeps no state between calls, with
 *     two exceptions: the per-GPU scratch of ssa_append_attention_static, and
 *     the fork/join events of ssa_append_attention_streams (two per host
 *     thread and device, created on first use).
 *   - "bf16" arguments are bfloat16 bit patterns (uint16_t); they are device
 *     pointers unless the name ends in _host.
 *   - stream is a hipStream_t passed as void* (NULL = the null stream).
 *
 * Memory layouts (row-major, dense, no padding):
 *   q, out         [T, Hq, D]       T = sum of q_len; rows grouped by request,
 *                                    requests in the order given to ssa_plan
 *   k_new, v_new   [T, Hkv, D]
 *   k_cache        [num_pages, Hkv, P, D]   key page: P slots of D values
 *   v_cache        [num_pages, Hkv, D, P]   value page: D rows of P slots
 *   block_table    int32 [num_reqs, max_pages_per_req]; token position t of
 *                  request i lives in page block_table[i][t / P], slot t % P.
 *                  Only the first ceil((u_i + c_i) / P) entries of a row are
 *                  read; their values must lie in [0, num_pages) (the caller's
 *                  responsibility: the library cannot check device memory).
 *   P (page_size) is 16; D (head_dim) is 64 or 128; 1 <= Hq / Hkv <= 16.
 */
#ifndef SSA_H
#define SSA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SSA_PAGE_SIZE 16

enum {
  SSA_OK = 0,
  SSA_ERR_NULL = -1,          /* a required pointer is NULL */
  SSA_ERR_SHAPE = -2,         /* Hq, Hkv not positive, Hq % Hkv != 0, or Hq/Hkv > 16 */
  SSA_ERR_HEAD_DIM = -3,      /* head_dim not 64 or 128 */
  SSA_ERR_PAGE_SIZE = -4,     /* page_size not 16 */
  SSA_ERR_LENGTH = -5,        /* negative q_len / ctx_len, or a length sum beyond 2^30 */
  SSA_ERR_PAGES = -6,         /* ceil((u+c)/P) > max_pages_per_req, or num_pages < 1 */
  SSA_ERR_PLAN_SIZE = -7,     /* the plan buffer is smaller than ssa_plan_size says */
  SSA_ERR_WORKSPACE = -8,     /* workspace NULL or smaller than the plan requires */
  SSA_ERR_PLAN_MISMATCH = -9, /* plan_host is not a plan of this shape (magic/hash) */
  SSA_ERR_HIP = -10,          /* a HIP launch failed */
  SSA_ERR_SCALE = -11,        /* softmax_scale negative or not finite */
  SSA_ERR_TUNING = -12,       /* a tuning field out of range */
  SSA_ERR_ARG = -13           /* another argument out of range (the other headers) */
};

/* Scene of a batch (Sec. 3.2, Eq. 3).  A batch with no new token is EMPTY. */
enum { SSA_SCENE_EMPTY = 0, SSA_SCENE_PURE_DECODE = 1, SSA_SCENE_PURE_PREFILL = 2,
       SSA_SCENE_MIXED = 3 };

typedef struct ssa_shape {
  int32_t num_q_heads;       /* Hq */
  int32_t num_kv_heads;      /* Hkv */
  int32_t head_dim;          /* D: 64 or 128 */
  int32_t page_size;         /* P: 16 */
  int32_t num_pages;         /* pages in each pool */
  int32_t max_pages_per_req; /* row stride of block_table */
  float softmax_scale;       /* >= 0; multiplies <q, k> before the softmax (1/sqrt(D) usually) */
} ssa_shape;

/*
 * Optional planner knobs (pass NULL to ssa_plan_size / ssa_plan for the
 * defaults).  Zero in a field selects its default.  Results do not depend on
 * them beyond floating-point summation order.
 *   chunk_tile_cols  columns (token x q-head-in-group pairs) per chunk work
 *                    item: 32, 64 or 128 (default 128)
 *   chunk_split_keys if > 0, a chunk tile's key range is cut into pieces of this
 *                    many keys (multiple of 32); default: chosen by the planner
 *   decode_split_keys a decode key range of k keys is cut into
 *                    max(1, round(k / decode_split_keys)) equal pieces, each a
 *                    multiple of 32 keys (multiple of 32; default 3072)
 *   num_cus          compute units the planner balances for (default 256)
 *   num_xcds         if > 1, die-aware placement: workgroups are taken to be
 *                    dealt to num_xcds dies round-robin (workgroup b on die
 *                    b mod num_xcds), and work items that read the same K/V
 *                    (one request and kv head of a chunk) go to one die
 *                    (default 1: off; on MI355X it measured no faster)
 *   mix_order        0 = chosen by the planner (default): when the chunk items
 *                    number at least 2 * num_cus, 3 if the decode part's
 *                    estimated time (its bytes at 0.7 of the HBM peak) is at
 *                    least 0.85 of the chunk part's (its flops at half the MFMA
 *                    peak), 4 if it is at least 0.25 of it; else 1;
 *                    1 = all chunk items (longest first) before the decode
 *                    items, 2 = the two kinds interleaved, 3 = paired:
 *                    the first num_cus chunk items, then decode items for the
 *                    second slot of every compute unit, then the rest
 *                    interleaved (workgroups 0 .. num_cus-1 are taken to land on
 *                    distinct units, the next num_cus on their second slots),
 *                    4 = as 3, then the other decode items, then the other
 *                    chunk items,
 *                    5 = for ssa_append_attention_streams: where the
 *                    two-stream split pays (head_dim 128, Hq/Hkv <= 8,
 *                    1.5 * num_cus to 2 * num_cus chunk items (one round of
 *                    two per compute unit), and at least 0.9 of the
 *                    decode rows' K/V bytes fit beside the chunk rows: bytes at
 *                    2.5 TB/s over the chunk rows' time at 0.95 PFLOP/s, the
 *                    rates measured on MI355X with the two side by side), all
 *                    chunk items first and the split recorded in the plan;
 *                    elsewhere as 0, and the call runs as one launch,
 *                    6 = the split forced (for tests): chunk items first, half
 *                    of the decode items beside the chunk rows, half after
 *   append_wait_polls  ssa_append_attention: polls (about 0.25 us each) before a
 *                    chunk item's wait for the rows appended in the same launch
 *                    gives up and sets SSA_STATUS_WAIT_TIMEOUT (default 2^21,
 *                    about half a second; a test sets a small value to force
 *                    the time-out from the host)
 */
typedef struct ssa_tuning {
  int32_t chunk_tile_cols;
  int32_t chunk_split_keys;
  int32_t decode_split_keys;
  int32_t num_cus;
  int32_t num_xcds;
  int32_t mix_order;
  int32_t append_wait_polls;
} ssa_tuning;

/*
 * Workspace status word.  The int32 at byte SSA_WS_STATUS_OFFSET of the
 * workspace collects error bits that the kernels of ssa_mixed_attention and
 * ssa_append_attention set (device-scope atomic OR) and never clear: the
 * launch still finishes, every workgroup exits, but the outputs it names may
 * be wrong.  Zero it with the rest of the workspace before first use; read it
 * (after the launch has completed) to check a launch, and zero it again after
 * a report.
 *   SSA_STATUS_WAIT_TIMEOUT   a chunk item of ssa_append_attention gave up
 *                             waiting for the workgroups that append this
 *                             launch's rows (the launch ran on, possibly with
 *                             stale key rows): the in-order dispatch that the
 *                             fused launch relies on did not hold, or
 *                             append_wait_polls was too small
 *   SSA_STATUS_PLAN_MISMATCH  the plan bytes a kernel read at plan_dev do not
 *                             carry the magic number and hash of plan_host (the
 *                             device copy is stale or was overwritten): the
 *                             kernel wrote nothing
 */
#define SSA_WS_STATUS_OFFSET 8
#define SSA_STATUS_WAIT_TIMEOUT 1
#define SSA_STATUS_PLAN_MISMATCH 2

/*
 * What ssa_plan derived from the batch.  Byte and flop counts are the
 * algorithmic work (what the method must move or compute), not the work the
 * kernels actually do.
 *   decode_bytes  K/V bytes of the decode rows, sum over D of (u+1)*Hkv*D*2*2,
 *                 plus their q and out rows (2*Hq*D*2 per row)
 *   chunk_bytes   K/V bytes of the chunk requests, (u+c)*Hkv*D*2*2 each, plus
 *                 their q and out rows
 *   chunk_flops   4*Hq*D*(c*u + c*(c+1)/2) summed over the prefill set
 *   decode_flops  4*Hq*D*(u+1) summed over the decode set
 *   append_bytes  bytes kv_append reads plus writes: T*Hkv*D*2*2*2
 *   x[0..6]       the paper's batch features x1..x7 (Tab. 1)
 * A request with c_i = 0 has no new token and runs nothing: it counts in
 * num_reqs only (not in num_decode_reqs, the features or the scene), as the
 * scheduler's batch forming leaves it out (ssa_chunker.h).
 */
typedef struct ssa_plan_info {
  int32_t num_reqs, num_tokens, num_decode_reqs, num_chunk_reqs;
  int32_t num_items, num_chunk_items, num_decode_items, num_merge_groups;
  int32_t num_append_segments, scene;
  double decode_bytes, chunk_bytes, chunk_flops, decode_flops, append_bytes;
  double x[7];
  int64_t ws_zero_bytes;  /* leading workspace bytes that must be zero at rest
                             (counters, status word, merge tickets); the rest
                             holds split records */
} ssa_plan_info;

/* Static description of an error code ("ok" for SSA_OK, "unknown" otherwise). */
const char* ssa_status_string(int code);

/*
 * Sizes of the plan blob and of the workspace for this batch.
 *   q_len_host[i] = c_i, ctx_len_host[i] = u_i (host arrays of num_reqs).
 *   num_reqs may be 0.  tuning may be NULL.
 * Errors: NULL, SHAPE, HEAD_DIM, PAGE_SIZE, SCALE, LENGTH, PAGES, TUNING.
 */
int ssa_plan_size(const ssa_shape* shape, const int32_t* q_len_host, const int32_t* ctx_len_host,
                  int32_t num_reqs, const ssa_tuning* tuning, size_t* plan_bytes,
                  size_t* workspace_bytes);

/*
 * Build the plan (pure host code, no HIP call): request starts, the decode /
 * chunk routing of Eq. 2, the work items of the attention launch, the merge
 * groups of split work items, the append segments, and info (may be NULL).
 * plan_host must hold plan_bytes >= ssa_plan_size's value; the blob is
 * position-independent and is used as is on the device after a byte copy.
 * Errors: those of ssa_plan_size, and PLAN_SIZE.
 */
int ssa_plan(const ssa_shape* shape, const int32_t* q_len_host, const int32_t* ctx_len_host,
             int32_t num_reqs, const ssa_tuning* tuning, void* plan_host, size_t plan_bytes,
             ssa_plan_info* info);

/*
 * Optional host-side check of a block table before a launch (pure host code).
 * The kernels read, for request i, entries block_table[i][0 .. n_i - 1] with
 * n_i = ceil((u_i + c_i) / P) and take each as a page index without checking
 * it; an index outside [0, num_pages) would make them read or write outside
 * the pools.  This call checks exactly those entries of block_table_host
 * (int32, [num_reqs, max_pages_per_req], a host copy of the table the launch
 * will use) against the plan's num_pages.  Other entries are not read.
 * Errors: NULL, the shape errors, PLAN_MISMATCH, PAGES (an entry out of range).
 */
int ssa_check_block_table(const ssa_shape* shape, const void* plan_host,
                          const int32_t* block_table_host);

/*
 * Layout conversion of a value pool, for callers that keep value pages in the
 * key pool's token-major layout.  It is not an operation of the paper: the
 * paged cache that every batch attends over (Sec. 3.2) only fixes which page
 * and slot hold a token, and these kernels read value pages dim-major.
 *   to_dim_major = 1: src [num_pages, Hkv, P, D] (P slots of D values) ->
 *                     dst [num_pages, Hkv, D, P] (D rows of P slots, v_cache
 *                     as the calls above take it);
 *   to_dim_major = 0: the inverse, dst [num_pages, Hkv, P, D].
 *   Uses num_kv_heads, head_dim, page_size and num_pages of the shape (the
 *   other fields are not read).  src and dst are device pointers, 16-byte
 *   aligned, to whole pools that must not overlap (no in-place conversion);
 *   the bytes are moved unchanged.  One kernel launch on stream.
 * Errors: NULL; SHAPE (num_kv_heads < 1); HEAD_DIM; PAGE_SIZE; PAGES
 * (num_pages < 1, or a grid beyond 2^31 workgroups); ARG (to_dim_major not 0 or
 * 1, a misaligned pointer, or overlapping pools); HIP.
 */
int ssa_v_pool_convert(const ssa_shape* shape, const uint16_t* src, uint16_t* dst,
                       int32_t to_dim_major, void* stream);

/*
 * KV append (one kernel): new token j of request i, at position t = u_i + j,
 * is copied bit for bit from k_new/v_new row (q_start_i + j) into page
 * block_table[i][t / P], slot t % P, of k_cache / v_cache.  No other pool
 * byte is written.  plan_host is the plan blob on the host (read for the
 * launch size and checked against shape); plan_dev is the same bytes where the
 * device can read them (a device copy, or plan_host itself if it is pinned
 * device-mapped host memory).
 * Errors: NULL, the shape errors, PLAN_MISMATCH, HIP.
 */
int ssa_kv_append(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                  const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache,
                  uint16_t* v_cache, const int32_t* block_table, void* stream);

/*
 * Mixed attention (exactly one kernel launch): out[q_start_i + j, h, :] =
 * softmax_t(scale * <q, k_t>) weighted sum of v_t over keys t = 0 .. u_i + j of
 * request i (kv head floor(h / G)), for every new token and q head, in bf16
 * (fp32 accumulation).  Reads the chunk's own keys from the pools, so
 * ssa_kv_append of the same plan must have run before it on the stream.
 * workspace: device memory of at least the plan's workspace size (never less
 * than 256 bytes).  Its first ws_zero_bytes bytes (ssa_plan_info) must be zero
 * when a call starts: zero-fill them before the first call, and again when the
 * workspace passes to a plan with a larger ws_zero_bytes (the bytes past a
 * plan's ws_zero_bytes hold its split records).  Each call leaves its counters
 * and tickets at zero again, and reports errors in the status word
 * (SSA_WS_STATUS_OFFSET).  Calls that share a workspace must not overlap in
 * time.
 * Errors: NULL, the shape errors, PLAN_MISMATCH, WORKSPACE, HIP.
 */
int ssa_mixed_attention(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                        const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                        const int32_t* block_table, uint16_t* out, void* workspace,
                        size_t workspace_bytes, void* stream);

/*
 * The two launches above with kernel timing: identical work and errors, plus
 * two optional HIP events (hipEvent_t as void*, created by the caller with
 * timing enabled; NULL = not recorded).  start_event takes the time the kernel
 * starts and stop_event the time it ends, stamped from the kernel's own
 * dispatch (hipExtLaunchKernel), so timing adds no packet to the stream and no
 * gap between the kernel and its neighbours.  Per-iteration kernel latencies
 * are what the paper's batch latency predictor is fitted on (Sec. 3.2, Eq. 5).
 * When the batch has no work (no launch), the events are not recorded.
 */
int ssa_kv_append_timed(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                        const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_cache,
                        uint16_t* v_cache, const int32_t* block_table, void* stream,
                        void* start_event, void* stop_event);

int ssa_mixed_attention_timed(const ssa_shape* shape, const void* plan_host,
                              const void* plan_dev, const uint16_t* q, const uint16_t* k_cache,
                              const uint16_t* v_cache, const int32_t* block_table, uint16_t* out,
                              void* workspace, size_t workspace_bytes, void* stream,
                              void* start_event, void* stop_event);

/*
 * ssa_kv_append followed by ssa_mixed_attention of the same plan, in ONE
 * kernel launch (one iteration, Sec. 3.2: the new K/V rows of B = {(c_i, u_i)}
 * enter their pages and every new token's output is computed).  Results are
 * the same as the two calls in sequence (the same pool image, bit for bit; the
 * same outputs, bit for bit).  Saves the second launch and the gap between two
 * dependent kernels.
 *   Arguments: as ssa_kv_append and ssa_mixed_attention; the workspace is
 *   required (its first words are the launch's counters, zero at rest and
 *   zero again after each call); events as in the _timed calls (NULL: none).
 *   Inside the launch, the rows of chunk requests (c_i > 1) are appended by
 *   workgroups of their own that come first in the grid and never wait; a
 *   chunk work item waits for them (device-scope counter, once) before it
 *   copies the first key block holding rows appended by this launch, and
 *   copies the blocks from there on at device scope.  This relies on
 *   workgroups being dispatched in index order, as the hardware does for one
 *   launch.  A decode request's single new row is read by its decode item
 *   from k_new / v_new and appended by that item itself (no other workgroup
 *   reads that slot), so decode work never waits.
 * Errors: those of ssa_kv_append and ssa_mixed_attention.
 */
int ssa_append_attention(const ssa_shape* shape, const void* plan_host, const void* plan_dev,
                         const uint16_t* q, const uint16_t* k_new, const uint16_t* v_new,
                         uint16_t* k_cache, uint16_t* v_cache, const int32_t* block_table,
                         uint16_t* out, void* workspace, size_t workspace_bytes, void* stream,
                         void* start_event, void* stop_event);

/*
 * ssa_append_attention without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The launch's counters, status word,
 * merge tickets and split records live in a scratch array of the library,
 * 32 MiB per GPU, held by each GPU the library runs on until the process ends;
 * the call allocates nothing.  On a device's first call the library takes the
 * array's device address (hipGetSymbolAddress); whenever a call's plan needs
 * a larger zeroed prefix (ssa_plan_info.ws_zero_bytes) than the previous
 * call's left, a small fill kernel on the same stream clears it first.
 *   Arguments, results and errors: those of ssa_append_attention without
 *   workspace / workspace_bytes; SSA_ERR_WORKSPACE if the plan needs more than
 *   the 32 MiB scratch (its workspace size from ssa_plan_size).  The status
 *   word is the scratch's own and is not visible to the caller.
 *   Every call on one GPU shares that GPU's scratch: calls that overlap in
 *   time on one GPU (two streams, two threads) race and must not be issued.
 */
int ssa_append_attention_static(const ssa_shape* shape, const void* plan_host,
                                const void* plan_dev, const uint16_t* q, const uint16_t* k_new,
                                const uint16_t* v_new, uint16_t* k_cache, uint16_t* v_cache,
                                const int32_t* block_table, uint16_t* out, void* stream,
                                void* start_event, void* stop_event);

/*
 * One iteration (Sec. 3.2) with the chunked-prefill rows (Sec. 2.1; Tab. 1
 * x1/x2) and the decode rows (Tab. 1 x4/x5) in launches of their own that run
 * at the same time on two streams, where the plan asks for it (tuning
 * mix_order 5 or 6); otherwise exactly ssa_append_attention on `stream`.  Same
 * inputs, outputs, pool image and workspace rules as ssa_append_attention.
 *   Why: a CU holds two chunk workgroups, and the decode kernel of this call is
 *   built to fit in the registers and LDS they leave (80 VGPRs per lane, 8 KB),
 *   so its workgroups stream the decode rows' K/V beside the chunk tiles
 *   instead of taking their slots, as the decode items of one launch do.  It
 *   pays where the chunk tiles fill both slots of every CU and the decode rows
 *   fit in their time (mix_order 5 decides; on the 70B-shaped batch the pair
 *   takes about 0.9 of the one launch).
 *   Split: the first streams_beside decode items of the plan (ssa_plan
 *   records how many) run on `decode_stream`, in launches of at most one
 *   workgroup per CU, beside the chunk rows' launch on `stream`; the other
 *   decode items run in one launch on `stream` after the chunk rows.  The chunk
 *   rows' outputs and the pool image are bit for bit those of
 *   ssa_append_attention with the same plan; the decode rows' outputs agree
 *   to within fp32 summation order (their kernel splits the head dim over its
 *   waves).
 *   stream, decode_stream: hipStream_t as void* (NULL: the null stream).  The
 *   call records an event on `stream` that `decode_stream` waits for, and
 *   makes `stream` wait for an event recorded on `decode_stream` after its
 *   launches: work queued on `stream` after the call sees the whole iteration.
 *   The events belong to the library, one pair per host thread and device.  The
 *   two streams should map to different hardware queues (on ROCm, streams are
 *   dealt round-robin to GPU_MAX_HW_QUEUES queues): on one queue the launches
 *   run one after the other, with the same results.
 *   One launch on `stream` (ssa_append_attention) instead: plans without the
 *   split, shapes the decode kernel does not take (head_dim 64, Hq/Hkv > 8),
 *   batches without decode rows.  A split plan without chunk rows runs its
 *   decode kernel on `stream` alone.
 *   start_event, stop_event: optional timing events (as in the _timed calls)
 *   stamped with the start and end of the chunk rows' launch, the iteration's
 *   longest kernel (of the one launch where the call runs as one, of the decode
 *   launch where a split plan has no chunk rows).  They do not mark the end of
 *   the decode launch: to time the whole iteration, or to know when its plan
 *   buffer may be reused, record an event on `stream` after the call.
 * Errors: those of ssa_append_attention.
 */
int ssa_append_attention_streams(const ssa_shape* shape, const void* plan_host,
                                 const void* plan_dev, const uint16_t* q, const uint16_t* k_new,
                                 const uint16_t* v_new, uint16_t* k_cache, uint16_t* v_cache,
                                 const int32_t* block_table, uint16_t* out, void* workspace,
                                 size_t workspace_bytes, void* stream, void* decode_stream,
                                 void* start_event, void* stop_event);

#ifdef __cplusplus
}
#endif

#endif /* SSA_H */
