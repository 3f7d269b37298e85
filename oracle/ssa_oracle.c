/*
 * CPU oracle for mixed chunked-prefill + decode attention over a paged KV cache.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or calls
 * this file; only the tests, the smoke check and the benchmark's CPU-baseline
 * leg do.  It shares no source with the HIP library.
 *
 * What it computes is the plain definition of the result, not the method that
 * reaches it faster:
 *
 *  - The iteration's batch is B = {(c_i, u_i)} (Sec. 3.2): request i computes
 *    c_i new tokens this iteration on top of u_i tokens already cached.
 *  - Chunked prefill (Sec. 1, Sec. 2.1): a chunk's new token j sits at absolute
 *    position u_i + j and attends causally to every key at positions
 *    0 .. u_i + j of its own request (the cached prefix, the earlier tokens of
 *    its own chunk, and itself).  A decode row (c_i = 1, Eq. 2) is the special
 *    case j = 0: it sees u_i + 1 keys.  c_i = 0 contributes no rows.
 *  - Grouped-query attention: q head h reads kv head floor(h / G), G = Hq/Hkv.
 *  - Softmax over scale * <q, k_t>, then the weighted sum of v_t.
 *
 * Arithmetic: every bf16 input is widened exactly to double; dot products,
 * maximum, exponentials, sums and the final division are in double; the
 * softmax is the two-pass textbook form (max, then sum of exp, then weighted
 * sum) - deliberately not the online form the kernels use.  The scale is the
 * caller's fp32 value widened to double.
 *
 * Layouts (the library's boundary contract):
 *   q        [T, Hq, D]          rows grouped by request, requests in order
 *   k_new    [T, Hkv, D], v_new [T, Hkv, D]
 *   k_cache  [num_pages, Hkv, P, D]   (key page: slot-major)
 *   v_cache  [num_pages, Hkv, D, P]   (value page: dim-major)
 *   block_table [num_reqs, max_pages_per_req]; position t of request i lives in
 *   page block_table[i][t / P], slot t % P.
 *   out      [T, Hq, D] (double)
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double bf16_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Address of element (page, head, slot, dim) in the key pool. */
static size_t k_index(int64_t page, int h, int slot, int d, int Hkv, int P, int D) {
  return (((size_t)page * Hkv + h) * P + slot) * D + d;
}

/* Address of element (page, head, dim, slot) in the value pool. */
static size_t v_index(int64_t page, int h, int d, int slot, int Hkv, int P, int D) {
  return (((size_t)page * Hkv + h) * D + d) * P + slot;
}

static void prefix_sum(const int32_t* q_len, int n, int64_t* q_start) {
  int64_t s = 0;
  for (int i = 0; i < n; ++i) {
    q_start[i] = s;
    s += q_len[i];
  }
}

/*
 * KV append: new token j of request i (position u_i + j) is copied, bit for
 * bit, into its page slot.  No other pool element changes.
 */
void oracle_kv_append(int Hkv, int D, int P, int num_reqs, const int32_t* q_len,
                      const int32_t* ctx_len, const int32_t* block_table,
                      int max_pages_per_req, const uint16_t* k_new, const uint16_t* v_new,
                      uint16_t* k_cache, uint16_t* v_cache) {
  int64_t* q_start = (int64_t*)malloc(sizeof(int64_t) * (num_reqs > 0 ? num_reqs : 1));
  prefix_sum(q_len, num_reqs, q_start);
  for (int i = 0; i < num_reqs; ++i) {
    for (int j = 0; j < q_len[i]; ++j) {
      int64_t t = (int64_t)ctx_len[i] + j;
      int64_t page = block_table[(size_t)i * max_pages_per_req + t / P];
      int slot = (int)(t % P);
      int64_t row = q_start[i] + j;
      for (int h = 0; h < Hkv; ++h) {
        for (int d = 0; d < D; ++d) {
          size_t src = ((size_t)row * Hkv + h) * D + d;
          k_cache[k_index(page, h, slot, d, Hkv, P, D)] = k_new[src];
          v_cache[v_index(page, h, d, slot, Hkv, P, D)] = v_new[src];
        }
      }
    }
  }
  free(q_start);
}

/*
 * One output row: query (request i, new token j, q head h) against keys
 * 0 .. u_i + j of request i.  scores has room for u_i + j + 1 doubles.
 */
static void attend_row(int i, int j, int h, int Hq, int Hkv, int D, int P, double scale,
                       const int32_t* ctx_len, const int32_t* block_table, int max_pages_per_req,
                       int64_t row, const uint16_t* q, const uint16_t* k_cache,
                       const uint16_t* v_cache, double* scores, double* o) {
  int G = Hq / Hkv;
  int g = h / G;
  int64_t pos = (int64_t)ctx_len[i] + j;
  const uint16_t* qrow = q + ((size_t)row * Hq + h) * D;
  const int32_t* bt = block_table + (size_t)i * max_pages_per_req;

  /* pass 1: logits and their maximum */
  double m = -INFINITY;
  for (int64_t t = 0; t <= pos; ++t) {
    int64_t page = bt[t / P];
    int slot = (int)(t % P);
    double dot = 0.0;
    for (int d = 0; d < D; ++d)
      dot += bf16_to_double(qrow[d]) * bf16_to_double(k_cache[k_index(page, g, slot, d, Hkv, P, D)]);
    scores[t] = scale * dot;
    if (scores[t] > m) m = scores[t];
  }
  /* pass 2: normaliser */
  double sum = 0.0;
  for (int64_t t = 0; t <= pos; ++t) {
    scores[t] = exp(scores[t] - m);
    sum += scores[t];
  }
  /* pass 3: weighted sum of values */
  for (int d = 0; d < D; ++d) o[d] = 0.0;
  for (int64_t t = 0; t <= pos; ++t) {
    int64_t page = bt[t / P];
    int slot = (int)(t % P);
    for (int d = 0; d < D; ++d)
      o[d] += scores[t] * bf16_to_double(v_cache[v_index(page, g, d, slot, Hkv, P, D)]);
  }
  for (int d = 0; d < D; ++d) o[d] /= sum;
}

/*
 * Full attention for every new token row and every q head.
 * num_threads <= 0 keeps the OpenMP default.  Returns the thread count used.
 */
int oracle_attention(int Hq, int Hkv, int D, int P, float scale, int num_reqs,
                     const int32_t* q_len, const int32_t* ctx_len, const int32_t* block_table,
                     int max_pages_per_req, const uint16_t* q, const uint16_t* k_cache,
                     const uint16_t* v_cache, double* out, int num_threads) {
  int64_t* q_start = (int64_t*)malloc(sizeof(int64_t) * (num_reqs > 0 ? num_reqs : 1));
  prefix_sum(q_len, num_reqs, q_start);
  int max_keys = 1;
  for (int i = 0; i < num_reqs; ++i)
    if (ctx_len[i] + q_len[i] > max_keys) max_keys = ctx_len[i] + q_len[i];
  int used = 1;
#ifdef _OPENMP
  if (num_threads > 0) omp_set_num_threads(num_threads);
#endif
  int64_t tasks = (int64_t)num_reqs * Hq;
#pragma omp parallel
  {
#ifdef _OPENMP
#pragma omp single
    used = omp_get_num_threads();
#endif
    double* scores = (double*)malloc(sizeof(double) * (size_t)max_keys);
#pragma omp for schedule(dynamic, 1)
    for (int64_t task = 0; task < tasks; ++task) {
      int i = (int)(task / Hq);
      int h = (int)(task % Hq);
      for (int j = 0; j < q_len[i]; ++j) {
        int64_t row = q_start[i] + j;
        attend_row(i, j, h, Hq, Hkv, D, P, (double)scale, ctx_len, block_table,
                   max_pages_per_req, row, q, k_cache, v_cache, scores,
                   out + ((size_t)row * Hq + h) * D);
      }
    }
    free(scores);
  }
  free(q_start);
  return used;
}

/*
 * The same definition evaluated only at selected (token row, q head) pairs,
 * for checking sampled outputs of full-size batches.  out_sel is [n_sel, D].
 */
int oracle_attention_rows(int Hq, int Hkv, int D, int P, float scale, int num_reqs,
                          const int32_t* q_len, const int32_t* ctx_len,
                          const int32_t* block_table, int max_pages_per_req, const uint16_t* q,
                          const uint16_t* k_cache, const uint16_t* v_cache,
                          const int64_t* sel_row, const int32_t* sel_head, int64_t n_sel,
                          double* out_sel, int num_threads) {
  int64_t* q_start = (int64_t*)malloc(sizeof(int64_t) * (num_reqs > 0 ? num_reqs : 1));
  prefix_sum(q_len, num_reqs, q_start);
  int max_keys = 1;
  for (int i = 0; i < num_reqs; ++i)
    if (ctx_len[i] + q_len[i] > max_keys) max_keys = ctx_len[i] + q_len[i];
  int used = 1;
#ifdef _OPENMP
  if (num_threads > 0) omp_set_num_threads(num_threads);
#endif
#pragma omp parallel
  {
#ifdef _OPENMP
#pragma omp single
    used = omp_get_num_threads();
#endif
    double* scores = (double*)malloc(sizeof(double) * (size_t)max_keys);
#pragma omp for schedule(dynamic, 1)
    for (int64_t s = 0; s < n_sel; ++s) {
      int64_t row = sel_row[s];
      int i = 0; /* owning request: the last one whose first row is <= row */
      while (i + 1 < num_reqs && q_start[i + 1] <= row) ++i;
      int j = (int)(row - q_start[i]);
      attend_row(i, j, sel_head[s], Hq, Hkv, D, P, (double)scale, ctx_len, block_table,
                 max_pages_per_req, row, q, k_cache, v_cache, scores, out_sel + (size_t)s * D);
    }
    free(scores);
  }
  free(q_start);
  return used;
}
