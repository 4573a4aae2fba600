/* CPU oracle for the KV-cache streaming path.  TEST INFRASTRUCTURE ONLY (see
 * dv_oracle.h).  Plain nested loops over the logical coordinates, one element
 * at a time, written for checking by eye rather than for speed.
 *
 * Reading of the paper that fixes what is copied:
 *  - the prompt pass fills every layer's K and V for all prompt tokens and
 *    each decode step appends one token per layer (Sec. 2.1), so a prompt
 *    stream selects tokens [0, len_b) and a step-i increment the single token
 *    len_b + i of each sequence (Sec. 4.1.1, Figure "cache_ft");
 *  - the small non-contiguous updates are aggregated in one contiguous buffer
 *    (Sec. 4.1.1, optimisation 1); the paper does not fix the order inside
 *    that buffer, so the wire order [layer][K|V][sequence][head][token][dim]
 *    is this implementation's choice (layer outermost so layer-by-layer
 *    chunks, optimisation 2, concatenate);
 *  - the receiver writes exactly the streamed positions (restore of a lost
 *    cache, Sec. 4.2.3; swap-in of a microbatch, Sec. 4.2.2).
 *
 * Planted-mistake builds: compiling with -DDVO_MUTANT=k changes one term of
 * the arithmetic below.  The CPU tests build each mutant and check that the
 * pins catch it; the normal build has DVO_MUTANT undefined.
 */
#include "dv_oracle.h"

#include <stdlib.h>
#include <string.h>

#ifndef DVO_MUTANT
#define DVO_MUTANT 0
#endif

int64_t dvo_storage_elems(const dvo_layout* c) {
  if (c->kind == DVO_PAGED)
    return c->layers * 2 * c->num_blocks * c->heads * c->block_size * c->head_dim;
  return c->layers * 2 * c->batch * c->heads * c->seq_cap * c->head_dim;
}

static int64_t token_capacity(const dvo_layout* c) {
  if (c->kind == DVO_PAGED) return c->max_blocks * c->block_size;
  return c->seq_cap;
}

int64_t dvo_elem_index(const dvo_layout* c, int64_t l, int64_t kv, int64_t b, int64_t h,
                       int64_t s, int64_t d) {
  const int64_t L = c->layers, H = c->heads, D = c->head_dim, B = c->batch;
  if (l < 0 || l >= L || kv < 0 || kv > 1 || b < 0 || b >= B || h < 0 || h >= H || s < 0 ||
      s >= token_capacity(c) || d < 0 || d >= D)
    return -1;
  if (c->kind == DVO_DENSE || (c->kind == DVO_KSPLIT && kv == 1)) {
    const int64_t S = c->seq_cap;
#if DVO_MUTANT == 1 /* planted: heads and sequences swapped */
    return ((((l * 2 + kv) * H + h) * B + b) * S + s) * D + d;
#elif DVO_MUTANT == 2 /* planted: K and V swapped */
    return (((((l * 2 + (1 - kv)) * B + b) * H + h) * S + s) * D + d);
#else
    return ((((l * 2 + kv) * B + b) * H + h) * S + s) * D + d;
#endif
  }
  if (c->kind == DVO_KSPLIT) {
    const int64_t S = c->seq_cap;
    const int64_t x = 16 / c->elem_bytes;
#if DVO_MUTANT == 3 /* planted: split key stored without the split */
    return ((((l * 2) * B + b) * H + h) * S + s) * D + d;
#else
    return (((((l * 2) * B + b) * H + h) * (D / x) + d / x) * S + s) * x + d % x;
#endif
  }
  if (c->kind == DVO_PAGED) {
    const int64_t bs = c->block_size, NB = c->num_blocks;
    const int64_t blk = c->block_table[b * c->max_blocks + s / bs];
    if (blk < 0 || blk >= NB) return -1;
#if DVO_MUTANT == 4 /* planted: block table ignored (identity) */
    return ((((l * 2 + kv) * NB + (b * c->max_blocks + s / bs) % NB) * H + h) * bs + s % bs) * D + d;
#else
    return ((((l * 2 + kv) * NB + blk) * H + h) * bs + s % bs) * D + d;
#endif
  }
  return -1;
}

int dvo_check(const dvo_layout* c, int64_t l0, int64_t l1, const int32_t* t0, const int32_t* t1) {
  if (c->elem_bytes <= 0 || c->layers <= 0 || c->heads <= 0 || c->head_dim <= 0 ||
      c->batch <= 0)
    return DVO_INVALID;
  if (c->kind == DVO_PAGED) {
    if (c->block_size <= 0 || c->num_blocks <= 0 || c->max_blocks <= 0 || !c->block_table)
      return DVO_INVALID;
  } else if (c->kind == DVO_DENSE || c->kind == DVO_KSPLIT) {
    if (c->seq_cap <= 0) return DVO_INVALID;
    if (c->kind == DVO_KSPLIT &&
        (16 % c->elem_bytes != 0 || c->head_dim % (16 / c->elem_bytes) != 0))
      return DVO_INVALID;
  } else {
    return DVO_INVALID;
  }
  if (l0 < 0 || l1 < l0 || l1 > c->layers) return DVO_RANGE;
  for (int64_t b = 0; b < c->batch; ++b) {
    if (t0[b] < 0 || t1[b] < t0[b] || t1[b] > token_capacity(c)) return DVO_RANGE;
    if (c->kind == DVO_PAGED) {
      for (int64_t s = t0[b]; s < t1[b]; ++s) {
        const int32_t blk = c->block_table[b * c->max_blocks + s / c->block_size];
        if (blk < 0 || blk >= c->num_blocks) return DVO_RANGE;
      }
    }
  }
  return DVO_OK;
}

int64_t dvo_wire_elems(const dvo_layout* c, int64_t l0, int64_t l1, const int32_t* t0,
                       const int32_t* t1) {
  int64_t N = 0;
  for (int64_t b = 0; b < c->batch; ++b) N += (int64_t)t1[b] - t0[b];
  return (l1 - l0) * 2 * c->heads * c->head_dim * N;
}

/* Exclusive prefix of the per-sequence token counts: P[b] = sum_{b'<b} n_b'.
 * Returns N.  P must hold batch entries. */
static int64_t token_prefix(const dvo_layout* c, const int32_t* t0, const int32_t* t1,
                            int64_t* P) {
  int64_t acc = 0;
  for (int64_t b = 0; b < c->batch; ++b) {
    P[b] = acc;
    acc += (int64_t)t1[b] - t0[b];
  }
  return acc;
}

/* Wire element index of X(l,kv,b,h,s,d), written out from the definition. */
static int64_t wire_index(const dvo_layout* c, int64_t l0, int64_t N, const int64_t* P,
                          const int32_t* t0, const int32_t* t1, int64_t l, int64_t kv,
                          int64_t b, int64_t h, int64_t s, int64_t d) {
  const int64_t H = c->heads, D = c->head_dim;
  const int64_t n_b = (int64_t)t1[b] - t0[b];
#if DVO_MUTANT == 5 /* planted: token and head order swapped inside a sequence */
  return ((l - l0) * 2 + kv) * N * H * D + P[b] * H * D + (s - t0[b]) * H * D + h * D + d;
#elif DVO_MUTANT == 6 /* planted: ragged prefix ignored (uniform stride) */
  return ((l - l0) * 2 + kv) * N * H * D + b * n_b * H * D + h * n_b * D + (s - t0[b]) * D + d;
#else
  return ((l - l0) * 2 + kv) * N * H * D + P[b] * H * D + h * n_b * D + (s - t0[b]) * D + d;
#endif
}

static void copy_elem(void* dst, int64_t di, const void* src, int64_t si, int64_t E) {
  memcpy((char*)dst + di * E, (const char*)src + si * E, (size_t)E);
}

int dvo_pack(const dvo_layout* c, const void* cache, int64_t l0, int64_t l1, const int32_t* t0,
             const int32_t* t1, void* wire) {
  int rc = dvo_check(c, l0, l1, t0, t1);
  if (rc != DVO_OK) return rc;
  int64_t* P = (int64_t*)malloc(sizeof(int64_t) * (size_t)c->batch);
  const int64_t N = token_prefix(c, t0, t1, P);
  for (int64_t l = l0; l < l1; ++l)
    for (int64_t kv = 0; kv < 2; ++kv)
      for (int64_t b = 0; b < c->batch; ++b)
        for (int64_t h = 0; h < c->heads; ++h)
          for (int64_t s = t0[b]; s < t1[b]; ++s)
            for (int64_t d = 0; d < c->head_dim; ++d)
              copy_elem(wire, wire_index(c, l0, N, P, t0, t1, l, kv, b, h, s, d), cache,
                        dvo_elem_index(c, l, kv, b, h, s, d), c->elem_bytes);
  free(P);
  return DVO_OK;
}

int dvo_unpack(const dvo_layout* c, void* cache, int64_t l0, int64_t l1, const int32_t* t0,
               const int32_t* t1, const void* wire) {
  int rc = dvo_check(c, l0, l1, t0, t1);
  if (rc != DVO_OK) return rc;
  int64_t* P = (int64_t*)malloc(sizeof(int64_t) * (size_t)c->batch);
  const int64_t N = token_prefix(c, t0, t1, P);
  for (int64_t l = l0; l < l1; ++l)
    for (int64_t kv = 0; kv < 2; ++kv)
      for (int64_t b = 0; b < c->batch; ++b)
        for (int64_t h = 0; h < c->heads; ++h)
          for (int64_t s = t0[b]; s < t1[b]; ++s)
            for (int64_t d = 0; d < c->head_dim; ++d)
              copy_elem(cache, dvo_elem_index(c, l, kv, b, h, s, d), wire,
                        wire_index(c, l0, N, P, t0, t1, l, kv, b, h, s, d), c->elem_bytes);
  free(P);
  return DVO_OK;
}

int dvo_copy_ranges(const dvo_layout* sl, const void* src, const dvo_layout* dl, void* dst,
                    int64_t l0, int64_t l1, const int32_t* t0, const int32_t* t1) {
  if (sl->layers != dl->layers || sl->heads != dl->heads || sl->head_dim != dl->head_dim ||
      sl->batch != dl->batch || sl->elem_bytes != dl->elem_bytes)
    return DVO_INVALID;
  int rc = dvo_check(sl, l0, l1, t0, t1);
  if (rc != DVO_OK) return rc;
  rc = dvo_check(dl, l0, l1, t0, t1);
  if (rc != DVO_OK) return rc;
  for (int64_t l = l0; l < l1; ++l)
    for (int64_t kv = 0; kv < 2; ++kv)
      for (int64_t b = 0; b < sl->batch; ++b)
        for (int64_t h = 0; h < sl->heads; ++h)
          for (int64_t s = t0[b]; s < t1[b]; ++s)
            for (int64_t d = 0; d < sl->head_dim; ++d)
              copy_elem(dst, dvo_elem_index(dl, l, kv, b, h, s, d), src,
                        dvo_elem_index(sl, l, kv, b, h, s, d), sl->elem_bytes);
  return DVO_OK;
}

int dvo_wire_to_storage(const dvo_layout* c, int64_t l0, int64_t l1, const int32_t* t0,
                        const int32_t* t1, const int64_t* w, int64_t n, int64_t* out) {
  int rc = dvo_check(c, l0, l1, t0, t1);
  if (rc != DVO_OK) return rc;
  const int64_t H = c->heads, D = c->head_dim;
  int64_t* P = (int64_t*)malloc(sizeof(int64_t) * (size_t)c->batch);
  const int64_t N = token_prefix(c, t0, t1, P);
  const int64_t total = (l1 - l0) * 2 * H * D * N;
  for (int64_t i = 0; i < n; ++i) {
    int64_t r = w[i];
    if (r < 0 || r >= total) {
      out[i] = -1;
      continue;
    }
    /* Invert the wire index: slab (layer, K|V), then sequence by the prefix,
     * then head, token and dimension. */
    const int64_t slab = r / (N * H * D);
    r -= slab * N * H * D;
    const int64_t l = l0 + slab / 2, kv = slab % 2;
    int64_t b = 0;
    while (!(P[b] * H * D <= r && r < (P[b] + (int64_t)t1[b] - t0[b]) * H * D)) ++b;
    r -= P[b] * H * D;
    const int64_t n_b = (int64_t)t1[b] - t0[b];
    const int64_t h = r / (n_b * D);
    r -= h * n_b * D;
    const int64_t s = t0[b] + r / D;
    const int64_t d = r % D;
    out[i] = dvo_elem_index(c, l, kv, b, h, s, d);
  }
  free(P);
  return DVO_OK;
}
