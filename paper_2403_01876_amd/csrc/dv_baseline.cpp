// Comparison baseline of the paper's evaluation (Sec. 5.1, "Baseline"): the
// non-contiguous cache region is moved with one copy call per contiguous
// region instead of being packed into a temporary buffer first.  It is not
// part of the streaming path; the benchmark times it against the buffered
// path (pack kernel + one copy), and the tests check it produces the same
// bytes in the same order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dv.h"

extern "C" {

// Dense caches only: for each (layer, K|V, sequence, head) of the ranges,
// one hipMemcpyAsync of the run of tokens [t0[b], t1[b]) into `dst` at its
// position in the contiguous buffer order of include/dv.h.  Returns the
// number of copy calls issued, or a negative dv_status.
DV_API int64_t dvb_per_region_copy(const dv_cache* c, int32_t mb, int32_t l0, int32_t l1,
                            const int32_t* t0, const int32_t* t1, void* dst, uint64_t dst_cap,
                            void* stream) {
  if (!c || c->kind != DV_DENSE || !c->mb_base || mb < 0 || mb >= c->num_mb || !t0 || !t1 ||
      !dst)
    return DV_ERR_INVALID;
  uint64_t need = 0;
  int rc = dv_packed_bytes(c, l0, l1, t0, t1, &need);
  if (rc != DV_OK) return rc;
  if (need > dst_cap) return DV_ERR_SPACE;
  const int64_t H = c->num_heads, B = c->batch, S = c->max_seq;
  const int64_t tok = (int64_t)c->head_dim * c->elem_bytes;
  int64_t N = 0;
  for (int64_t b = 0; b < B; ++b) N += t1[b] - t0[b];
  const char* base = static_cast<const char*>(c->mb_base[mb]);
  char* out = static_cast<char*>(dst);
  hipStream_t st = static_cast<hipStream_t>(stream);
  int64_t calls = 0;
  for (int64_t l = l0; l < l1; ++l)
    for (int64_t kv = 0; kv < 2; ++kv) {
      int64_t p = 0;  // tokens of earlier sequences
      for (int64_t b = 0; b < B; ++b) {
        const int64_t n = t1[b] - t0[b];
        for (int64_t h = 0; h < H && n > 0; ++h) {
          const char* src = base + ((((l * 2 + kv) * B + b) * H + h) * S + t0[b]) * tok;
          char* d = out + (((l - l0) * 2 + kv) * N * H + p * H + h * n) * tok;
          if (hipMemcpyAsync(d, src, n * tok, hipMemcpyDefault, st) != hipSuccess)
            return DV_ERR_HIP;
          ++calls;
        }
        p += n;
      }
    }
  return calls;
}

}  // extern "C"
