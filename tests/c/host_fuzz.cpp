// Host-side fuzz of the C ABI's argument checks, built with AddressSanitizer
// and UndefinedBehaviorSanitizer (tests/test_host_sanitizers.py).
//
// Random descriptors, ranges and pointers -- extents from a mix of valid,
// zero, negative, boundary and huge values; null, misaligned and aligned
// made-up addresses -- go through every entry point.  Each call must return a
// dv_status, and the sanitizers must stay silent: no out-of-bounds read of
// the caller's arrays, no signed overflow in the size arithmetic.  The
// made-up addresses are never dereferenced by the host checks; a call that
// passes them reaches the HIP runtime, which must refuse it.  So this program
// runs only where no GPU is visible (the test checks), and its own arrays
// always hold as many entries as the descriptor says.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "../../include/dv.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;

uint64_t next() {  // SplitMix64 (Steele, Lea and Flood, OOPSLA 2014)
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

int64_t pick(const std::vector<int64_t>& v) { return v[next() % v.size()]; }

// An int32 extent: small valid values most of the time, else an edge.
int32_t extent(int32_t small_max) {
  if (next() % 4) return 1 + (int32_t)(next() % small_max);
  return (int32_t)pick({0, -1, -7, 1, 2, 16, 64, 1 << 16, (1 << 24) + 1, (1 << 30),
                        INT32_MAX, INT32_MIN});
}

// A made-up address: mostly far from the descriptor's regions (which start
// at 2^40), sometimes null, misaligned or inside them.
void* address() {
  switch (next() % 8) {
    case 0: return nullptr;
    case 1: return (void*)(uintptr_t)((1ull << 40) + 8);  // misaligned
    case 2: return (void*)(uintptr_t)((1ull << 40) + (next() % 64) * (1ull << 34));
    default: return (void*)(uintptr_t)((1ull << 46) + (next() % 64) * (1ull << 40));
  }
}

bool is_status(int64_t rc) { return rc <= 0 && rc >= -5; }

int failures = 0;

// Status counts per entry point, printed at the end: they show how far the
// random calls got (sized, refused by which check, or handed to the runtime).
struct Tally {
  const char* name;
  long count[6];
};
std::vector<Tally> g_tally;

void expect_status(int64_t rc, const char* what, int iter) {
  if (!is_status(rc)) {
    fprintf(stderr, "iteration %d: %s returned %lld\n", iter, what, (long long)rc);
    ++failures;
    return;
  }
  for (Tally& t : g_tally)
    if (t.name == what || strcmp(t.name, what) == 0) {
      ++t.count[-rc];
      return;
    }
  Tally t = {what, {0, 0, 0, 0, 0, 0}};
  t.count[-rc] = 1;
  g_tally.push_back(t);
}

}  // namespace

int main(int argc, char** argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 20000;
  if (argc > 2) g_state = strtoull(argv[2], nullptr, 0);
  for (int it = 0; it < iters; ++it) {
    // a valid descriptor and ranges first, then 0-2 fields set to an edge
    dv_cache c;
    memset(&c, 0, sizeof c);
    c.kind = (int32_t)(next() % 3);
    c.mem = DV_MEM_DEVICE;
    c.elem_bytes = (int32_t)pick({1, 2, 4, 8});
    c.head_dim = (int32_t)(pick({1, 2, 4, 8, 16, 32, 64}) * 16 / c.elem_bytes);
    c.num_layers = 1 + (int32_t)(next() % 4);
    c.num_heads = 1 + (int32_t)(next() % 8);
    // the caller's arrays hold `batch` entries, so batch stays within them
    c.batch = (int32_t)pick({1, 2, 3, 63, 64, 65, 130});
    c.max_seq = 1 + (int32_t)(next() % 96);
    c.block_size = 1 + (int32_t)(next() % 16);
    c.num_blocks = 1 + (int32_t)(next() % 64);
    c.max_blocks = 1 + (int32_t)(next() % 8);
    c.num_mb = 1 + (int32_t)(next() % 3);
    const int nmb = 3;
    std::vector<void*> bases(nmb), owners(nmb);
    std::vector<const int32_t*> tables(nmb);
    for (int i = 0; i < nmb; ++i) {  // disjoint made-up regions, 2^34 bytes apart
      bases[i] = (void*)(uintptr_t)((1ull << 40) + (uint64_t)i * (1ull << 34));
      tables[i] = (const int32_t*)(uintptr_t)((1ull << 42) + (uint64_t)i * (1ull << 34));
      owners[i] = next() % 2 ? nullptr
                             : (void*)(uintptr_t)((1ull << 43) + (uint64_t)i * (1ull << 34));
    }
    c.mb_base = bases.data();
    c.block_table = tables.data();
    c.block_owner = next() % 2 ? (int32_t* const*)owners.data() : nullptr;
    const int nb = c.batch;
    const int64_t cap_tok = c.kind == DV_PAGED ? (int64_t)c.block_size * c.max_blocks : c.max_seq;
    std::vector<int32_t> t0(nb), t1(nb), pos(nb);
    for (int b = 0; b < nb; ++b) {
      t0[b] = (int32_t)(next() % (uint64_t)(cap_tok + 1));
      t1[b] = t0[b] + (int32_t)(next() % (uint64_t)(cap_tok - t0[b] + 1));
      pos[b] = (int32_t)(next() % (uint64_t)cap_tok) - (next() % 8 == 0 ? (int32_t)cap_tok : 0);
    }
    for (int m = (int)(next() % 3); m > 0; --m) {
      const int32_t edge = (int32_t)pick({0, -1, -7, 1 << 16, (1 << 24) + 1, 1 << 30, INT32_MAX,
                                          INT32_MIN, 3});
      switch (next() % 16) {
        case 0: c.kind = (int32_t)pick({-1, 3, INT32_MAX}); break;
        case 1: c.mem = (int32_t)pick({-1, 2}); break;
        case 2: c.elem_bytes = (int32_t)pick({0, -2, 3, 16}); break;
        case 3: c.num_layers = edge; break;
        case 4: c.num_heads = edge; break;
        case 5: c.head_dim = (int32_t)pick({0, -64, 7, 1 << 19, (1 << 19) + 8, 1 << 20}); break;
        case 6: c.batch = (int32_t)pick({0, -1}); break;  // never above the arrays
        case 7: c.max_seq = edge; break;
        case 8: c.block_size = edge; break;
        case 9: c.num_blocks = edge; break;
        case 10: c.max_blocks = edge; break;
        case 11: c.num_mb = (int32_t)pick({0, -1}); break;
        case 12: bases[next() % nmb] = address(); break;
        case 13: c.mb_base = nullptr; break;
        case 14: tables[next() % nmb] = (const int32_t*)address(); break;
        default: {
          const int b = (int)(next() % nb);
          const int32_t v = (int32_t)pick({-1, INT32_MAX, INT32_MIN, (int32_t)cap_tok + 1});
          if (next() % 2) t0[b] = v; else t1[b] = v;
          pos[b] = v;
        }
      }
    }
    const int32_t* r0 = next() % 8 ? t0.data() : nullptr;
    const int32_t* r1 = next() % 16 ? t1.data() : nullptr;
    const int32_t* rp = next() % 16 ? pos.data() : nullptr;
    int32_t l0 = (int32_t)pick({0, 0, 1, -1, 2});
    int32_t l1 = (int32_t)pick({1, 2, 4, 0, -1, INT32_MAX});
    if (next() % 8 == 0 && c.num_layers > 0) {  // the descriptor's last layer
      l0 = c.num_layers - 1;
      l1 = c.num_layers;
    }
    const int32_t mb = (int32_t)pick({0, 0, 1, -1, 2, INT32_MAX});
    void* buf = address();
    const uint64_t cap = (uint64_t)pick({0, 16, 1 << 20, 1ll << 40, -1});
    uint64_t out = 0;

    expect_status(dv_cache_bytes(&c, &out), "dv_cache_bytes", it);
    expect_status(dv_packed_bytes(&c, l0, l1, r0, r1, &out), "dv_packed_bytes", it);
    expect_status(dv_stream_out_prompt(&c, mb, l0, l1, r0, r1, buf, cap, &out, nullptr),
                  "dv_stream_out_prompt", it);
    expect_status(dv_stream_out_token(&c, mb, l0, l1, rp, buf, cap, &out, nullptr),
                  "dv_stream_out_token", it);
    expect_status(dv_stream_in(&c, mb, l0, l1, r0, r1, buf, cap, nullptr), "dv_stream_in", it);
    expect_status(dv_stream_in_noalloc(&c, mb, l0, l1, r0, r1, buf, cap, nullptr),
                  "dv_stream_in_noalloc", it);
    expect_status(dv_block_claims(&c, mb, r0, r1, (int32_t*)address(), nullptr),
                  "dv_block_claims", it);

    dv_cache h = c;  // a host mirror: same shape, its own capacity and kind
    h.mem = (int32_t)(next() % 2);
    h.max_seq = extent(96);
    expect_status(dv_swap_out(&c, mb, &h, (int32_t)pick({0, 1, -1}), l0, l1, r0, r1, nullptr),
                  "dv_swap_out", it);
    expect_status(dv_swap_in(&h, (int32_t)pick({0, 1, -1}), &c, mb, l0, l1, r0, r1, nullptr),
                  "dv_swap_in", it);

    dv_swapper* s = nullptr;
    const int rs = dv_swapper_create(next() % 16 ? &c : nullptr, next() % 16 ? &h : nullptr, &s);
    expect_status(rs, "dv_swapper_create", it);
    if (rs == DV_OK && s) {
      expect_status(dv_swapper_prefetch(s, mb, r1), "dv_swapper_prefetch", it);
      expect_status(dv_swapper_destroy(s), "dv_swapper_destroy", it);
    }
    dv_streamer* st = nullptr;
    const int rt = dv_streamer_create(next() % 16 ? &c : nullptr, mb, address(), cap, address(),
                                      cap, &st);
    expect_status(rt, "dv_streamer_create", it);
    if (rt == DV_OK && st) expect_status(dv_streamer_destroy(st), "dv_streamer_destroy", it);
    if (!dv_status_string((int)(next() % 9) - 6)) {
      fprintf(stderr, "iteration %d: null status string\n", it);
      ++failures;
    }
  }
  for (const Tally& t : g_tally)
    printf("%-22s ok %ld invalid %ld range %ld space %ld unsupported %ld hip %ld\n", t.name,
           t.count[0], t.count[1], t.count[2], t.count[3], t.count[4], t.count[5]);
  printf("%d iterations, %d failures\n", iters, failures);
  return failures ? 1 : 0;
}
