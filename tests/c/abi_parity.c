/* The boundary used from plain C on the GPU: a C99 program, linked against
 * libdv.so and the HIP runtime only (no Python, no torch), streams caches
 * through every streaming entry point on its own hipStream_t and compares
 * each result byte for byte with the CPU oracle (test infrastructure,
 * linked here to compute the expected bytes).  Inputs come from the seeded
 * host generator.
 *
 * Cases: dense and split-key prompt streams (layer sub-range, ragged and
 * empty ranges, several tiles per run) into sentinel receivers; decode-step
 * tokens with inactive sequences; a paged gather through a permuted table
 * and a scatter into another permutation with and without the owner-map
 * workspace; swaps to and from a pinned host mirror of another capacity on
 * both engines (one-token rows by kernel, long rows by DMA).
 *
 * Prints one line per case and "abi parity ok" at the end; exits 1 on a
 * mismatch and 2 on a runtime error. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "dv.h"
#include "dv_oracle.h"

void dvsynth_host_fill(void* out, uint64_t nbytes, uint64_t seed, uint64_t first_byte);

#define HIPCHECK(x)                                                                  \
  do {                                                                               \
    hipError_t e_ = (x);                                                             \
    if (e_ != hipSuccess) {                                                          \
      fprintf(stderr, "%s:%d %s\n", __FILE__, __LINE__, hipGetErrorString(e_));      \
      exit(2);                                                                       \
    }                                                                                \
  } while (0)

#define EXPECT(c, what)                                           \
  do {                                                            \
    if (!(c)) {                                                   \
      fprintf(stderr, "FAILED %s (%s:%d)\n", what, __FILE__, __LINE__); \
      exit(1);                                                    \
    }                                                             \
  } while (0)

static int cases = 0;

static uint8_t* host_filled(size_t n, uint64_t seed) {
  uint8_t* h = (uint8_t*)malloc(n ? n : 1);
  EXPECT(h != NULL, "host allocation");
  dvsynth_host_fill(h, n, seed, 0);
  return h;
}

static uint8_t* host_const(size_t n, int byte) {
  uint8_t* h = (uint8_t*)malloc(n ? n : 1);
  EXPECT(h != NULL, "host allocation");
  memset(h, byte, n);
  return h;
}

static void* to_device(const void* h, size_t n) {
  void* d = NULL;
  HIPCHECK(hipMalloc(&d, n ? n : 16));
  if (n) HIPCHECK(hipMemcpy(d, h, n, hipMemcpyHostToDevice));
  return d;
}

static uint8_t* to_host(const void* d, size_t n) {
  uint8_t* h = (uint8_t*)malloc(n ? n : 1);
  EXPECT(h != NULL, "host allocation");
  if (n) HIPCHECK(hipMemcpy(h, d, n, hipMemcpyDeviceToHost));
  return h;
}

static void same(const void* a, const void* b, size_t n, const char* what) {
  EXPECT(memcmp(a, b, n) == 0, what);
}

/* Small LCG for test tables (input generation only). */
static uint64_t lcg_state = 12345;
static uint32_t lcg_below(uint32_t n) {
  lcg_state = lcg_state * 6364136223846793005ull + 1442695040888963407ull;
  return (uint32_t)((lcg_state >> 33) % n);
}

static void permutation(int32_t* p, int n) {
  for (int i = 0; i < n; ++i) p[i] = i;
  for (int i = n - 1; i > 0; --i) {
    const int j = (int)lcg_below((uint32_t)i + 1);
    const int32_t t = p[i];
    p[i] = p[j];
    p[j] = t;
  }
}

static dv_cache dense_desc(int kind, int L, int H, int D, int B, int S, int mem, void** base) {
  dv_cache c;
  memset(&c, 0, sizeof c);
  c.kind = kind;
  c.mem = mem;
  c.elem_bytes = 2;
  c.num_layers = L;
  c.num_heads = H;
  c.head_dim = D;
  c.batch = B;
  c.max_seq = S;
  c.num_mb = 1;
  c.mb_base = base;
  return c;
}

static dvo_layout dense_oracle(int kind, int L, int H, int D, int B, int S) {
  dvo_layout o;
  memset(&o, 0, sizeof o);
  o.kind = kind == DV_DENSE ? DVO_DENSE : DVO_KSPLIT;
  o.elem_bytes = 2;
  o.layers = L;
  o.heads = H;
  o.head_dim = D;
  o.batch = B;
  o.seq_cap = S;
  return o;
}

/* Prompt-style stream out of a filled cache and back into a sentinel one. */
static void case_stream(hipStream_t st, int kind, int L, int H, int D, int B, int S, int l0,
                        int l1, const int32_t* t0, const int32_t* t1, uint64_t seed,
                        const char* name) {
  dvo_layout o = dense_oracle(kind, L, H, D, B, S);
  const size_t bytes = (size_t)dvo_storage_elems(&o) * 2;
  uint8_t* host = host_filled(bytes, seed);
  void* cache = to_device(host, bytes);
  void* base[1] = {cache};
  dv_cache c = dense_desc(kind, L, H, D, B, S, DV_MEM_DEVICE, base);

  /* decode-step tokens: one past each range end (inactive where that is at
     capacity or the range is empty) */
  enum { kMaxB = 256 };
  EXPECT(B <= kMaxB, "batch of the test");
  int32_t pos[kMaxB], a[kMaxB], e[kMaxB];
  for (int b = 0; b < B; ++b) {
    pos[b] = (t1[b] > t0[b] && t1[b] < S) ? t1[b] : -1;
    a[b] = pos[b] < 0 ? 0 : pos[b];
    e[b] = pos[b] < 0 ? 0 : pos[b] + 1;
  }
  uint64_t need = 0, tneed = 0;
  EXPECT(dv_packed_bytes(&c, l0, l1, t0, t1, &need) == DV_OK, "sizing");
  EXPECT(dv_packed_bytes(&c, l0, l1, a, e, &tneed) == DV_OK, "token sizing");
  EXPECT((int64_t)need == dvo_wire_elems(&o, l0, l1, t0, t1) * 2, "size against the oracle");
  uint8_t* exp = host_const(need, 0);
  EXPECT(dvo_pack(&o, host, l0, l1, t0, t1, exp) == DVO_OK, "oracle pack");
  void* wire = NULL;
  HIPCHECK(hipMalloc(&wire, (need > tneed ? need : tneed) + 16));
  uint64_t out = 0;
  EXPECT(dv_stream_out_prompt(&c, 0, l0, l1, t0, t1, wire, need, &out, st) == DV_OK,
         "dv_stream_out_prompt");
  EXPECT(out == need, "stream size");
  HIPCHECK(hipStreamSynchronize(st));
  uint8_t* got = to_host(wire, need);
  same(got, exp, need, "stream-out against the oracle");

  uint8_t* rexp = host_const(bytes, 0xA5);
  void* recv = to_device(rexp, bytes);
  void* rbase[1] = {recv};
  dv_cache r = dense_desc(kind, L, H, D, B, S, DV_MEM_DEVICE, rbase);
  EXPECT(dv_stream_in(&r, 0, l0, l1, t0, t1, wire, need, st) == DV_OK, "dv_stream_in");
  HIPCHECK(hipStreamSynchronize(st));
  EXPECT(dvo_unpack(&o, rexp, l0, l1, t0, t1, exp) == DVO_OK, "oracle unpack");
  uint8_t* rgot = to_host(recv, bytes);
  same(rgot, rexp, bytes, "stream-in against the oracle");

  if (tneed > 0) {
    uint8_t* texp = host_const(tneed, 0);
    EXPECT(dvo_pack(&o, host, l0, l1, a, e, texp) == DVO_OK, "oracle token pack");
    EXPECT(dv_stream_out_token(&c, 0, l0, l1, pos, wire, tneed, &out, st) == DV_OK,
           "dv_stream_out_token");
    EXPECT(out == tneed, "token size");
    HIPCHECK(hipStreamSynchronize(st));
    uint8_t* tgot = to_host(wire, tneed);
    same(tgot, texp, tneed, "token stream-out against the oracle");
    EXPECT(dv_stream_in(&r, 0, l0, l1, a, e, wire, tneed, st) == DV_OK, "token stream-in");
    HIPCHECK(hipStreamSynchronize(st));
    EXPECT(dvo_unpack(&o, rexp, l0, l1, a, e, texp) == DVO_OK, "oracle token unpack");
    free(rgot);
    rgot = to_host(recv, bytes);
    same(rgot, rexp, bytes, "token stream-in against the oracle");
    free(tgot);
    free(texp);
  }
  printf("%s: %llu bytes streamed, %llu per token step, bit-exact\n", name,
         (unsigned long long)need, (unsigned long long)tneed);
  ++cases;
  free(host);
  free(exp);
  free(got);
  free(rexp);
  free(rgot);
  HIPCHECK(hipFree(cache));
  HIPCHECK(hipFree(recv));
  HIPCHECK(hipFree(wire));
}

/* Paged gather through a permuted table, scatter into another permutation
   (table order, pool order through the owner-map workspace, and pool order
   through the library's own map with dv_stream_in_noalloc). */
static void case_paged(hipStream_t st) {
  enum { L = 2, H = 6, D = 128, B = 5, BS = 16, MAXB = 12 };
  const int32_t t0[B] = {0, 17, 0, 5, 40};
  const int32_t t1[B] = {150, 17, 33, 100, 190};
  int32_t used[B], nb = 0;
  for (int b = 0; b < B; ++b) {
    used[b] = (t1[b] + BS - 1) / BS;
    nb += used[b];
  }
  int32_t perm_a[64], perm_b[64], bt_a[B * MAXB], bt_b[B * MAXB];
  EXPECT(nb <= 64, "pool size");
  permutation(perm_a, nb);
  permutation(perm_b, nb);
  /* sequence b's first used[b] logical blocks take the next pool blocks of
     each permutation; the rest of its row is unmapped */
  int k = 0;
  for (int b = 0; b < B; ++b) {
    for (int j = 0; j < MAXB; ++j) {
      bt_a[b * MAXB + j] = j < used[b] ? perm_a[k + j] : -1;
      bt_b[b * MAXB + j] = j < used[b] ? perm_b[k + j] : -1;
    }
    k += used[b];
  }

  dvo_layout oa, ob;
  memset(&oa, 0, sizeof oa);
  oa.kind = DVO_PAGED;
  oa.elem_bytes = 2;
  oa.layers = L;
  oa.heads = H;
  oa.head_dim = D;
  oa.batch = B;
  oa.block_size = BS;
  oa.num_blocks = nb;
  oa.max_blocks = MAXB;
  oa.block_table = bt_a;
  ob = oa;
  ob.block_table = bt_b;
  const size_t bytes = (size_t)dvo_storage_elems(&oa) * 2;
  uint8_t* host = host_filled(bytes, 77);
  void* pool = to_device(host, bytes);
  void* dbt_a = to_device(bt_a, sizeof bt_a);
  void* dbt_b = to_device(bt_b, sizeof bt_b);
  void* base[1] = {pool};
  const int32_t* tab_a[1] = {(const int32_t*)dbt_a};
  dv_cache c;
  memset(&c, 0, sizeof c);
  c.kind = DV_PAGED;
  c.mem = DV_MEM_DEVICE;
  c.elem_bytes = 2;
  c.num_layers = L;
  c.num_heads = H;
  c.head_dim = D;
  c.batch = B;
  c.block_size = BS;
  c.num_blocks = nb;
  c.max_blocks = MAXB;
  c.num_mb = 1;
  c.mb_base = base;
  c.block_table = tab_a;

  uint64_t need = 0, out = 0;
  EXPECT(dv_packed_bytes(&c, 0, L, t0, t1, &need) == DV_OK, "paged sizing");
  uint8_t* exp = host_const(need, 0);
  EXPECT(dvo_pack(&oa, host, 0, L, t0, t1, exp) == DVO_OK, "oracle paged pack");
  void* wire = NULL;
  HIPCHECK(hipMalloc(&wire, need));
  EXPECT(dv_stream_out_prompt(&c, 0, 0, L, t0, t1, wire, need, &out, st) == DV_OK,
         "paged gather");
  HIPCHECK(hipStreamSynchronize(st));
  uint8_t* got = to_host(wire, need);
  same(got, exp, need, "paged gather against the oracle");

  uint8_t* rexp = host_const(bytes, 0x3C);
  EXPECT(dvo_unpack(&ob, rexp, 0, L, t0, t1, exp) == DVO_OK, "oracle paged unpack");
  void* owner = NULL;
  HIPCHECK(hipMalloc(&owner, (size_t)nb * 4));
  static const char* const kScatter[3] = {
      "paged scatter in table order against the oracle",
      "paged scatter in pool order against the oracle",
      "paged scatter without allocation (dv_stream_in_noalloc) against the oracle"};
  for (int order = 0; order < 3; ++order) {
    uint8_t* sentinel = host_const(bytes, 0x3C);
    void* recv = to_device(sentinel, bytes);
    void* rbase[1] = {recv};
    const int32_t* tab_b[1] = {(const int32_t*)dbt_b};
    int32_t* own[1] = {(int32_t*)owner};
    dv_cache r = c;
    r.mb_base = rbase;
    r.block_table = tab_b;
    r.block_owner = order == 1 ? own : NULL;
    const int rc = order == 2 ? dv_stream_in_noalloc(&r, 0, 0, L, t0, t1, wire, need, st)
                              : dv_stream_in(&r, 0, 0, L, t0, t1, wire, need, st);
    EXPECT(rc == DV_OK, "paged scatter");
    HIPCHECK(hipStreamSynchronize(st));
    uint8_t* rgot = to_host(recv, bytes);
    same(rgot, rexp, bytes, kScatter[order]);
    free(sentinel);
    free(rgot);
    HIPCHECK(hipFree(recv));
  }
  printf("paged: %d pool blocks, %llu bytes gathered and scattered three ways, bit-exact\n", nb,
         (unsigned long long)need);
  ++cases;
  free(host);
  free(exp);
  free(got);
  free(rexp);
  HIPCHECK(hipFree(pool));
  HIPCHECK(hipFree(dbt_a));
  HIPCHECK(hipFree(dbt_b));
  HIPCHECK(hipFree(wire));
  HIPCHECK(hipFree(owner));
}

/* Swap out to and back in from a pinned host mirror of another capacity. */
static void case_swap(hipStream_t st, const int32_t* t0, const int32_t* t1, const char* name) {
  enum { L = 2, H = 3, D = 128, B = 4, SD = 600, SH = 520 };
  dvo_layout od = dense_oracle(DV_DENSE, L, H, D, B, SD);
  dvo_layout oh = dense_oracle(DV_DENSE, L, H, D, B, SH);
  const size_t dbytes = (size_t)dvo_storage_elems(&od) * 2;
  const size_t hbytes = (size_t)dvo_storage_elems(&oh) * 2;
  uint8_t* src = host_filled(dbytes, 99);
  void* slot = to_device(src, dbytes);
  void* mirror = NULL;
  HIPCHECK(hipHostMalloc(&mirror, hbytes, hipHostMallocDefault));
  memset(mirror, 0x6B, hbytes);
  void* dbase[1] = {slot};
  void* hbase[1] = {mirror};
  dv_cache dev = dense_desc(DV_DENSE, L, H, D, B, SD, DV_MEM_DEVICE, dbase);
  dv_cache hst = dense_desc(DV_DENSE, L, H, D, B, SH, DV_MEM_HOST_PINNED, hbase);

  uint8_t* hexp = host_const(hbytes, 0x6B);
  EXPECT(dvo_copy_ranges(&od, src, &oh, hexp, 0, L, t0, t1) == DVO_OK, "oracle copy out");
  EXPECT(dv_swap_out(&dev, 0, &hst, 0, 0, L, t0, t1, st) == DV_OK, "dv_swap_out");
  HIPCHECK(hipStreamSynchronize(st));
  same(mirror, hexp, hbytes, "swap-out against the oracle");

  /* back into a cleared slot */
  uint8_t* dexp = host_const(dbytes, 0);
  HIPCHECK(hipMemset(slot, 0, dbytes));
  EXPECT(dvo_copy_ranges(&oh, hexp, &od, dexp, 0, L, t0, t1) == DVO_OK, "oracle copy in");
  EXPECT(dv_swap_in(&hst, 0, &dev, 0, 0, L, t0, t1, st) == DV_OK, "dv_swap_in");
  HIPCHECK(hipStreamSynchronize(st));
  uint8_t* dgot = to_host(slot, dbytes);
  same(dgot, dexp, dbytes, "swap-in against the oracle");
  printf("%s: bit-exact both ways\n", name);
  ++cases;
  free(src);
  free(hexp);
  free(dexp);
  free(dgot);
  HIPCHECK(hipFree(slot));
  HIPCHECK(hipHostFree(mirror));
}

/* The swap scheduler: three host microbatches through two slots for two
   rounds; each step writes one token per sequence into its slot, and the
   scheduler swaps that update out.  Every mirror then equals the oracle's. */
static void case_scheduler(hipStream_t st) {
  enum { L = 2, H = 3, D = 64, B = 3, S = 64, M = 3, ROUNDS = 2 };
  dvo_layout od = dense_oracle(DV_DENSE, L, H, D, B, S);
  const size_t bytes = (size_t)dvo_storage_elems(&od) * 2;
  void* slots[2];
  void* mirrors[M];
  uint8_t* exp[M];
  int32_t len[M][B];
  for (int i = 0; i < 2; ++i) {
    HIPCHECK(hipMalloc(&slots[i], bytes));
    HIPCHECK(hipMemset(slots[i], 0, bytes));
  }
  for (int x = 0; x < M; ++x) {
    exp[x] = host_filled(bytes, 200 + x);
    HIPCHECK(hipHostMalloc(&mirrors[x], bytes, hipHostMallocDefault));
    memcpy(mirrors[x], exp[x], bytes);
    for (int b = 0; b < B; ++b) len[x][b] = 20 + 3 * b + x;
  }
  dv_cache dev = dense_desc(DV_DENSE, L, H, D, B, S, DV_MEM_DEVICE, slots);
  dev.num_mb = 2;
  dv_cache hst = dense_desc(DV_DENSE, L, H, D, B, S, DV_MEM_HOST_PINNED, mirrors);
  hst.num_mb = M;
  dv_swapper* sw = NULL;
  EXPECT(dv_swapper_create(&dev, &hst, &sw) == DV_OK, "dv_swapper_create");
  const int32_t one[B] = {1, 1, 1};
  uint64_t n = 0;
  {
    int32_t t1[B];
    for (int b = 0; b < B; ++b) t1[b] = one[b];
    EXPECT(dv_packed_bytes(&dev, 0, L, NULL, t1, &n) == DV_OK, "token size");
  }
  void* wire = NULL;
  HIPCHECK(hipMalloc(&wire, n));
  EXPECT(dv_swapper_prefetch(sw, 0, len[0]) == DV_OK, "first prefetch");
  for (int k = 0; k < ROUNDS * M; ++k) {
    const int x = k % M, xn = (k + 1) % M;
    if (k + 1 < ROUNDS * M)
      EXPECT(dv_swapper_prefetch(sw, xn, len[xn]) == DV_OK, "prefetch");
    int32_t slot = -1;
    EXPECT(dv_swapper_begin_step(sw, x, st, &slot) == DV_OK, "begin_step");
    int32_t t1[B];
    for (int b = 0; b < B; ++b) t1[b] = len[x][b] + 1;
    uint8_t* tok = host_filled(n, 700 + k);
    HIPCHECK(hipMemcpyAsync(wire, tok, n, hipMemcpyHostToDevice, st));
    EXPECT(dv_stream_in(&dev, slot, 0, L, len[x], t1, wire, n, st) == DV_OK, "step's token");
    EXPECT(dvo_unpack(&od, exp[x], 0, L, len[x], t1, tok) == DVO_OK, "oracle token");
    EXPECT(dv_swapper_end_step(sw, x, st, len[x], t1) == DV_OK, "end_step");
    HIPCHECK(hipStreamSynchronize(st));  /* the token's host buffer is reused */
    free(tok);
    for (int b = 0; b < B; ++b) len[x][b] += 1;
  }
  EXPECT(dv_swapper_sync(sw) == DV_OK, "dv_swapper_sync");
  EXPECT(dv_swapper_destroy(sw) == DV_OK, "dv_swapper_destroy");
  for (int x = 0; x < M; ++x) same(mirrors[x], exp[x], bytes, "scheduler mirror against the oracle");
  printf("swap scheduler: %d microbatches, %d rounds through 2 slots, bit-exact\n", M, ROUNDS);
  ++cases;
  for (int x = 0; x < M; ++x) {
    free(exp[x]);
    HIPCHECK(hipHostFree(mirrors[x]));
  }
  for (int i = 0; i < 2; ++i) HIPCHECK(hipFree(slots[i]));
  HIPCHECK(hipFree(wire));
}

int main(void) {
  int ndev = 0;
  HIPCHECK(hipGetDeviceCount(&ndev));
  EXPECT(ndev > 0, "a GPU");
  HIPCHECK(hipSetDevice(0));
  hipStream_t st;
  HIPCHECK(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));
  EXPECT(dv_api_version() == DV_API_VERSION, "library version matches the header");

  {
    /* 3 layers, 5 heads x 64 dims, 6 sequences, capacity 300: ragged and
       empty ranges, runs of several 8 KB tiles, layers [1, 3) */
    const int32_t t0[6] = {0, 7, 0, 299, 13, 40};
    const int32_t t1[6] = {300, 7, 1, 300, 277, 233};
    case_stream(st, DV_DENSE, 3, 5, 64, 6, 300, 1, 3, t0, t1, 11, "dense");
    case_stream(st, DV_DENSE_KSPLIT, 3, 5, 64, 6, 300, 0, 3, t0, t1, 12, "split key");
  }
  {
    /* 70 sequences: two launch groups */
    int32_t t0[70], t1[70];
    for (int b = 0; b < 70; ++b) {
      t0[b] = (int32_t)lcg_below(40);
      t1[b] = t0[b] + (int32_t)lcg_below(60);
    }
    case_stream(st, DV_DENSE, 2, 2, 128, 70, 100, 0, 2, t0, t1, 13, "dense, 70 sequences");
  }
  case_paged(st);
  {
    const int32_t t0[4] = {100, 0, 5, 519};
    const int32_t t1[4] = {101, 1, 6, 520};
    case_swap(st, t0, t1, "swap of one-token rows (kernel engine)");
  }
  {
    const int32_t t0[4] = {0, 0, 8, 0};
    const int32_t t1[4] = {512, 300, 520, 0};
    case_swap(st, t0, t1, "swap of long rows (DMA engine)");
  }
  case_scheduler(st);
  HIPCHECK(hipStreamDestroy(st));
  printf("abi parity ok: %d cases\n", cases);
  return 0;
}
