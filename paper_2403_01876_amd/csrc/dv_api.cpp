// C-ABI entry points: host-side validation, sizing and kernel/DMA dispatch.
// Everything is checked before the first enqueue, so an error return leaves
// the streams and all memory untouched.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "../../include/dv.h"
#include "dv_host.h"
#include "dv_internal.h"

namespace {

using dv::kSeqPerLaunch;

// Swaps whose rows (one sequence's tokens of one head) are narrower than
// this go through the copy kernel instead of DMA.  Measured on MI355X for
// the OPT-66B stage: a one-token update (256-byte rows) took 162 us by one
// 2-D DMA and 2.5 ms by per-sequence DMA with ragged positions, against
// about 100 us by kernel; rows of whole prompts move faster by DMA
// (57 GB/s against 54 GB/s).
constexpr int64_t kNarrowRowBytes = 64 * 1024;

// Streams whose longest (sequence, head) run has at most this many 16-byte
// units use the flattened short-run kernel; longer runs use the tiled
// kernels, whose 512-unit tiles would otherwise leave most lanes idle.
constexpr int64_t kSmallRunUnits = 256;

// A validated view of one microbatch of a cache, sizes in 16-byte units.
struct View {
  int kind;
  int mem;
  int64_t L, H, D, B, E;
  int64_t du;        // units per token
  int64_t cap;       // token capacity per sequence
  int64_t S;         // dense kinds: max_seq
  int64_t bs, NB, max_blocks;
  char* base;
  const int32_t* bt;
  int32_t* owner;    // paged: optional owner-map workspace [NB]
  uint64_t bytes;    // storage bytes of the microbatch
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// The layout of a descriptor, without a microbatch (sizing calls).
int layout_of(const dv_cache* c, View* v) {
  if (!c || !c->mb_base) return DV_ERR_INVALID;
  if (c->elem_bytes <= 0 || c->num_layers <= 0 || c->num_heads <= 0 || c->head_dim <= 0 ||
      c->batch <= 0 || c->num_mb <= 0)
    return DV_ERR_INVALID;
  if (((int64_t)c->head_dim * c->elem_bytes) % 16 != 0) return DV_ERR_INVALID;
  if (c->mem != DV_MEM_DEVICE && c->mem != DV_MEM_HOST_PINNED) return DV_ERR_INVALID;
  v->kind = c->kind;
  v->mem = c->mem;
  v->L = c->num_layers;
  v->H = c->num_heads;
  v->D = c->head_dim;
  v->B = c->batch;
  v->E = c->elem_bytes;
  v->du = v->D * v->E / 16;
  v->S = v->bs = v->NB = v->max_blocks = 0;
  v->bt = nullptr;
  v->owner = nullptr;
  if (c->kind == DV_DENSE || c->kind == DV_DENSE_KSPLIT) {
    if (c->max_seq <= 0) return DV_ERR_INVALID;
    v->S = v->cap = c->max_seq;
    v->bytes = (uint64_t)v->L * 2 * v->B * v->H * v->S * v->du * 16;
  } else if (c->kind == DV_PAGED) {
    if (c->block_size <= 0 || c->num_blocks <= 0 || c->max_blocks <= 0 || !c->block_table)
      return DV_ERR_INVALID;
    v->bs = c->block_size;
    v->NB = c->num_blocks;
    v->max_blocks = c->max_blocks;
    v->cap = v->bs * v->max_blocks;
    v->bytes = (uint64_t)v->L * 2 * v->NB * v->H * v->bs * v->du * 16;
  } else {
    return DV_ERR_INVALID;
  }
  // Extents whose products the kernels take in 32-bit arithmetic (a launch's
  // first slab index, 2 * layer + 1, among them).
  if (v->L > (1 << 24) || v->cap > (1 << 24) || v->du > (1 << 16) || v->H * v->du > (1 << 20) ||
      v->cap * v->du > (1ll << 30))
    return DV_ERR_UNSUPPORTED;
  // The paged kernel flattens (head pair, unit) over two heads of one block:
  // 2 * block_size * du units must stay well inside int32.
  if (c->kind == DV_PAGED && v->bs * v->du > (1ll << 29)) return DV_ERR_UNSUPPORTED;
  // Every byte count derived from the descriptor stays far inside 64 bits:
  // its storage and the longest stream it can produce (all layers, every
  // sequence at full capacity) must be below 2^48 bytes.
  using u128 = unsigned __int128;
  const u128 per_token = (u128)v->L * 2 * v->H * v->du * 16;
  const u128 rows = c->kind == DV_PAGED ? (u128)v->NB * v->bs : (u128)v->B * v->S;
  const u128 limit = (u128)1 << 48;
  if (per_token * rows >= limit || per_token * v->B * v->cap >= limit) return DV_ERR_UNSUPPORTED;
  v->base = nullptr;
  return DV_OK;
}

// The layout plus microbatch mb's base address (and table, owner map).
int view_of(const dv_cache* c, int32_t mb, View* v) {
  const int rc = layout_of(c, v);
  if (rc != DV_OK) return rc;
  if (mb < 0 || mb >= c->num_mb) return DV_ERR_RANGE;
  v->base = static_cast<char*>(c->mb_base[mb]);
  if (!v->base || !aligned16(v->base)) return DV_ERR_INVALID;
  if (c->kind == DV_PAGED) {
    v->bt = c->block_table[mb];
    if (!v->bt) return DV_ERR_INVALID;
    v->owner = c->block_owner ? c->block_owner[mb] : nullptr;
    if ((reinterpret_cast<uintptr_t>(v->owner) & 3u) != 0) return DV_ERR_INVALID;
  }
  return DV_OK;
}

// Checks the ranges and returns the per-sequence (t0, n) and N.
int ranges_of(const View& v, int32_t l0, int32_t l1, const int32_t* t0, const int32_t* t1,
              std::vector<int32_t>* r0, std::vector<int32_t>* rn, int64_t* N) {
  if (!t1) return DV_ERR_INVALID;
  if (l0 < 0 || l1 < l0 || l1 > v.L) return DV_ERR_RANGE;
  r0->resize(v.B);
  rn->resize(v.B);
  int64_t total = 0;
  for (int64_t b = 0; b < v.B; ++b) {
    const int64_t a = t0 ? t0[b] : 0, e = t1[b];
    if (a < 0 || e < a || e > v.cap) return DV_ERR_RANGE;
    (*r0)[b] = (int32_t)a;
    (*rn)[b] = (int32_t)(e - a);
    total += e - a;
  }
  *N = total;
  return DV_OK;
}

uint64_t wire_bytes(const View& v, int32_t l0, int32_t l1, int64_t N) {
  return (uint64_t)(l1 - l0) * 2 * v.H * v.du * 16 * (uint64_t)N;
}

bool overlaps(const void* a, uint64_t na, const void* b, uint64_t nb) {
  if (na == 0 || nb == 0) return false;
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

// DV_ERR_HIP for a failed runtime call; with DV_DEBUG set in the environment
// the runtime's error name is also printed to stderr.
int hip_fail(hipError_t e, const char* what) {
  if (e == hipSuccess) return DV_OK;
  static const bool debug = getenv("DV_DEBUG") != nullptr;
  if (debug) fprintf(stderr, "libdv: %s failed: %s\n", what, hipGetErrorName(e));
  return DV_ERR_HIP;
}

int hip_status(hipError_t e) { return hip_fail(e, "hipMemcpy2DAsync"); }

// Whether [p, p + n) overlaps a paged view's block table, which the kernels
// read while the call writes: the table must stay out of everything written.
bool overlaps_table(const View& v, const void* p, uint64_t n) {
  return v.bt && overlaps(p, n, v.bt, (uint64_t)v.B * v.max_blocks * 4);
}

// Whether a paged stream-in with an owner-map workspace scatters in pool
// order: at most kPoolSeqMax sequences (their ranges travel in the launch's
// arguments), at least five ninths of the pool's blocks written, and every
// count inside the kernels' 32-bit arithmetic.  Pool order launches a
// workgroup for every block, and one that finds nothing to write still costs
// its launch and owner lookup: on MI355X, for the LLaMA-2-70B pool, pool
// order lost 4 % to table order with 47 % of the blocks written and 1 % with
// 52 %, broke even near 54 % and won 1.5 % at 57 %, 3 % at 62 % and 7 % at
// 95 %.
bool pool_order_applies(const View& v, const std::vector<int32_t>& t0,
                        const std::vector<int32_t>& n, int64_t N) {
  const int64_t ngrp = (v.H + dv::kPagedHeads - 1) / dv::kPagedHeads;
  if (v.B > dv::kPoolSeqMax || N >= (1ll << 31) || v.NB * ngrp >= (1ll << 31) ||
      v.B * v.max_blocks >= (1ll << 31))
    return false;
  int64_t tiles = 0;
  for (int64_t b = 0; b < v.B; ++b)
    if (n[b] > 0) tiles += ((t0[b] + n[b] + v.bs - 1) / v.bs - t0[b] / v.bs) * ngrp;
  return 9 * tiles >= 5 * v.NB * ngrp;
}

// Paged stream-in in pool order for more than 64 sequences: the owner map
// of the whole call (one clearing launch, one building launch per group of
// 64 sequences), then one launch over every (slab, pool block, head pair).
int pool_order_stream_in(const View& v, int32_t l0, int32_t l1, const std::vector<int32_t>& t0,
                         const std::vector<int32_t>& n, int64_t N, void* wire, hipStream_t st) {
  dv::OwnerArgs o;
  memset(&o, 0, sizeof o);
  o.owner = v.owner;
  o.bt = v.bt;
  o.block_size = (int32_t)v.bs;
  o.num_blocks = (int32_t)v.NB;
  o.max_blocks = (int32_t)v.max_blocks;
  hipError_t e = dv::launch_owner_clear(o, st);
  if (e != hipSuccess) return hip_fail(e, "owner map launch");
  for (int64_t g0 = 0; g0 < v.B; g0 += kSeqPerLaunch) {
    o.nseq = (int32_t)std::min<int64_t>(kSeqPerLaunch, v.B - g0);
    o.b0 = (int32_t)g0;
    memset(&o.r, 0, sizeof o.r);
    bool any = false;
    for (int i = 0; i < o.nseq; ++i) {
      o.r.t0[i] = t0[g0 + i];
      o.r.n[i] = n[g0 + i];
      any = any || n[g0 + i] > 0;
    }
    if (!any) continue;
    e = dv::launch_owner_build(o, st);
    if (e != hipSuccess) return hip_fail(e, "owner map launch");
  }
  dv::PoolOrderArgs a;
  memset(&a, 0, sizeof a);
  a.pool = v.base;
  a.wire = wire;
  a.owner = v.owner;
  a.s_slab = v.NB * v.H * v.bs * v.du;
  a.s_blk = v.H * v.bs * v.du;
  a.s_h = v.bs * v.du;
  a.m = {2 * l0, 1, 0, 0, N * v.H * v.du};
  a.du = (int32_t)v.du;
  a.heads = (int32_t)v.H;
  a.nseq = (int32_t)v.B;
  a.max_blocks = (int32_t)v.max_blocks;
  a.block_size = (int32_t)v.bs;
  a.num_blocks = (int32_t)v.NB;
  int64_t p = 0;
  for (int64_t b = 0; b < v.B; ++b) {
    a.t0[b] = t0[b];
    a.n[b] = n[b];
    a.p[b] = (int32_t)p;  // below 2^31: N is
    p += n[b];
  }
  const int64_t ngrp = (v.H + dv::kPagedHeads - 1) / dv::kPagedHeads;
  e = dv::launch_paged_pool_order(a, (uint32_t)(v.NB * ngrp), 2 * (uint32_t)(l1 - l0), st);
  return hip_fail(e, "paged pool-order launch");
}

// Enqueue the pack (dir = kPack) or unpack of the validated ranges.  The wire
// is at `wire`; per (layer, K|V) slab it holds N*H*du units.
int run_stream(int dir, const View& v, int32_t l0, int32_t l1, const std::vector<int32_t>& t0,
               const std::vector<int32_t>& n, int64_t N, void* wire, hipStream_t st) {
  if (N == 0 || l1 == l0) return DV_OK;
  const int64_t w_slab = N * v.H * v.du;
  const uint32_t nl = (uint32_t)(l1 - l0);
  int32_t max_n = 0;
  for (int32_t x : n) max_n = std::max(max_n, x);
  const bool single = max_n <= 1;
  // Runs of at most kSmallRunUnits units per (sequence, head) go through the
  // flattened short-run kernel instead of the tiled ones.
  const bool small = !single && (int64_t)max_n * v.du <= kSmallRunUnits;

  // Every launch group's grid, checked before anything is enqueued so that a
  // refusal leaves the stream untouched.  Single tokens need no check: at
  // most 64 * heads * du < 2^26 units per launch.
  if (!single) {
    const int64_t ngrp = (v.H + dv::kPagedHeads - 1) / dv::kPagedHeads;
    for (int64_t g0 = 0; g0 < v.B; g0 += kSeqPerLaunch) {
      const int64_t g1 = std::min<int64_t>(g0 + kSeqPerLaunch, v.B);
      int64_t grid = 0, ktiles = 0;
      for (int64_t b = g0; b < g1; ++b) {
        const int64_t a = t0[b], k = n[b];
        if (k == 0) continue;
        if (small)
          grid += k * v.H * v.du;
        else if (v.kind == DV_PAGED)
          grid += ((a + k + v.bs - 1) / v.bs - a / v.bs) * ngrp;
        else
          grid += v.H * ((k * v.du + dv::kDenseTile - 1) / dv::kDenseTile);
        ktiles += v.H * ((k + dv::kKsplitTile - 1) / dv::kKsplitTile);
      }
      if (!small && v.kind == DV_DENSE_KSPLIT) grid = std::max(grid, ktiles);
      if (grid >= (1ll << 31)) return DV_ERR_UNSUPPORTED;
    }
  }

  // Paged stream-in in pool order: up to 64 sequences through paged_kernel
  // in the loop below, more through one launch over the whole call.
  const bool pool_order = dir == dv::kUnpack && v.kind == DV_PAGED && !single && !small &&
                          v.owner && pool_order_applies(v, t0, n, N);
  if (pool_order && v.B > kSeqPerLaunch) return pool_order_stream_in(v, l0, l1, t0, n, N, wire, st);

  int64_t p_group = 0;  // tokens of all earlier launch groups
  for (int64_t g0 = 0; g0 < v.B; g0 += kSeqPerLaunch) {
    const int nseq = (int)std::min<int64_t>(kSeqPerLaunch, v.B - g0);
    int64_t ntok = 0;
    for (int i = 0; i < nseq; ++i) ntok += n[g0 + i];
    if (ntok == 0) continue;
    char* wire_g = static_cast<char*>(wire) + (uint64_t)p_group * v.H * v.du * 16;
    p_group += ntok;

    dv::SeqRanges r;
    memset(&r, 0, sizeof r);
    for (int i = 0; i < nseq; ++i) {
      r.t0[i] = t0[g0 + i];
      r.n[i] = n[g0 + i];
    }

    if (single) {
      dv::TokenArgs a;
      memset(&a, 0, sizeof a);
      a.cache = v.base;
      a.wire = wire_g;
      a.bt = v.bt;
      a.du = (int32_t)v.du;
      a.heads = (int32_t)v.H;
      a.nseq = nseq;
      a.b0 = (int32_t)g0;
      for (int i = 0; i < kSeqPerLaunch; ++i) a.pos[i] = (i < nseq && r.n[i] == 1) ? r.t0[i] : -1;
      const uint32_t units = (uint32_t)(ntok * v.H * v.du);
      hipError_t e;
      if (v.kind == DV_PAGED) {
        a.paged = 1;
        a.block_size = (int32_t)v.bs;
        a.num_blocks = (int32_t)v.NB;
        a.max_blocks = (int32_t)v.max_blocks;
        a.s_slab = v.NB * v.H * v.bs * v.du;
        a.s_blk = v.H * v.bs * v.du;
        a.s_h = v.bs * v.du;
        a.s_tok = v.du;
        a.s_e = 1;
        a.m = {2 * l0, 1, 0, 0, w_slab};
        e = dv::launch_token(dir, a, units, 2 * nl, st);
      } else {
        a.s_slab = v.B * v.H * v.S * v.du;
        a.s_b = v.H * v.S * v.du;
        a.s_h = v.S * v.du;
        if (v.kind == DV_DENSE) {
          a.s_tok = v.du;
          a.s_e = 1;
          a.m = {2 * l0, 1, 0, 0, w_slab};
          e = dv::launch_token(dir, a, units, 2 * nl, st);
        } else {
          // split key slabs: groups S units apart, tokens 1 unit apart
          a.s_tok = 1;
          a.s_e = v.S;
          a.m = {2 * l0, 2, 0, 0, w_slab};
          e = dv::launch_token(dir, a, units, nl, st);
          if (e == hipSuccess) {
            a.s_tok = v.du;
            a.s_e = 1;
            a.m = {2 * l0 + 1, 2, 1, 0, w_slab};
            e = dv::launch_token(dir, a, units, nl, st);
          }
        }
      }
      if (e != hipSuccess) return hip_fail(e, "token kernel launch");
      continue;
    }

    if (small) {
      dv::SmallRunArgs a;
      memset(&a, 0, sizeof a);
      a.cache = v.base;
      a.wire = wire_g;
      a.bt = v.bt;
      a.du = (int32_t)v.du;
      a.heads = (int32_t)v.H;
      a.nseq = nseq;
      a.b0 = (int32_t)g0;
      a.r = r;
      const int64_t units = ntok * v.H * v.du;  // below 2^31: checked above
      hipError_t e;
      if (v.kind == DV_PAGED) {
        a.paged = 1;
        a.block_size = (int32_t)v.bs;
        a.num_blocks = (int32_t)v.NB;
        a.max_blocks = (int32_t)v.max_blocks;
        a.s_slab = v.NB * v.H * v.bs * v.du;
        a.s_blk = v.H * v.bs * v.du;
        a.s_h = v.bs * v.du;
        a.s_tok = v.du;
        a.s_e = 1;
        a.m = {2 * l0, 1, 0, 0, w_slab};
        e = dv::launch_small_runs(dir, a, (uint32_t)units, 2 * nl, st);
      } else {
        a.s_slab = v.B * v.H * v.S * v.du;
        a.s_b = v.H * v.S * v.du;
        a.s_h = v.S * v.du;
        if (v.kind == DV_DENSE) {
          a.s_tok = v.du;
          a.s_e = 1;
          a.m = {2 * l0, 1, 0, 0, w_slab};
          e = dv::launch_small_runs(dir, a, (uint32_t)units, 2 * nl, st);
        } else {
          // split key slabs: groups S units apart, tokens 1 unit apart
          a.s_tok = 1;
          a.s_e = v.S;
          a.m = {2 * l0, 2, 0, 0, w_slab};
          e = dv::launch_small_runs(dir, a, (uint32_t)units, nl, st);
          if (e == hipSuccess) {
            a.s_tok = v.du;
            a.s_e = 1;
            a.m = {2 * l0 + 1, 2, 1, 0, w_slab};
            e = dv::launch_small_runs(dir, a, (uint32_t)units, nl, st);
          }
        }
      }
      if (e != hipSuccess) return hip_fail(e, "short-run kernel launch");
      continue;
    }

    if (v.kind == DV_PAGED) {
      dv::PagedArgs a;
      memset(&a, 0, sizeof a);
      a.pool = v.base;
      a.wire = wire_g;
      a.bt = v.bt;
      a.s_slab = v.NB * v.H * v.bs * v.du;
      a.s_blk = v.H * v.bs * v.du;
      a.s_h = v.bs * v.du;
      a.m = {2 * l0, 1, 0, 0, w_slab};
      a.du = (int32_t)v.du;
      a.heads = (int32_t)v.H;
      a.nseq = nseq;
      a.b0 = (int32_t)g0;
      a.block_size = (int32_t)v.bs;
      a.num_blocks = (int32_t)v.NB;
      a.max_blocks = (int32_t)v.max_blocks;
      a.r = r;
      const int64_t ngrp = (v.H + dv::kPagedHeads - 1) / dv::kPagedHeads;
      int64_t tiles = 0;
      for (int i = 0; i < nseq; ++i)
        if (r.n[i] > 0) tiles += ((r.t0[i] + r.n[i] + v.bs - 1) / v.bs - r.t0[i] / v.bs) * ngrp;
      if (pool_order) {  // all sequences in this one group
        dv::OwnerArgs o;
        memset(&o, 0, sizeof o);
        o.owner = v.owner;
        o.bt = v.bt;
        o.nseq = nseq;
        o.block_size = (int32_t)v.bs;
        o.num_blocks = (int32_t)v.NB;
        o.max_blocks = (int32_t)v.max_blocks;
        o.r = r;
        hipError_t e = dv::launch_owner_clear(o, st);
        if (e == hipSuccess) e = dv::launch_owner_build(o, st);
        if (e != hipSuccess) return hip_fail(e, "owner map launch");
        a.owner = v.owner;
        tiles = v.NB * ngrp;  // below 2^31: checked by pool_order_applies
      }
      const hipError_t e = dv::launch_paged(dir, a, (uint32_t)tiles, 2 * nl, st);
      if (e != hipSuccess) return hip_fail(e, "paged kernel launch");
      continue;
    }

    dv::DenseRunArgs a;
    memset(&a, 0, sizeof a);
    a.cache = v.base;
    a.wire = wire_g;
    a.s_slab = v.B * v.H * v.S * v.du;
    a.s_b = v.H * v.S * v.du;
    a.s_h = v.S * v.du;
    a.du = (int32_t)v.du;
    a.heads = (int32_t)v.H;
    a.nseq = nseq;
    a.b0 = (int32_t)g0;
    a.r = r;
    int64_t tiles = 0;
    for (int i = 0; i < nseq; ++i)
      tiles += v.H * (((int64_t)r.n[i] * v.du + dv::kDenseTile - 1) / dv::kDenseTile);
    if (v.kind == DV_DENSE) {
      a.m = {2 * l0, 1, 0, 0, w_slab};
      const hipError_t e = dv::launch_dense_runs(dir, a, (uint32_t)tiles, 2 * nl, st);
      if (e != hipSuccess) return hip_fail(e, "dense kernel launch");
      continue;
    }
    // split key: value slabs are dense runs, key slabs go through LDS
    a.m = {2 * l0 + 1, 2, 1, 0, w_slab};
    hipError_t e = dv::launch_dense_runs(dir, a, (uint32_t)tiles, nl, st);
    if (e != hipSuccess) return hip_fail(e, "dense kernel launch");
    dv::KsplitArgs k;
    memset(&k, 0, sizeof k);
    k.cache = v.base;
    k.wire = wire_g;
    k.s_slab = a.s_slab;
    k.s_b = a.s_b;
    k.s_h = a.s_h;
    k.m = {2 * l0, 2, 0, 0, w_slab};
    k.du = (int32_t)v.du;
    k.heads = (int32_t)v.H;
    k.nseq = nseq;
    k.b0 = (int32_t)g0;
    k.seq_cap = (int32_t)v.S;
    k.r = r;
    int64_t ktiles = 0;
    for (int i = 0; i < nseq; ++i)
      ktiles += v.H * (((int64_t)r.n[i] + dv::kKsplitTile - 1) / dv::kKsplitTile);
    e = dv::launch_ksplit(dir, k, (uint32_t)ktiles, nl, st);
    if (e != hipSuccess) return hip_fail(e, "split-key kernel launch");
  }
  return DV_OK;
}

int check_kind_supported(const View& v) {
  if (v.kind == DV_DENSE_KSPLIT && (16 % v.E != 0 || v.du > dv::kKsplitMaxDu))
    return DV_ERR_UNSUPPORTED;
  return DV_OK;
}

int stream_out(const dv_cache* src, int32_t mb, int32_t l0, int32_t l1, const int32_t* t0,
               const int32_t* t1, void* dst, uint64_t dst_cap, uint64_t* out_bytes,
               void* stream) {
  View v;
  int rc = view_of(src, mb, &v);
  if (rc != DV_OK) return rc;
  std::vector<int32_t> r0, rn;
  int64_t N = 0;
  rc = ranges_of(v, l0, l1, t0, t1, &r0, &rn, &N);
  if (rc != DV_OK) return rc;
  const uint64_t need = wire_bytes(v, l0, l1, N);
  if (out_bytes) *out_bytes = need;
  if (need > dst_cap) return DV_ERR_SPACE;
  if (need == 0) return DV_OK;
  if (!dst || !aligned16(dst)) return DV_ERR_INVALID;
  if (overlaps(dst, need, v.base, v.bytes) || overlaps_table(v, dst, need))
    return DV_ERR_INVALID;
  rc = check_kind_supported(v);
  if (rc != DV_OK) return rc;
  return run_stream(dv::kPack, v, l0, l1, r0, rn, N, dst, static_cast<hipStream_t>(stream));
}

// Copy rows of the validated ranges between two dense caches with DMA.
int swap_copy(const dv_cache* from, int32_t from_mb, const dv_cache* to, int32_t to_mb,
              int32_t l0, int32_t l1, const int32_t* t0, const int32_t* t1, void* stream,
              int from_mem, int to_mem) {
  View a, b;
  int rc = view_of(from, from_mb, &a);
  if (rc != DV_OK) return rc;
  rc = view_of(to, to_mb, &b);
  if (rc != DV_OK) return rc;
  if (a.kind != DV_DENSE || b.kind != DV_DENSE) return DV_ERR_UNSUPPORTED;
  if (a.L != b.L || a.H != b.H || a.D != b.D || a.B != b.B || a.E != b.E) return DV_ERR_INVALID;
  if (a.mem != from_mem || b.mem != to_mem) return DV_ERR_INVALID;
  std::vector<int32_t> r0, rn;
  int64_t N = 0;
  rc = ranges_of(a, l0, l1, t0, t1, &r0, &rn, &N);
  if (rc != DV_OK) return rc;
  for (int64_t i = 0; i < b.B; ++i)
    if ((int64_t)r0[i] + rn[i] > b.cap) return DV_ERR_RANGE;
  if (overlaps(a.base, a.bytes, b.base, b.bytes)) return DV_ERR_INVALID;
  if (N == 0 || l1 == l0) return DV_OK;

  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t max_n = 0;
  for (int32_t x : rn) max_n = std::max(max_n, x);
  if ((int64_t)max_n * a.du * 16 < kNarrowRowBytes) {
    // Narrow rows (a decode step's update): one kernel copies them straight
    // between the slot and the pinned mirror; DMA would take one descriptor
    // per row (or one call per row block when the ranges are ragged).
    // Every launch group's grid is checked before anything is enqueued.
    for (int64_t g0 = 0; g0 < a.B; g0 += kSeqPerLaunch) {
      int64_t units = 0;
      for (int64_t b = g0; b < std::min<int64_t>(g0 + kSeqPerLaunch, a.B); ++b)
        units += (int64_t)rn[b] * a.H * a.du;
      if (units >= (1ll << 31)) return DV_ERR_UNSUPPORTED;
    }
    const uint32_t nl = (uint32_t)(l1 - l0);
    for (int64_t g0 = 0; g0 < a.B; g0 += kSeqPerLaunch) {
      const int nseq = (int)std::min<int64_t>(kSeqPerLaunch, a.B - g0);
      dv::CopyArgs k;
      memset(&k, 0, sizeof k);
      int64_t units = 0;
      for (int i = 0; i < nseq; ++i) {
        k.r.t0[i] = r0[g0 + i];
        k.r.n[i] = rn[g0 + i];
        units += (int64_t)rn[g0 + i] * a.H * a.du;
      }
      if (units == 0) continue;
      k.src = a.base;
      k.dst = b.base;
      k.s_slab = a.B * a.H * a.S * a.du;
      k.s_b = a.H * a.S * a.du;
      k.s_h = a.S * a.du;
      k.d_slab = b.B * b.H * b.S * b.du;
      k.d_b = b.H * b.S * b.du;
      k.d_h = b.S * b.du;
      k.slab0 = 2 * l0;
      k.du = (int32_t)a.du;
      k.heads = (int32_t)a.H;
      k.nseq = nseq;
      k.b0 = (int32_t)g0;
      const hipError_t e = dv::launch_copy(k, (uint32_t)units, 2 * nl, st);
      if (e != hipSuccess) return hip_fail(e, "copy kernel launch");
    }
    return DV_OK;
  }

  const hipMemcpyKind kind =
      from_mem == DV_MEM_DEVICE ? hipMemcpyDeviceToHost : hipMemcpyHostToDevice;
  const size_t tok = (size_t)a.du * 16;
  const size_t ap = (size_t)a.S * tok, bp = (size_t)b.S * tok;  // row pitches
  bool uniform = true;
  for (int64_t i = 1; i < a.B; ++i)
    if (r0[i] != r0[0] || rn[i] != rn[0]) uniform = false;
  if (uniform) {
    // Rows (slab, b, h) of the layer range are consecutive at one pitch.
    const size_t row0 = (size_t)2 * l0 * a.B * a.H;
    const size_t rows = (size_t)2 * (l1 - l0) * a.B * a.H;
    return hip_status(hipMemcpy2DAsync(b.base + row0 * bp + r0[0] * tok, bp,
                                       a.base + row0 * ap + r0[0] * tok, ap, rn[0] * tok, rows,
                                       kind, st));
  }
  for (int64_t slab = 2 * l0; slab < 2 * l1; ++slab) {
    for (int64_t s = 0; s < a.B; ++s) {
      if (rn[s] == 0) continue;
      const size_t row0 = (size_t)(slab * a.B + s) * a.H;
      hipError_t e = hipMemcpy2DAsync(b.base + row0 * bp + r0[s] * tok, bp,
                                      a.base + row0 * ap + r0[s] * tok, ap, rn[s] * tok,
                                      (size_t)a.H, kind, st);
      if (e != hipSuccess) return hip_fail(e, "hipMemcpy2DAsync");
    }
  }
  return DV_OK;
}

}  // namespace

namespace dv {

hipError_t create_side_streams(hipStream_t* shared_queue, hipStream_t* own_queue) {
  *shared_queue = *own_queue = nullptr;
  hipError_t e = hipStreamCreateWithFlags(shared_queue, hipStreamNonBlocking);
  if (e != hipSuccess) return e;
  int device = 0, cus = 0;
  e = hipGetDevice(&device);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
  if (e != hipSuccess || cus <= 0) return e != hipSuccess ? e : hipErrorInvalidDevice;
  std::vector<uint32_t> mask((cus + 31) / 32, 0xffffffffu);  // every CU
  if (cus % 32) mask.back() = (1u << (cus % 32)) - 1u;
  return hipExtStreamCreateWithCUMask(own_queue, (uint32_t)mask.size(), mask.data());
}

}  // namespace dv

extern "C" {

int dv_api_version(void) { return DV_API_VERSION; }

const char* dv_status_string(int status) {
  switch (status) {
    case DV_OK: return "ok";
    case DV_ERR_INVALID: return "invalid argument";
    case DV_ERR_RANGE: return "range outside the cache";
    case DV_ERR_SPACE: return "buffer too small";
    case DV_ERR_UNSUPPORTED: return "unsupported layout or size";
    case DV_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int dv_cache_bytes(const dv_cache* c, uint64_t* out_bytes) {
  View v;
  int rc = layout_of(c, &v);
  if (rc != DV_OK) return rc;
  if (out_bytes) *out_bytes = v.bytes;
  return DV_OK;
}

int dv_packed_bytes(const dv_cache* c, int32_t l0, int32_t l1, const int32_t* t0,
                    const int32_t* t1, uint64_t* out_bytes) {
  View v;
  int rc = layout_of(c, &v);
  if (rc != DV_OK) return rc;
  std::vector<int32_t> r0, rn;
  int64_t N = 0;
  rc = ranges_of(v, l0, l1, t0, t1, &r0, &rn, &N);
  if (rc != DV_OK) return rc;
  if (out_bytes) *out_bytes = wire_bytes(v, l0, l1, N);
  return DV_OK;
}

int dv_stream_out_prompt(const dv_cache* src, int32_t mb, int32_t l0, int32_t l1,
                         const int32_t* t0, const int32_t* t1, void* dst, uint64_t dst_cap,
                         uint64_t* out_bytes, void* stream) {
  return stream_out(src, mb, l0, l1, t0, t1, dst, dst_cap, out_bytes, stream);
}

int dv_stream_out_token(const dv_cache* src, int32_t mb, int32_t l0, int32_t l1,
                        const int32_t* pos, void* dst, uint64_t dst_cap, uint64_t* out_bytes,
                        void* stream) {
  if (!src || !pos || src->batch <= 0) return DV_ERR_INVALID;
  std::vector<int32_t> a(src->batch), e(src->batch);
  for (int32_t b = 0; b < src->batch; ++b) {
    if (pos[b] == INT32_MAX) return DV_ERR_RANGE;  // before pos + 1 is formed
    a[b] = pos[b] < 0 ? 0 : pos[b];
    e[b] = pos[b] < 0 ? 0 : pos[b] + 1;
  }
  return stream_out(src, mb, l0, l1, a.data(), e.data(), dst, dst_cap, out_bytes, stream);
}

}  // extern "C"

namespace dv {
int noalloc_owner_map(hipStream_t stream, int32_t** out);  // dv_noalloc.hip
}  // namespace dv

namespace {

// dv_stream_in, and with `noalloc` dv_stream_in_noalloc: a paged receiver's
// owner map then lives in the library's static per-device array instead of
// the caller's workspace.
int stream_in(const dv_cache* dst, int32_t mb, int32_t l0, int32_t l1, const int32_t* t0,
              const int32_t* t1, const void* src, uint64_t src_bytes, void* stream,
              bool noalloc) {
  dv_cache own;
  if (noalloc && dst) {
    own = *dst;
    own.block_owner = nullptr;  // the caller's workspace, if any, is ignored
    dst = &own;
  }
  View v;
  int rc = view_of(dst, mb, &v);
  if (rc != DV_OK) return rc;
  if (noalloc && v.kind == DV_PAGED && v.NB > DV_NOALLOC_MAX_BLOCKS) return DV_ERR_UNSUPPORTED;
  std::vector<int32_t> r0, rn;
  int64_t N = 0;
  rc = ranges_of(v, l0, l1, t0, t1, &r0, &rn, &N);
  if (rc != DV_OK) return rc;
  const uint64_t need = wire_bytes(v, l0, l1, N);
  if (src_bytes < need) return DV_ERR_SPACE;
  if (need == 0) return DV_OK;
  if (!src || !aligned16(src)) return DV_ERR_INVALID;
  if (overlaps(src, need, v.base, v.bytes) || overlaps_table(v, v.base, v.bytes))
    return DV_ERR_INVALID;
  if (v.owner && (overlaps(v.owner, (uint64_t)v.NB * 4, v.base, v.bytes) ||
                  overlaps(v.owner, (uint64_t)v.NB * 4, src, need) ||
                  overlaps_table(v, v.owner, (uint64_t)v.NB * 4)))
    return DV_ERR_INVALID;
  rc = check_kind_supported(v);
  if (rc != DV_OK) return rc;
  if (noalloc && v.kind == DV_PAGED) {
    rc = dv::noalloc_owner_map(static_cast<hipStream_t>(stream), &v.owner);
    if (rc != DV_OK) return rc;
  }
  return run_stream(dv::kUnpack, v, l0, l1, r0, rn, N, const_cast<void*>(src),
                    static_cast<hipStream_t>(stream));
}

}  // namespace

extern "C" {

int dv_stream_in(const dv_cache* dst, int32_t mb, int32_t l0, int32_t l1, const int32_t* t0,
                 const int32_t* t1, const void* src, uint64_t src_bytes, void* stream) {
  return stream_in(dst, mb, l0, l1, t0, t1, src, src_bytes, stream, false);
}

int dv_stream_in_noalloc(const dv_cache* dst, int32_t mb, int32_t l0, int32_t l1,
                         const int32_t* t0, const int32_t* t1, const void* src,
                         uint64_t src_bytes, void* stream) {
  return stream_in(dst, mb, l0, l1, t0, t1, src, src_bytes, stream, true);
}

int dv_block_claims(const dv_cache* c, int32_t mb, const int32_t* t0, const int32_t* t1,
                    int32_t* counts, void* stream) {
  View v;
  int rc = view_of(c, mb, &v);
  if (rc != DV_OK) return rc;
  if (v.kind != DV_PAGED) return DV_ERR_UNSUPPORTED;
  std::vector<int32_t> r0, rn;
  int64_t N = 0;
  rc = ranges_of(v, 0, (int32_t)v.L, t0, t1, &r0, &rn, &N);
  if (rc != DV_OK) return rc;
  if (!counts || (reinterpret_cast<uintptr_t>(counts) & 3u) != 0) return DV_ERR_INVALID;
  if (overlaps(counts, (uint64_t)v.NB * 4, v.base, v.bytes) ||
      overlaps_table(v, counts, (uint64_t)v.NB * 4))
    return DV_ERR_INVALID;
  hipStream_t st = static_cast<hipStream_t>(stream);
  for (int64_t g0 = 0; g0 < v.B; g0 += kSeqPerLaunch) {
    const int nseq = (int)std::min<int64_t>(kSeqPerLaunch, v.B - g0);
    dv::OwnerArgs o;
    memset(&o, 0, sizeof o);
    o.owner = counts;
    o.bt = v.bt;
    o.nseq = nseq;
    o.block_size = (int32_t)v.bs;
    o.num_blocks = (int32_t)v.NB;
    o.max_blocks = (int32_t)v.max_blocks;
    o.b0 = (int32_t)g0;
    for (int i = 0; i < nseq; ++i) {
      o.r.t0[i] = r0[g0 + i];
      o.r.n[i] = rn[g0 + i];
    }
    const hipError_t e = dv::launch_block_claims(o, g0 == 0, st);
    if (e != hipSuccess) return hip_fail(e, "block claims launch");
  }
  return DV_OK;
}

int dv_swap_out(const dv_cache* dev, int32_t slot, const dv_cache* host, int32_t host_mb,
                int32_t l0, int32_t l1, const int32_t* t0, const int32_t* t1, void* stream) {
  return swap_copy(dev, slot, host, host_mb, l0, l1, t0, t1, stream, DV_MEM_DEVICE,
                   DV_MEM_HOST_PINNED);
}

int dv_swap_in(const dv_cache* host, int32_t host_mb, const dv_cache* dev, int32_t slot,
               int32_t l0, int32_t l1, const int32_t* t0, const int32_t* t1, void* stream) {
  return swap_copy(host, host_mb, dev, slot, l0, l1, t0, t1, stream, DV_MEM_HOST_PINNED,
                   DV_MEM_DEVICE);
}

}  // extern "C"
