// Pack / unpack kernels for gfx950.  Pure data movement: every lane moves
// 16-byte words with nontemporal global loads and stores (the data is
// streamed once, so it should not displace L2/MALL contents), no arithmetic
// touches the payload and no MFMA is involved.
//
// Work resolution: a launch covers at most 64 sequences, one per lane of a
// wavefront.  Each workgroup recomputes, with one 64-lane inclusive scan, the
// prefix of per-sequence tile counts and token counts; a ballot of
// "prefix <= my tile" then gives the workgroup's sequence directly.  The
// per-sequence ranges travel by value in the kernel arguments, so nothing is
// copied to the device before a launch.
#include "dv_internal.h"

namespace dv {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 ld_nt(const u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st_nt(u32x4 v, u32x4* p) { __builtin_nontemporal_store(v, p); }

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// Inclusive prefix sum across the 64 lanes of a wavefront.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int lane = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

// Index of the first lane whose inclusive prefix exceeds `item` (prefixes
// are non-decreasing across lanes, so the lanes at or below `item` form a
// prefix of the wavefront).
__device__ __forceinline__ int owner_lane(int incl, int item) {
  return __popcll(__ballot(incl <= item));
}

// Workgroup IDs are dealt round-robin to the chip's 8 XCDs (each with its
// own L2).  The bulk kernels re-deal the linearised (tile, slab) grid so each
// XCD streams a contiguous range of it: workgroup `lin` runs on XCD lin % 8
// and takes item lin / 8 of that XCD's range; XCD x owns total / 8 items
// (one more if x < total % 8) starting at x * (total / 8) + min(x, total % 8).
// The map is a bijection on [0, total) whatever order the hardware actually
// deals workgroups in; on MI355X it lifts the dense copy from 74 % to 77-79 %
// of HBM peak.  (The paged kernels do not use it; see xcd_chunk_tile.)
__device__ __forceinline__ void xcd_tile(int* tile, int64_t* slab_row) {
  const uint64_t total = (uint64_t)gridDim.x * gridDim.y;
  const uint64_t lin = blockIdx.x + (uint64_t)blockIdx.y * gridDim.x;
  const uint64_t q = total / 8, r = total % 8, x = lin % 8;
  const uint64_t t = x * q + (x < r ? x : r) + lin / 8;
  *tile = (int)(t % gridDim.x);
  *slab_row = (int64_t)(t / gridDim.x);
}

// Pool-order scatters: the linearised (tile, slab) grid dealt to the XCDs in
// chunks of kPoolChunk consecutive items.  Workgroup `lin` runs on XCD lin %
// 8 and takes item (lin / 8) % C of that XCD's (lin / 8) / C-th chunk; round
// r gives chunk 8r + x to XCD x.  Items past the last whole round keep their
// place.  A bijection on [0, total), whatever order the hardware actually
// deals workgroups in.  On MI355X it lifts the LLaMA-2-70B pool-order
// scatter from 75 % to 77 % of HBM peak, where contiguous eighths (as
// xcd_tile) cost it 2 points and cost the table-order gather 6.
__device__ __forceinline__ void xcd_chunk_tile(int* tile, int64_t* slab_row) {
  const uint64_t total = (uint64_t)gridDim.x * gridDim.y;
  const uint64_t lin = blockIdx.x + (uint64_t)blockIdx.y * gridDim.x;
  constexpr uint64_t C = kPoolChunk;
  const uint64_t full = total / (8 * C) * (8 * C);
  uint64_t t = lin;
  if (lin < full) {
    const uint64_t x = lin % 8, k = lin / 8;
    t = ((k / C) * 8 + x) * C + k % C;
  }
  *tile = (int)(t % gridDim.x);
  *slab_row = (int64_t)(t / gridDim.x);
}

// ---------------------------------------------------------------------------
// Dense runs: grid (tiles_per_slab, nslabs); a tile is kDenseTile units of
// one (sequence, head) run.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(kThreads) dense_runs_kernel(DenseRunArgs a) {
  const int lane = lane_id();
  int n = 0, t0 = 0;
  if (lane < a.nseq) {
    n = a.r.n[lane];
    t0 = a.r.t0[lane];
  }
  const int run = n * a.du;
  const int tpr = (run + kDenseTile - 1) / kDenseTile;
  const int tiles = tpr * a.heads;
  const int incl = wave_incl_scan(tiles);
  const int tok_incl = wave_incl_scan(n);

  int tile;
  int64_t y;
  xcd_tile(&tile, &y);
  const int b = owner_lane(incl, tile);
  const int excl_b = __shfl(incl - tiles, b, 64);
  const int tpr_b = __shfl(tpr, b, 64);
  const int run_b = __shfl(run, b, 64);
  const int t0_b = __shfl(t0, b, 64);
  const int p_b = __shfl(tok_incl - n, b, 64);

  const int r = tile - excl_b;
  const int h = r / tpr_b;
  const int k = r - h * tpr_b;

  const int64_t slab = a.m.slab0 + y * a.m.slab_step;
  const int64_t wslab = a.m.wslab0 + y * a.m.slab_step;
  u32x4* cache = (u32x4*)a.cache + slab * a.s_slab + (int64_t)(a.b0 + b) * a.s_b +
                 (int64_t)h * a.s_h + (int64_t)t0_b * a.du + (int64_t)k * kDenseTile;
  u32x4* wire = (u32x4*)a.wire + wslab * a.m.w_slab + (int64_t)p_b * a.heads * a.du +
                (int64_t)h * run_b + (int64_t)k * kDenseTile;
  const u32x4* src = (D == kPack) ? cache : wire;
  u32x4* dst = (D == kPack) ? wire : cache;
  const int count = min(kDenseTile, run_b - k * kDenseTile);

  // Loads carry no per-lane guard (a lane past the tile's end re-reads the
  // tile's last unit), so they issue back to back with a single wait; a
  // guarded load would make the compiler wait after every one.
  u32x4 v[kDenseUnroll];
#pragma unroll
  for (int i = 0; i < kDenseUnroll; ++i)
    v[i] = ld_nt(src + min(i * kThreads + (int)threadIdx.x, count - 1));
#pragma unroll
  for (int i = 0; i < kDenseUnroll; ++i) {
    const int idx = i * kThreads + threadIdx.x;
    if (idx < count) st_nt(v[i], dst + idx);
  }
}

// ---------------------------------------------------------------------------
// Paged blocks: grid (tiles_per_slab, nslabs); a tile is the part of one
// block of one sequence inside its token range, for kPagedHeads heads.  For
// a fixed (slab, block) the pool holds the heads back to back, so the tile's
// pool side is one contiguous piece; on the wire side each head's tokens are
// contiguous.  Two heads of a 16-token, 128-dim block make an 8 KB tile, the
// size the dense kernel streams best at.
//
// Table order (owner == null): tiles enumerate (sequence, logical block,
// head pair) and find the pool block through the table, so consecutive
// workgroups read consecutive wire bytes.  Pool order (owner set, unpack
// only): tiles enumerate (pool block, head pair) and find the sequence and
// logical block through the owner map, so consecutive workgroups write
// consecutive pool bytes -- on MI355X writes scattered by a random table
// cost more than reads scattered the same way.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(kThreads) paged_kernel(PagedArgs a) {
  static_assert(kPagedHeads == 2, "the (head, unit) split below assumes two heads per tile");
  const int lane = lane_id();
  const int bs = a.block_size;
  const int ngrp = (a.heads + kPagedHeads - 1) / kPagedHeads;
  int n = 0, t0 = 0, tiles = 0;
  if (lane < a.nseq) {
    n = a.r.n[lane];
    t0 = a.r.t0[lane];
    if (n > 0) tiles = ((t0 + n + bs - 1) / bs - t0 / bs) * ngrp;
  }
  const int tok_incl = wave_incl_scan(n);

  // Table order keeps the hardware's round-robin dealing: pool blocks are
  // scattered by the block table anyway, and on MI355X every XCD-grouped
  // order measured was slower (by 2-8 %).  Pool order deals chunks of tiles.
  int tile = blockIdx.x;
  int64_t y = blockIdx.y;
  if (a.owner) xcd_chunk_tile(&tile, &y);
  int b, j, grp, blk;
  if (a.owner) {
    blk = tile / ngrp;
    grp = tile - blk * ngrp;
    const int own = a.owner[blk];
    if (own < 0) return;  // block not written by this call
    b = own / a.max_blocks;
    j = own - b * a.max_blocks;
    if (b >= a.nseq) return;
  } else {
    const int incl = wave_incl_scan(tiles);
    b = owner_lane(incl, tile);
    const int tj = tile - __shfl(incl - tiles, b, 64);
    grp = tj % ngrp;
    j = __shfl(t0, b, 64) / bs + tj / ngrp;  // logical block
    blk = a.bt[(int64_t)(a.b0 + b) * a.max_blocks + j];
    if (blk < 0 || blk >= a.num_blocks) return;  // unmapped block: skipped
  }
  const int n_b = __shfl(n, b, 64);
  const int t0_b = __shfl(t0, b, 64);
  const int p_b = __shfl(tok_incl - n, b, 64);
  const int s_lo = max(t0_b, j * bs);
  const int s_hi = min(t0_b + n_b, (j + 1) * bs);
  if (s_lo >= s_hi) return;

  const int run = (s_hi - s_lo) * a.du;  // units per head in this tile
  const int64_t slab = a.m.slab0 + y * a.m.slab_step;
  const int64_t wslab = a.m.wslab0 + y * a.m.slab_step;
  const int h0 = grp * kPagedHeads;
  u32x4* pool = (u32x4*)a.pool + slab * a.s_slab + (int64_t)blk * a.s_blk +
                (int64_t)h0 * a.s_h + (int64_t)(s_lo - j * bs) * a.du;
  const int64_t w_h = (int64_t)n_b * a.du;  // wire units per head of this sequence
  u32x4* wire = (u32x4*)a.wire + wslab * a.m.w_slab + (int64_t)p_b * a.heads * a.du +
                (int64_t)h0 * w_h + (int64_t)(s_lo - t0_b) * a.du;

  // Flattened (head, unit) index over the tile; loads unguarded as in the
  // dense kernel (a lane past the end re-reads the last unit).  With two
  // heads the index is below 2 * run, so one comparison names the head (an
  // integer division here cost 3-4 % of the gather's bandwidth).
  const int total = min(kPagedHeads, a.heads - h0) * run;
  for (int base = 0; base < total; base += kPagedUnroll * kThreads) {
    u32x4 v[kPagedUnroll];
    int hh[kPagedUnroll], ee[kPagedUnroll];
#pragma unroll
    for (int i = 0; i < kPagedUnroll; ++i) {
      const int idx = min(base + i * kThreads + (int)threadIdx.x, total - 1);
      hh[i] = idx >= run ? 1 : 0;
      ee[i] = idx - hh[i] * run;
      v[i] = ld_nt((D == kPack) ? pool + hh[i] * a.s_h + ee[i] : wire + hh[i] * w_h + ee[i]);
    }
#pragma unroll
    for (int i = 0; i < kPagedUnroll; ++i) {
      if (base + i * kThreads + (int)threadIdx.x < total)
        st_nt(v[i], (D == kPack) ? wire + hh[i] * w_h + ee[i] : pool + hh[i] * a.s_h + ee[i]);
    }
  }
}

// Pool order for calls of more than 64 sequences (stream-in only): grid
// (num_blocks * head pairs, nslabs); as paged_kernel's pool order, but one
// launch covers every sequence of the call, a sequence's range and token
// prefix coming from the arguments instead of a wavefront scan.  (For up to
// 64 sequences paged_kernel is used: there the ranges load in parallel with
// the owner entry, where here they depend on it; measured on MI355X this
// kernel was 2.8 % slower on the LLaMA-2-70B pool's 32 sequences.)
__global__ void __launch_bounds__(kThreads) paged_pool_kernel(PoolOrderArgs a) {
  const int bs = a.block_size;
  const int ngrp = (a.heads + kPagedHeads - 1) / kPagedHeads;
  int tile;
  int64_t y;
  xcd_chunk_tile(&tile, &y);
  const int blk = tile / ngrp;
  const int grp = tile - blk * ngrp;
  const int own = __builtin_amdgcn_readfirstlane(a.owner[blk]);
  if (own < 0) return;  // block not written by this call
  const int b = own / a.max_blocks;
  const int j = own - b * a.max_blocks;
  if (b >= a.nseq) return;
  const int n_b = a.n[b];
  const int t0_b = a.t0[b];
  const int p_b = a.p[b];
  const int s_lo = max(t0_b, j * bs);
  const int s_hi = min(t0_b + n_b, (j + 1) * bs);
  if (s_lo >= s_hi) return;

  const int run = (s_hi - s_lo) * a.du;
  const int64_t slab = a.m.slab0 + y * a.m.slab_step;
  const int64_t wslab = a.m.wslab0 + y * a.m.slab_step;
  const int h0 = grp * kPagedHeads;
  u32x4* pool = (u32x4*)a.pool + slab * a.s_slab + (int64_t)blk * a.s_blk +
                (int64_t)h0 * a.s_h + (int64_t)(s_lo - j * bs) * a.du;
  const int64_t w_h = (int64_t)n_b * a.du;
  u32x4* wire = (u32x4*)a.wire + wslab * a.m.w_slab + (int64_t)p_b * a.heads * a.du +
                (int64_t)h0 * w_h + (int64_t)(s_lo - t0_b) * a.du;
  const int total = min(kPagedHeads, a.heads - h0) * run;
  for (int base = 0; base < total; base += kPagedUnroll * kThreads) {
    u32x4 v[kPagedUnroll];
    int hh[kPagedUnroll], ee[kPagedUnroll];
#pragma unroll
    for (int i = 0; i < kPagedUnroll; ++i) {
      const int idx = min(base + i * kThreads + (int)threadIdx.x, total - 1);
      hh[i] = idx >= run ? 1 : 0;
      ee[i] = idx - hh[i] * run;
      v[i] = ld_nt(wire + hh[i] * w_h + ee[i]);
    }
#pragma unroll
    for (int i = 0; i < kPagedUnroll; ++i) {
      if (base + i * kThreads + (int)threadIdx.x < total) st_nt(v[i], pool + hh[i] * a.s_h + ee[i]);
    }
  }
}

// Owner map (see OwnerArgs): a clearing pass, then one lane per table entry.
__global__ void __launch_bounds__(kThreads) owner_clear_kernel(OwnerArgs a) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i < a.num_blocks) a.owner[i] = -1;
}

__global__ void __launch_bounds__(kThreads) claims_clear_kernel(OwnerArgs a) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i < a.num_blocks) a.owner[i] = 0;
}

// One lane per table entry, as owner_build_kernel; counts instead of storing.
__global__ void __launch_bounds__(kThreads) claims_count_kernel(OwnerArgs a) {
  const int b = blockIdx.y;
  const int j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= a.max_blocks) return;
  const int t0 = a.r.t0[b], t1 = t0 + a.r.n[b];
  if (t0 >= t1 || (j + 1) * a.block_size <= t0 || j * a.block_size >= t1) return;
  const int blk = a.bt[(int64_t)(a.b0 + b) * a.max_blocks + j];
  if (blk < 0 || blk >= a.num_blocks) return;
  atomicAdd(&a.owner[blk], 1);
}

__global__ void __launch_bounds__(kThreads) owner_build_kernel(OwnerArgs a) {
  const int b = blockIdx.y;
  const int j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= a.max_blocks) return;
  const int t0 = a.r.t0[b], t1 = t0 + a.r.n[b];
  if (t0 >= t1 || (j + 1) * a.block_size <= t0 || j * a.block_size >= t1) return;
  const int gb = a.b0 + b;  // the sequence's index in the call
  const int blk = a.bt[(int64_t)gb * a.max_blocks + j];
  if (blk < 0 || blk >= a.num_blocks) return;
  a.owner[blk] = gb * a.max_blocks + j;
}

// ---------------------------------------------------------------------------
// Single tokens: grid (ceil(units_per_slab / 256), nslabs).  Lane u of a
// slab moves wire unit u; the active sequences are ranked once per
// workgroup into LDS together with the cache offset of their token.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(kThreads) token_kernel(TokenArgs a) {
  __shared__ int64_t s_base[kSeqPerLaunch];
  const int lane = lane_id();
  const int p = lane < a.nseq ? a.pos[lane] : -1;
  const uint64_t act = __ballot(p >= 0);
  const int nact = __popcll(act);
  if (threadIdx.x < 64 && p >= 0) {
    const int rank = __popcll(act & ((1ull << lane) - 1ull));
    const int b = a.b0 + lane;
    int64_t base;
    if (!a.paged) {
      base = (int64_t)b * a.s_b + (int64_t)p * a.s_tok;
    } else {
      const int blk = a.bt[(int64_t)b * a.max_blocks + p / a.block_size];
      base = (blk >= 0 && blk < a.num_blocks)
                 ? (int64_t)blk * a.s_blk + (int64_t)(p % a.block_size) * a.s_tok
                 : -1;
    }
    s_base[rank] = base;
  }
  __syncthreads();

  const int hd = a.heads * a.du;
  const int u = blockIdx.x * kThreads + threadIdx.x;
  if (u >= nact * hd) return;
  const int rank = u / hd;
  const int rem = u - rank * hd;
  const int h = rem / a.du;
  const int e = rem - h * a.du;
  const int64_t base = s_base[rank];
  if (base < 0) return;  // unmapped block: skipped

  const int64_t y = blockIdx.y;
  const int64_t slab = a.m.slab0 + y * a.m.slab_step;
  const int64_t wslab = a.m.wslab0 + y * a.m.slab_step;
  u32x4* cache = (u32x4*)a.cache + slab * a.s_slab + base + (int64_t)h * a.s_h +
                 (int64_t)e * a.s_e;
  u32x4* wire = (u32x4*)a.wire + wslab * a.m.w_slab + u;
  if (D == kPack)
    st_nt(ld_nt(cache), wire);
  else
    st_nt(ld_nt(wire), cache);
}

// ---------------------------------------------------------------------------
// Short runs: grid (ceil(units_per_slab / (256 * U)), nslabs).  Each lane
// moves U wire units of the flattened (sequence, head, token, unit) order
// of its slab, 256 units apart; the per-sequence prefix of run sizes sits in
// LDS and a 6-step binary search names each unit's sequence (the
// single-token kernel above skips the search, since there every run is one
// token).  Loads are clamped to the last unit and issue before any store.
// ---------------------------------------------------------------------------
template <int D, int U>
__global__ void __launch_bounds__(kThreads) small_runs_kernel(SmallRunArgs a) {
  __shared__ int s_incl[kSeqPerLaunch];  // inclusive prefix of n_b * heads * du
  __shared__ int s_run[kSeqPerLaunch];   // n_b * du: units per head of sequence b
  __shared__ int s_t0[kSeqPerLaunch];
  const int lane = lane_id();
  if (threadIdx.x < 64) {
    int n = 0, t0 = 0;
    if (lane < a.nseq) {
      n = a.r.n[lane];
      t0 = a.r.t0[lane];
    }
    s_incl[lane] = wave_incl_scan(n * a.heads * a.du);
    s_run[lane] = n * a.du;
    s_t0[lane] = t0;
  }
  __syncthreads();
  const int total = s_incl[kSeqPerLaunch - 1];
  const int64_t y = blockIdx.y;
  const int64_t slab = a.m.slab0 + y * a.m.slab_step;
  const int64_t wslab = a.m.wslab0 + y * a.m.slab_step;
  u32x4* cache_slab = (u32x4*)a.cache + slab * a.s_slab;
  u32x4* wire_slab = (u32x4*)a.wire + wslab * a.m.w_slab;
  int64_t co[U];
  bool ok[U];
  u32x4 v[U];
#pragma unroll
  for (int i = 0; i < U; ++i) {
    const int u0 = (blockIdx.x * U + i) * kThreads + threadIdx.x;
    const int u = min(u0, total - 1);
    // The first sequence whose inclusive prefix exceeds u (it has n_b > 0).
    int lo = 0, hi = kSeqPerLaunch - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (s_incl[mid] > u) hi = mid; else lo = mid + 1;
    }
    const int b = lo;
    const int run = s_run[b];
    const int rem = u - (s_incl[b] - run * a.heads);
    const int h = rem / run;
    const int e = rem - h * run;  // unit within the (sequence, head) run
    const int t = e / a.du;
    const int g = e - t * a.du;   // 16-byte group within the token
    const int s = s_t0[b] + t;    // token position in the cache
    ok[i] = u0 < total;
    if (!a.paged) {
      co[i] = (int64_t)(a.b0 + b) * a.s_b + (int64_t)s * a.s_tok;
    } else {
      const int blk = a.bt[(int64_t)(a.b0 + b) * a.max_blocks + s / a.block_size];
      ok[i] = ok[i] && blk >= 0 && blk < a.num_blocks;  // unmapped block: skipped
      co[i] = (int64_t)(ok[i] ? blk : 0) * a.s_blk + (int64_t)(s % a.block_size) * a.s_tok;
    }
    co[i] += (int64_t)h * a.s_h + (int64_t)g * a.s_e;
    v[i] = ld_nt((D == kPack) ? cache_slab + co[i] : wire_slab + u);
  }
#pragma unroll
  for (int i = 0; i < U; ++i) {
    const int u = (blockIdx.x * U + i) * kThreads + threadIdx.x;
    if (ok[i]) st_nt(v[i], (D == kPack) ? wire_slab + u : cache_slab + co[i]);
  }
}

// ---------------------------------------------------------------------------
// Split-key slab: grid (tiles_per_slab, nslabs); a tile is 64 tokens of one
// (sequence, head).  The cache holds the head as [group][token] (each group
// 16 bytes), the wire as [token][group]: the tile is read with lanes along
// the contiguous axis of the source, transposed through LDS (dynamic, 64
// rows of du + 1 units: the padding unit keeps column accesses on distinct
// banks), and written with lanes along the contiguous axis of the
// destination.  Both passes take 4 units per lane at a time with clamped,
// unguarded loads, so the loads of a pass issue back to back (a guarded load
// per group left most of the load latency exposed: 70 % -> 77 % of HBM peak
// on the OPT-13B shape).
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(kThreads) ksplit_kernel(KsplitArgs a) {
  static_assert(kKsplitTile == 64, "cache-side units split as (group, token) = (j >> 6, j & 63)");
  extern __shared__ u32x4 lds[];
  const int lane = lane_id();
  int n = 0, t0 = 0;
  if (lane < a.nseq) {
    n = a.r.n[lane];
    t0 = a.r.t0[lane];
  }
  const int tpr = (n + kKsplitTile - 1) / kKsplitTile;
  const int tiles = tpr * a.heads;
  const int incl = wave_incl_scan(tiles);
  const int tok_incl = wave_incl_scan(n);

  int tile;
  int64_t y;
  xcd_tile(&tile, &y);
  const int b = owner_lane(incl, tile);
  const int excl_b = __shfl(incl - tiles, b, 64);
  const int tpr_b = __shfl(tpr, b, 64);
  const int n_b = __shfl(n, b, 64);
  const int t0_b = __shfl(t0, b, 64);
  const int p_b = __shfl(tok_incl - n, b, 64);
  const int r = tile - excl_b;
  const int h = r / tpr_b;
  const int k = r - h * tpr_b;
  const int tok0 = k * kKsplitTile;              // first token of the tile, range-relative
  const int ntk = min(kKsplitTile, n_b - tok0);  // tokens in the tile
  const int du = a.du;
  const int pitch = du + 1;

  const int64_t slab = a.m.slab0 + y * a.m.slab_step;
  const int64_t wslab = a.m.wslab0 + y * a.m.slab_step;
  u32x4* head = (u32x4*)a.cache + slab * a.s_slab + (int64_t)(a.b0 + b) * a.s_b +
                (int64_t)h * a.s_h + t0_b + tok0;  // group 0 of the tile's first token
  u32x4* wire = (u32x4*)a.wire + wslab * a.m.w_slab + (int64_t)p_b * a.heads * du +
                (int64_t)h * n_b * du + (int64_t)tok0 * du;
  const int64_t S = a.seq_cap;
  // Cache side: unit j = group * 64 + token (tokens fastest); wire side:
  // unit idx = token * du + group.
  const int cache_units = du * kKsplitTile;
  const int wire_units = ntk * du;
  constexpr int kChunk = 4;
  if (D == kPack) {
    for (int base = 0; base < cache_units; base += kChunk * kThreads) {
      u32x4 v[kChunk];
#pragma unroll
      for (int i = 0; i < kChunk; ++i) {
        const int j = min(base + i * kThreads + (int)threadIdx.x, cache_units - 1);
        v[i] = ld_nt(head + (j >> 6) * S + min(j & 63, ntk - 1));
      }
#pragma unroll
      for (int i = 0; i < kChunk; ++i) {
        const int j = base + i * kThreads + (int)threadIdx.x;
        if (j < cache_units && (j & 63) < ntk) lds[(j & 63) * pitch + (j >> 6)] = v[i];
      }
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < wire_units; idx += kThreads) {
      const int t = idx / du;
      st_nt(lds[t * pitch + (idx - t * du)], wire + idx);
    }
  } else {
    for (int base = 0; base < wire_units; base += kChunk * kThreads) {
      u32x4 v[kChunk];
#pragma unroll
      for (int i = 0; i < kChunk; ++i)
        v[i] = ld_nt(wire + min(base + i * kThreads + (int)threadIdx.x, wire_units - 1));
#pragma unroll
      for (int i = 0; i < kChunk; ++i) {
        const int idx = base + i * kThreads + (int)threadIdx.x;
        if (idx < wire_units) {
          const int t = idx / du;
          lds[t * pitch + (idx - t * du)] = v[i];
        }
      }
    }
    __syncthreads();
    for (int j = threadIdx.x; j < cache_units; j += kThreads)
      if ((j & 63) < ntk) st_nt(lds[(j & 63) * pitch + (j >> 6)], head + (j >> 6) * S + (j & 63));
  }
}

// ---------------------------------------------------------------------------
// Cache-to-cache copy: grid (ceil(units_per_slab / (256 * kCopyUnroll)),
// nslabs).  Unit u of a slab is the u-th 16-byte unit of the ranges taken
// in (sequence, head, token, unit) order, i.e. the wire order, but it moves
// straight from the source cache to the same logical place in the
// destination cache.  Used for swaps whose rows are too narrow for DMA to
// run efficiently (a decode step's one-token update is 256-byte rows); on
// pinned host memory each lane's store or load crosses the host link.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kThreads) copy_kernel(CopyArgs a) {
  __shared__ int s_incl[kSeqPerLaunch];
  const int lane = lane_id();
  if (threadIdx.x < 64) {
    const int n = lane < a.nseq ? a.r.n[lane] : 0;
    s_incl[lane] = wave_incl_scan(n * a.heads * a.du);
  }
  __syncthreads();
  const int total = s_incl[kSeqPerLaunch - 1];
  const int64_t slab = a.slab0 + (int64_t)blockIdx.y;
  int64_t so[kCopyUnroll], dst_off[kCopyUnroll];
  bool ok[kCopyUnroll];
#pragma unroll
  for (int i = 0; i < kCopyUnroll; ++i) {
    const int u0 = (blockIdx.x * kCopyUnroll + i) * kThreads + threadIdx.x;
    ok[i] = u0 < total;
    const int u = min(u0, total - 1);
    // sequence: first lane whose inclusive prefix exceeds u
    int lo = 0, hi = kSeqPerLaunch - 1;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (s_incl[mid] > u) hi = mid; else lo = mid + 1;
    }
    const int b = lo;
    const int run = a.r.n[b] * a.du;
    const int rem = u - (s_incl[b] - run * a.heads);
    const int h = rem / run;
    const int e = rem - h * run + a.r.t0[b] * a.du;
    so[i] = slab * a.s_slab + (int64_t)(a.b0 + b) * a.s_b + (int64_t)h * a.s_h + e;
    dst_off[i] = slab * a.d_slab + (int64_t)(a.b0 + b) * a.d_b + (int64_t)h * a.d_h + e;
  }
  const u32x4* src = (const u32x4*)a.src;
  u32x4* dst = (u32x4*)a.dst;
  u32x4 v[kCopyUnroll];
#pragma unroll
  for (int i = 0; i < kCopyUnroll; ++i) v[i] = ld_nt(src + so[i]);
#pragma unroll
  for (int i = 0; i < kCopyUnroll; ++i)
    if (ok[i]) st_nt(v[i], dst + dst_off[i]);
}

}  // namespace

namespace {

// Launch with the runtime's own status for this launch (a stale error left by
// an unrelated earlier call is not picked up, unlike hipGetLastError).
template <typename Args>
hipError_t launch(const void* fn, dim3 grid, const Args& a, hipStream_t s, size_t lds = 0) {
  if (grid.x == 0 || grid.y == 0) return hipSuccess;
  void* args[] = {const_cast<Args*>(&a)};
  return hipLaunchKernel(fn, grid, dim3(kThreads), args, lds, s);
}

}  // namespace

hipError_t launch_dense_runs(int dir, const DenseRunArgs& a, uint32_t tiles_per_slab,
                             uint32_t nslabs, hipStream_t s) {
  const void* fn = dir == kPack ? (const void*)&dense_runs_kernel<kPack>
                                : (const void*)&dense_runs_kernel<kUnpack>;
  return launch(fn, dim3(tiles_per_slab, nslabs), a, s);
}

hipError_t launch_paged(int dir, const PagedArgs& a, uint32_t tiles_per_slab, uint32_t nslabs,
                        hipStream_t s) {
  const void* fn =
      dir == kPack ? (const void*)&paged_kernel<kPack> : (const void*)&paged_kernel<kUnpack>;
  return launch(fn, dim3(tiles_per_slab, nslabs), a, s);
}

// Workgroups of kThreads lanes covering n items (n up to INT32_MAX).
static uint32_t groups_of(int32_t n) { return (uint32_t)(((int64_t)n + kThreads - 1) / kThreads); }

hipError_t launch_paged_pool_order(const PoolOrderArgs& a, uint32_t tiles_per_slab,
                                   uint32_t nslabs, hipStream_t s) {
  return launch((const void*)&paged_pool_kernel, dim3(tiles_per_slab, nslabs), a, s);
}

hipError_t launch_owner_clear(const OwnerArgs& a, hipStream_t s) {
  return launch((const void*)&owner_clear_kernel, dim3(groups_of(a.num_blocks)), a, s);
}

hipError_t launch_owner_build(const OwnerArgs& a, hipStream_t s) {
  return launch((const void*)&owner_build_kernel, dim3(groups_of(a.max_blocks), a.nseq), a, s);
}

hipError_t launch_block_claims(const OwnerArgs& a, bool clear, hipStream_t s) {
  if (clear) {
    const hipError_t e =
        launch((const void*)&claims_clear_kernel, dim3(groups_of(a.num_blocks)), a, s);
    if (e != hipSuccess) return e;
  }
  return launch((const void*)&claims_count_kernel, dim3(groups_of(a.max_blocks), a.nseq), a, s);
}

hipError_t launch_token(int dir, const TokenArgs& a, uint32_t units_per_slab, uint32_t nslabs,
                        hipStream_t s) {
  const void* fn =
      dir == kPack ? (const void*)&token_kernel<kPack> : (const void*)&token_kernel<kUnpack>;
  return launch(fn, dim3((units_per_slab + kThreads - 1) / kThreads, nslabs), a, s);
}

hipError_t launch_small_runs(int dir, const SmallRunArgs& a, uint32_t units_per_slab,
                             uint32_t nslabs, hipStream_t s) {
  // Two units per lane once a launch moves 8 MB or more; measured on MI355X
  // for 2-16 tokens per sequence, one unit per lane is faster below that
  // (fewer dependent steps per lane) and two above (fewer workgroups).
  const bool two = (uint64_t)units_per_slab * nslabs >= (1ull << 19);
  const void* fn;
  if (dir == kPack)
    fn = two ? (const void*)&small_runs_kernel<kPack, 2> : (const void*)&small_runs_kernel<kPack, 1>;
  else
    fn = two ? (const void*)&small_runs_kernel<kUnpack, 2>
             : (const void*)&small_runs_kernel<kUnpack, 1>;
  const uint32_t per = kThreads * (two ? 2 : 1);
  return launch(fn, dim3((units_per_slab + per - 1) / per, nslabs), a, s);
}

hipError_t launch_ksplit(int dir, const KsplitArgs& a, uint32_t tiles_per_slab, uint32_t nslabs,
                         hipStream_t s) {
  const void* fn =
      dir == kPack ? (const void*)&ksplit_kernel<kPack> : (const void*)&ksplit_kernel<kUnpack>;
  // The tile's LDS, rounded up for tiles of 16 KB or more so that at most 4
  // workgroups share a CU's 160 KB: on MI355X 8 workgroups of 16 KB tiles
  // ran 2-3 % slower than 4, while 8 KB tiles ran 13 % faster with 8.
  size_t lds = (size_t)kKsplitTile * (a.du + 1) * sizeof(uint32_t) * 4;
  if (a.du >= 16 && lds < kKsplitLdsFor4) lds = kKsplitLdsFor4;
  return launch(fn, dim3(tiles_per_slab, nslabs), a, s, lds);
}

hipError_t launch_copy(const CopyArgs& a, uint32_t units_per_slab, uint32_t nslabs,
                       hipStream_t s) {
  const uint32_t per = kThreads * kCopyUnroll;
  return launch((const void*)&copy_kernel, dim3((units_per_slab + per - 1) / per, nslabs), a, s);
}

}  // namespace dv
