// Internal launch descriptors shared by the host dispatch (dv_api.cpp) and
// the kernels (dv_kernels.hip).  Units are 16 bytes throughout: every cache
// and wire address handled here is a multiple of 16 bytes, which lets each
// lane move one 128-bit word per access.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dv {

// Sequences handled by one launch: one per lane of a 64-wide wavefront, so
// per-sequence prefix sums are a single wavefront scan.
constexpr int kSeqPerLaunch = 64;
constexpr int kThreads = 256;

enum Dir : int { kPack = 0, kUnpack = 1 };

struct SeqRanges {
  int32_t t0[kSeqPerLaunch];  // first token of each sequence's range
  int32_t n[kSeqPerLaunch];   // tokens in the range (0 = sequence skipped)
};

// Slab = one (layer, K|V) half of the cache; grid row y handles cache slab
// slab0 + y*slab_step, whose data sits in wire slab wslab0 + y*slab_step.
struct SlabMap {
  int32_t slab0, slab_step, wslab0, pad;
  int64_t w_slab;  // wire units per slab: N * heads * du
};

// Dense runs: for each (sequence, head) the range is one contiguous run of
// n*du units in the cache and in the wire.
struct DenseRunArgs {
  void* cache;     // microbatch base
  void* wire;      // wire base advanced to this launch's first sequence
  int64_t s_slab;  // cache units per slab
  int64_t s_b;     // cache units per sequence
  int64_t s_h;     // cache units per head
  SlabMap m;
  int32_t du;      // units per token (head_dim * elem_bytes / 16)
  int32_t heads;
  int32_t nseq;    // sequences in this launch (<= 64)
  int32_t b0;      // index of the launch's first sequence
  SeqRanges r;
};

// Paged blocks: one workgroup per (slab, block, head pair).  Blocks are
// taken in table order -- (sequence, logical block) -- or, when `owner` is
// set, in pool order through the owner map (launches with all sequences in
// one group, b0 = 0).
struct PagedArgs {
  void* pool;
  void* wire;
  const int32_t* bt;     // this microbatch's block table [batch][max_blocks]
  const int32_t* owner;  // pool order: [num_blocks] owner map, else null
  int64_t s_slab;        // pool units per slab (NB * heads * bs * du)
  int64_t s_blk;         // pool units per block (heads * bs * du)
  int64_t s_h;           // pool units per head in a block (bs * du)
  SlabMap m;
  int32_t du, heads, nseq, b0;
  int32_t block_size, num_blocks, max_blocks, pad;
  SeqRanges r;
};

// Sequences a pool-order stream-in covers in one launch: their ranges and
// token prefixes travel in the arguments (3 KB).
constexpr int kPoolSeqMax = 256;

// Paged stream-in in pool order for calls of more than 64 sequences: one
// workgroup per (slab, pool block, head pair) of the whole call; the owner
// map names each block's (sequence, logical block), and the sequence's
// range and exclusive token prefix (over the call, < 2^31) come from the
// arrays below.
struct PoolOrderArgs {
  void* pool;
  void* wire;             // the call's contiguous buffer
  const int32_t* owner;   // [num_blocks] owner map
  int64_t s_slab, s_blk, s_h;  // as PagedArgs
  SlabMap m;
  int32_t du, heads, nseq, max_blocks;
  int32_t block_size, num_blocks, pad0, pad1;
  int32_t t0[kPoolSeqMax];  // first token of each sequence's range
  int32_t n[kPoolSeqMax];   // tokens in the range
  int32_t p[kPoolSeqMax];   // tokens of all earlier sequences
};
static_assert(sizeof(PoolOrderArgs) <= 3584, "pool-order arguments stay well under 4 KB");

// Owner map of a paged table over the streamed ranges: owner[blk] =
// b * max_blocks + j for each entry (b, j) whose logical block j holds a
// streamed token of sequence b and whose block blk is in [0, num_blocks);
// -1 for every other block.  Built by one clearing launch and one launch
// per group of up to 64 sequences, b0 being the group's first sequence.
struct OwnerArgs {
  int32_t* owner;
  const int32_t* bt;
  int32_t nseq, block_size, num_blocks, max_blocks;
  int32_t b0, pad;  // index of the launch's first sequence
  SeqRanges r;
};

// Single-token ranges (decode-step increments): one unit per lane over the
// flattened (active sequence, head, unit) space of each slab.
struct TokenArgs {
  void* cache;
  void* wire;
  const int32_t* bt;  // paged only
  int64_t s_slab;
  int64_t s_b;        // dense: units per sequence
  int64_t s_blk;      // paged: units per block
  int64_t s_h;        // units per head (dense: S*du; paged: bs*du; split key: S*du)
  int64_t s_tok;      // units per token (du, or 1 in a split key slab)
  int64_t s_e;        // units between consecutive 16-byte groups of one token
                      // (1, or S in a split key slab)
  SlabMap m;
  int32_t du, heads, nseq, b0;
  int32_t paged, block_size, num_blocks, max_blocks;
  int32_t pos[kSeqPerLaunch];  // token of each sequence, < 0 = inactive
};

// Short runs (a few tokens per sequence, e.g. a decode step that accepts
// several tokens): one 16-byte unit per lane over the flattened wire order
// of each slab, (sequence, head, token, unit), so no lane idles the way it
// would in a tile sized for long runs.  Unit e of sequence b's run for head
// h holds token t0 + e / du, group e % du, at cache offset
// (t0 + e / du) * s_tok + (e % du) * s_e from the (sequence, head) base;
// paged caches find the token's block through the table.
struct SmallRunArgs {
  void* cache;
  void* wire;
  const int32_t* bt;  // paged only
  int64_t s_slab;
  int64_t s_b;        // dense: units per sequence
  int64_t s_blk;      // paged: units per block
  int64_t s_h;        // units per head
  int64_t s_tok;      // units per token (du, or 1 in a split key slab)
  int64_t s_e;        // units between consecutive 16-byte groups of a token (1, or S)
  SlabMap m;
  int32_t du, heads, nseq, b0;
  int32_t paged, block_size, num_blocks, max_blocks;
  SeqRanges r;
};

// Split-key slab: 64-token tiles transposed through LDS.
struct KsplitArgs {
  void* cache;
  void* wire;
  int64_t s_slab, s_b, s_h;  // as dense
  SlabMap m;
  int32_t du;  // 16-byte groups per token (head_dim * elem_bytes / 16), <= kKsplitMaxDu
  int32_t heads, nseq, b0;
  int32_t seq_cap;  // S: units between consecutive groups of one head
  int32_t pad;
  SeqRanges r;
};
// Cache-to-cache copy of the same logical positions between two dense
// caches (device slot <-> pinned host mirror) for narrow rows.
struct CopyArgs {
  void* src;
  void* dst;
  int64_t s_slab, s_b, s_h;  // source strides (units); token stride du
  int64_t d_slab, d_b, d_h;  // destination strides (units)
  int32_t slab0;             // grid row y copies slab slab0 + y
  int32_t du, heads, nseq, b0;
  int32_t pad;
  SeqRanges r;
};
constexpr int kCopyUnroll = 2;

constexpr int kKsplitTile = 64;
constexpr int kKsplitMaxDu = 32;  // LDS tile at most 64 x 33 units (33.8 KB)
constexpr size_t kKsplitLdsFor4 = 39 * 1024;  // 4 per CU fit in 160 KB, 5 do not

// Launchers (dv_kernels.hip).  Each returns the hipError_t of its launch.
hipError_t launch_dense_runs(int dir, const DenseRunArgs& a, uint32_t tiles_per_slab,
                             uint32_t nslabs, hipStream_t s);
hipError_t launch_paged(int dir, const PagedArgs& a, uint32_t tiles_per_slab, uint32_t nslabs,
                        hipStream_t s);
hipError_t launch_paged_pool_order(const PoolOrderArgs& a, uint32_t tiles_per_slab,
                                   uint32_t nslabs, hipStream_t s);
// Sets every entry of the owner map to -1.
hipError_t launch_owner_clear(const OwnerArgs& a, hipStream_t s);
// Fills the owner map from the table for sequences [b0, b0 + nseq).
hipError_t launch_owner_build(const OwnerArgs& a, hipStream_t s);
// Counts, per pool block, the table entries over the ranges of sequences
// [b0, b0 + nseq) that map to it, into `a.owner` (int32 counts), clearing
// the counts first when `clear` is set.
hipError_t launch_block_claims(const OwnerArgs& a, bool clear, hipStream_t s);
hipError_t launch_token(int dir, const TokenArgs& a, uint32_t units_per_slab, uint32_t nslabs,
                        hipStream_t s);
hipError_t launch_small_runs(int dir, const SmallRunArgs& a, uint32_t units_per_slab,
                             uint32_t nslabs, hipStream_t s);
hipError_t launch_ksplit(int dir, const KsplitArgs& a, uint32_t tiles_per_slab, uint32_t nslabs,
                         hipStream_t s);
hipError_t launch_copy(const CopyArgs& a, uint32_t units_per_slab, uint32_t nslabs, hipStream_t s);

// Units each dense-run workgroup moves (tiles are counted on the host with
// the same constant).  Two 16-byte units per lane (8 KB per workgroup) keeps
// register use low enough for full occupancy; measured on MI355X against 1,
// 3, 4, 8 and 16 units per lane on the OPT-13B stage shape.
constexpr int kDenseUnroll = 2;
constexpr int kDenseTile = kThreads * kDenseUnroll;

// Heads per paged tile and 16-byte units per lane per pass (tiles are
// counted on the host with kPagedHeads).  Measured on MI355X against 1, 4
// and all heads per tile on the LLaMA-2-70B paged shape.  The kernel splits
// a tile's flattened (head, unit) index with one comparison, which holds
// for two heads only.
constexpr int kPagedHeads = 2;
constexpr int kPagedUnroll = 2;

// Pool-order scatters deal their (tile, slab) grid to the 8 XCDs in chunks
// of this many consecutive tiles (8 pool blocks of one slab at 8 heads; 256
// KB for the LLaMA-2-70B pool).  Measured on MI355X on that pool against the
// hardware's round-robin dealing, contiguous eighths and chunks of 8, 16, 48
// and 64 tiles; table-order kernels keep the round-robin order, which was
// fastest for them.
constexpr int kPoolChunk = 32;

}  // namespace dv
