// Comparison baselines, not part of the streaming path.
//
// dvb_per_region_copy is the baseline of the paper's evaluation (Sec. 5.1,
// "Baseline"): the non-contiguous cache region is moved with one copy call
// per contiguous region instead of being packed into a temporary buffer
// first.  The benchmark times it against the buffered path (pack kernel +
// one copy), and the tests check it produces the same bytes in the same
// order.
//
// dvb_plain_copy is the copy ceiling the pack and unpack kernels are set
// against: a contiguous 16-byte copy with their per-lane shape (two
// nontemporal units per lane, loads before stores, 256 lanes per workgroup)
// and their XCD dealing, so the only difference left is the cache layout.
//
// dvb_block_copy is the ceiling of the paged kernels: a plain copy of whole
// blocks, one side in the order a block table gives and the other
// sequential, in the paged kernel's launch shape (8 KB per workgroup,
// consecutive workgroups on consecutive pieces of one block, no XCD
// dealing).  It has the paged gather's (or the table-order scatter's) random
// block placement without the streamed ranges and the head split.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/dv.h"

namespace {

constexpr int kCopyThreads = 256;
constexpr int kCopyUnroll = 2;
constexpr uint32_t kXcds = 8;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// The hardware deals workgroups to the 8 XCDs in turn.  Workgroup b is
// renumbered so that XCD b % 8 copies one contiguous share of the tiles:
// XCD x owns the (tiles + 7 - x) / 8 workgroups with b % 8 == x, placed after
// the shares of XCDs 0 .. x-1.  A bijection on [0, tiles).
__device__ uint32_t xcd_tile(uint32_t b, uint32_t tiles) {
  const uint32_t x = b % kXcds, i = b / kXcds;
  uint32_t start = 0;
  for (uint32_t y = 0; y < x; ++y) start += (tiles + kXcds - 1 - y) / kXcds;
  return start + i;
}

__global__ void __launch_bounds__(kCopyThreads)
    plain_copy_kernel(const u32x4* src, u32x4* dst, uint64_t units, uint32_t tiles) {
  const uint64_t u0 = (uint64_t)xcd_tile(blockIdx.x, tiles) * (kCopyThreads * kCopyUnroll) +
                      threadIdx.x;
  u32x4 v[kCopyUnroll];
#pragma unroll
  for (int k = 0; k < kCopyUnroll; ++k) {
    uint64_t u = u0 + (uint64_t)k * kCopyThreads;
    if (u >= units) u = units - 1;  // clamped: every load issues before any store
    v[k] = __builtin_nontemporal_load(src + u);
  }
#pragma unroll
  for (int k = 0; k < kCopyUnroll; ++k) {
    const uint64_t u = u0 + (uint64_t)k * kCopyThreads;
    if (u < units) __builtin_nontemporal_store(v[k], dst + u);
  }
}

// One workgroup per 8 KB piece; block c of the sequential side pairs with
// block order[c] of the other side (skipped if outside [0, nblocks)).
__global__ void __launch_bounds__(kCopyThreads)
    block_copy_kernel(const u32x4* src, u32x4* dst, const int32_t* order, uint32_t nblocks,
                      uint32_t pieces, int scatter) {
  constexpr uint32_t kPiece = kCopyThreads * kCopyUnroll;  // units per workgroup
  const uint32_t c = blockIdx.x / pieces, p = blockIdx.x - c * pieces;
  const int32_t o = order[c];
  if (o < 0 || (uint32_t)o >= nblocks) return;
  const uint64_t seq = ((uint64_t)c * pieces + p) * kPiece;
  const uint64_t rnd = ((uint64_t)o * pieces + p) * kPiece;
  const u32x4* from = src + (scatter ? seq : rnd);
  u32x4* to = dst + (scatter ? rnd : seq);
  u32x4 v[kCopyUnroll];
#pragma unroll
  for (int k = 0; k < kCopyUnroll; ++k)
    v[k] = __builtin_nontemporal_load(from + k * kCopyThreads + threadIdx.x);
#pragma unroll
  for (int k = 0; k < kCopyUnroll; ++k)
    __builtin_nontemporal_store(v[k], to + k * kCopyThreads + threadIdx.x);
}

}  // namespace

extern "C" {

// Copies `nblocks` blocks of `block_bytes` (a multiple of 8192; addresses
// 16-byte aligned, the two regions disjoint): with scatter == 0 block
// order[c] of `src` to block c of `dst` (random reads), else block c of `src`
// to block order[c] of `dst` (random writes).  `order` is a device int32
// array [nblocks], a permutation of [0, nblocks) for the copy to be whole;
// entries outside that range are skipped.  DV_OK, DV_ERR_INVALID,
// DV_ERR_UNSUPPORTED (2^31 or more pieces of 8 KB), DV_ERR_HIP.
DV_API int dvb_block_copy(void* dst, const void* src, const int32_t* order, uint32_t nblocks,
                          uint32_t block_bytes, int scatter, void* stream) {
  const uintptr_t d = reinterpret_cast<uintptr_t>(dst), s = reinterpret_cast<uintptr_t>(src);
  const uint64_t piece = (uint64_t)kCopyThreads * kCopyUnroll * 16;
  if (!dst || !src || !order || (d & 15u) || (s & 15u) ||
      (reinterpret_cast<uintptr_t>(order) & 3u) || block_bytes == 0 || block_bytes % piece)
    return DV_ERR_INVALID;
  const uint64_t bytes = (uint64_t)nblocks * block_bytes;
  if (d < s + bytes && s < d + bytes && bytes) return DV_ERR_INVALID;
  if (nblocks == 0) return DV_OK;
  const uint64_t grid = (uint64_t)nblocks * (block_bytes / piece);
  if (grid >= (1ull << 31)) return DV_ERR_UNSUPPORTED;
  const u32x4* from = static_cast<const u32x4*>(src);
  u32x4* to = static_cast<u32x4*>(dst);
  uint32_t nb = nblocks, pieces = (uint32_t)(block_bytes / piece);
  int sc = scatter ? 1 : 0;
  void* args[] = {&from, &to, &order, &nb, &pieces, &sc};
  return hipLaunchKernel(reinterpret_cast<const void*>(&block_copy_kernel), dim3((uint32_t)grid),
                         dim3(kCopyThreads), args, 0, static_cast<hipStream_t>(stream)) ==
                 hipSuccess
             ? DV_OK
             : DV_ERR_HIP;
}

// Copies `bytes` (a multiple of 16; both addresses 16-byte aligned, the
// regions disjoint) from `src` to `dst` on `stream`.  DV_OK, DV_ERR_INVALID,
// DV_ERR_UNSUPPORTED (2^31 or more tiles of 8 KB), DV_ERR_HIP.
DV_API int dvb_plain_copy(void* dst, const void* src, uint64_t bytes, void* stream) {
  const uintptr_t d = reinterpret_cast<uintptr_t>(dst), s = reinterpret_cast<uintptr_t>(src);
  if (!dst || !src || (d & 15u) || (s & 15u) || (bytes & 15u)) return DV_ERR_INVALID;
  if (d < s + bytes && s < d + bytes && bytes) return DV_ERR_INVALID;
  if (bytes == 0) return DV_OK;
  const uint64_t units = bytes / 16;
  const uint64_t tiles = (units + kCopyThreads * kCopyUnroll - 1) / (kCopyThreads * kCopyUnroll);
  if (tiles >= (1ull << 31)) return DV_ERR_UNSUPPORTED;
  const u32x4* from = static_cast<const u32x4*>(src);
  u32x4* to = static_cast<u32x4*>(dst);
  uint64_t n = units;
  uint32_t t = (uint32_t)tiles;
  void* args[] = {&from, &to, &n, &t};
  return hipLaunchKernel(reinterpret_cast<const void*>(&plain_copy_kernel), dim3(t),
                         dim3(kCopyThreads), args, 0, static_cast<hipStream_t>(stream)) ==
                 hipSuccess
             ? DV_OK
             : DV_ERR_HIP;
}

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
