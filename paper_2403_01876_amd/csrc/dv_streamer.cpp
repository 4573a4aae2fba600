// Background cache streamer: the paper's layer-by-layer prompt streaming and
// token streaming in parallel with computation (Sec. 4.1.1, optimisations 2
// and 3), driven by a background host thread as the paper describes.
//
// The compute thread calls dv_streamer_push after queuing the work that
// produces a region (a prompt layer, a decode step's token).  push records
// an event on the compute stream and hands a request to the worker thread;
// the worker waits for that event on the host, then, on the streamer's side
// stream, packs the region into device staging (the buffered copy of
// optimisation 1) and copies the staged chunk to its destination.  The side
// stream has a hardware queue of its own unless the compute stream is the
// legacy null stream.  The compute thread pays one event
// record and a queue push per region; the GPU overlaps the streaming with
// whatever the compute stream runs next.
//
// The copy to a host destination is issued in pitched form.  HIP runs a
// plain device-to-pinned-host copy as a blit kernel on the compute units,
// whose waves then sit on the PCIe writes and keep the compute kernels they
// should hide behind off the CUs (a 0.1 ms GEMM measured 2.2 ms beside one);
// the pitched copy goes to the SDMA engines and leaves the CUs to compute.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <new>
#include <thread>
#include <vector>

#include "../../include/dv.h"
#include "dv_host.h"

namespace {

constexpr int kEventPool = 64;
// Row width of the pitched host copies: whole rows go as one copy, the
// remainder as a one-row copy.
constexpr uint64_t kHostRow = 256u << 10;
// A dense source whose longest (sequence, head) run is at least this long
// goes to a host destination by the DMA engines directly, as the swaps do:
// one pitched copy per (layer, K|V, sequence) over the heads' runs, or one
// for the whole region when every sequence has the same range.  No pack
// kernel then shares the compute units with the compute stream.
constexpr uint64_t kDmaRunBytes = 64u << 10;

struct Request {
  int32_t l0, l1;
  std::vector<int32_t> t0, t1;
  uint64_t staging_off, dst_off, bytes;
  int event;  // index into the pool
  hipStream_t side;  // the side stream form for the pushing compute stream
};

}  // namespace

struct dv_streamer {
  dv_cache src;
  std::vector<void*> bases;
  std::vector<const int32_t*> tables;
  int32_t mb = 0;
  char* staging = nullptr;
  uint64_t staging_cap = 0;
  char* dst = nullptr;
  uint64_t dst_cap = 0;
  bool dst_host = false;  // destination in host memory: pitched (SDMA) copies
  int device = 0;
  // The side stream in two forms (see create_side_streams): [0] on HIP's
  // shared hardware queues, for a compute stream that is the legacy null
  // stream; [1] on a hardware queue of its own, for any other.
  hipStream_t side[2] = {};
  hipEvent_t events[kEventPool] = {};
  std::vector<int> free_events;
  std::deque<Request> queue;
  int busy = 0;  // requests taken by the worker and not yet complete
  int error = DV_OK;
  bool stop = false;
  std::mutex m;
  std::condition_variable cv;
  std::thread worker;
};

namespace {

hipError_t copy_out(dv_streamer* s, hipStream_t side, char* dst, const char* src, uint64_t n) {
  if (!s->dst_host) return hipMemcpyAsync(dst, src, n, hipMemcpyDefault, side);
  const uint64_t rows = n / kHostRow, tail = n - rows * kHostRow;
  if (rows) {
    const hipError_t e = hipMemcpy2DAsync(dst, kHostRow, src, kHostRow, kHostRow, rows,
                                          hipMemcpyDeviceToHost, side);
    if (e != hipSuccess) return e;
  }
  if (tail)
    return hipMemcpy2DAsync(dst + rows * kHostRow, tail, src + rows * kHostRow, tail, tail, 1,
                            hipMemcpyDeviceToHost, side);
  return hipSuccess;
}

// Whether request r goes by the DMA engines straight from the cache.
bool dma_direct(const dv_streamer* s, const Request& r) {
  if (!s->dst_host || s->src.kind != DV_DENSE) return false;
  const uint64_t tok = (uint64_t)s->src.head_dim * s->src.elem_bytes;
  int32_t longest = 0;
  for (int32_t b = 0; b < s->src.batch; ++b) longest = std::max(longest, r.t1[b] - r.t0[b]);
  return (uint64_t)longest * tok >= kDmaRunBytes;
}

// The region of request r, in the contiguous buffer's order, from the dense
// cache to dst + r.dst_off: row (slab, sequence b, head h) holds b's run of
// h, at pitch max_seq * tok in the cache and n_b * tok in the buffer.
hipError_t dma_gather(dv_streamer* s, const Request& r, hipStream_t side) {
  const dv_cache& c = s->src;
  const uint64_t tok = (uint64_t)c.head_dim * c.elem_bytes, B = c.batch, H = c.num_heads;
  const uint64_t row = (uint64_t)c.max_seq * tok;  // cache pitch of one (slab, b, h) run
  const char* cache = static_cast<const char*>(c.mb_base[s->mb]);
  char* out = s->dst + r.dst_off;
  uint64_t N = 0;
  bool uniform = true;
  for (uint64_t b = 0; b < B; ++b) {
    N += (uint64_t)(r.t1[b] - r.t0[b]);
    if (r.t0[b] != r.t0[0] || r.t1[b] != r.t1[0]) uniform = false;
  }
  if (uniform) {  // rows (slab, b, h) follow each other at one pitch on both sides
    const uint64_t n = (uint64_t)(r.t1[0] - r.t0[0]);
    if (n == 0) return hipSuccess;
    return hipMemcpy2DAsync(out, n * tok, cache + 2 * r.l0 * B * H * row + r.t0[0] * tok, row,
                            n * tok, 2 * (uint64_t)(r.l1 - r.l0) * B * H, hipMemcpyDeviceToHost,
                            side);
  }
  for (uint64_t slab = 2 * r.l0; slab < 2 * (uint64_t)r.l1; ++slab) {
    uint64_t p = 0;  // tokens of earlier sequences
    for (uint64_t b = 0; b < B; ++b) {
      const uint64_t n = (uint64_t)(r.t1[b] - r.t0[b]);
      if (n > 0) {
        const hipError_t e = hipMemcpy2DAsync(
            out + ((slab - 2 * r.l0) * N + p) * H * tok, n * tok,
            cache + (slab * B + b) * H * row + r.t0[b] * tok, row, n * tok, H,
            hipMemcpyDeviceToHost, side);
        if (e != hipSuccess) return e;
      }
      p += n;
    }
  }
  return hipSuccess;
}

void run_worker(dv_streamer* s) {
  (void)hipSetDevice(s->device);
  for (;;) {
    Request r;
    {
      std::unique_lock<std::mutex> lk(s->m);
      s->cv.wait(lk, [s] { return s->stop || !s->queue.empty(); });
      if (s->queue.empty()) return;  // stop requested and nothing left
      r = std::move(s->queue.front());
      s->queue.pop_front();
      ++s->busy;
    }
    int rc = DV_OK;
    // Nothing the worker queues ever waits on the GPU.  A packet held back
    // by a dependency sits as a blocked barrier in the side stream's
    // hardware queue, and on some of the queues HIP hands out such a barrier
    // added 20-30 us to every kernel of the compute stream while it waited.
    // So the worker waits on the host: for the producing work before it
    // queues the pack (rather than hipStreamWaitEvent), and for the copy
    // before it takes the next request (rather than queuing the next pack
    // behind a copy still on the SDMA engines).
    if (hipEventSynchronize(s->events[r.event]) != hipSuccess) rc = DV_ERR_HIP;
    {
      std::lock_guard<std::mutex> lk(s->m);
      s->free_events.push_back(r.event);
    }
    s->cv.notify_all();
    if (rc == DV_OK && r.bytes > 0) {
      if (dma_direct(s, r)) {
        if (dma_gather(s, r, r.side) != hipSuccess) rc = DV_ERR_HIP;
      } else {
        rc = dv_stream_out_prompt(&s->src, s->mb, r.l0, r.l1, r.t0.data(), r.t1.data(),
                                  s->staging + r.staging_off, r.bytes, nullptr, r.side);
        if (rc == DV_OK &&
            copy_out(s, r.side, s->dst + r.dst_off, s->staging + r.staging_off, r.bytes) !=
                hipSuccess)
          rc = DV_ERR_HIP;
      }
      if (rc == DV_OK && hipStreamSynchronize(r.side) != hipSuccess) rc = DV_ERR_HIP;
    }
    {
      std::lock_guard<std::mutex> lk(s->m);
      if (rc != DV_OK && s->error == DV_OK) s->error = rc;
      --s->busy;
    }
    s->cv.notify_all();
  }
}

void release(dv_streamer* s) {
  if (s->worker.joinable()) {
    {
      std::lock_guard<std::mutex> lk(s->m);
      s->stop = true;
    }
    s->cv.notify_all();
    s->worker.join();
  }
  for (hipStream_t x : s->side)
    if (x) (void)hipStreamSynchronize(x);
  for (hipEvent_t e : s->events)
    if (e) (void)hipEventDestroy(e);
  for (hipStream_t x : s->side)
    if (x) (void)hipStreamDestroy(x);
  delete s;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlaps(const void* a, uint64_t na, const void* b, uint64_t nb) {
  if (na == 0 || nb == 0) return false;
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

}  // namespace

extern "C" {

int dv_streamer_create(const dv_cache* src, int32_t mb, void* staging, uint64_t staging_cap,
                       void* dst, uint64_t dst_cap, dv_streamer** out) {
  if (!src || !out || !src->mb_base || !staging || !dst || !aligned16(staging) ||
      !aligned16(dst))
    return DV_ERR_INVALID;
  uint64_t bytes = 0;
  int rc = dv_cache_bytes(src, &bytes);
  if (rc != DV_OK) return rc;
  if (mb < 0 || mb >= src->num_mb) return DV_ERR_RANGE;
  // Staging, destination and the source microbatch must be disjoint: the
  // worker packs into staging and copies staging to the destination.
  if (overlaps(staging, staging_cap, src->mb_base[mb], bytes) ||
      overlaps(dst, dst_cap, src->mb_base[mb], bytes) ||
      overlaps(staging, staging_cap, dst, dst_cap))
    return DV_ERR_INVALID;
  // A paged source's block table is read by every pack: neither the staging
  // nor the destination may cover it.
  if (src->kind == DV_PAGED) {
    const void* table = src->block_table[mb];
    const uint64_t table_bytes = (uint64_t)src->batch * src->max_blocks * 4;
    if (overlaps(staging, staging_cap, table, table_bytes) ||
        overlaps(dst, dst_cap, table, table_bytes))
      return DV_ERR_INVALID;
  }
  dv_streamer* s = new (std::nothrow) dv_streamer();
  if (!s) return DV_ERR_INVALID;
  s->src = *src;
  s->bases.assign(src->mb_base, src->mb_base + src->num_mb);
  s->src.mb_base = s->bases.data();
  if (src->kind == DV_PAGED && src->block_table) {
    s->tables.assign(src->block_table, src->block_table + src->num_mb);
    s->src.block_table = s->tables.data();
  }
  s->src.block_owner = nullptr;  // packs only: the owner map is never used
  s->mb = mb;
  s->staging = static_cast<char*>(staging);
  s->staging_cap = staging_cap;
  s->dst = static_cast<char*>(dst);
  s->dst_cap = dst_cap;
  // Device memory reports hipMemoryTypeDevice; pinned host memory reports
  // hipMemoryTypeHost and pageable memory is unknown to HIP (an error here).
  hipPointerAttribute_t pa{};
  if (hipPointerGetAttributes(&pa, dst) == hipSuccess) {
    s->dst_host = pa.type == hipMemoryTypeHost || pa.type == hipMemoryTypeUnregistered;
  } else {
    (void)hipGetLastError();
    s->dst_host = true;
  }
  if (hipGetDevice(&s->device) != hipSuccess ||
      dv::create_side_streams(&s->side[0], &s->side[1]) != hipSuccess) {
    release(s);
    return DV_ERR_HIP;
  }
  for (int i = 0; i < kEventPool; ++i) {
    if (hipEventCreateWithFlags(&s->events[i], hipEventDisableTiming | hipEventBlockingSync) !=
        hipSuccess) {
      release(s);
      return DV_ERR_HIP;
    }
    s->free_events.push_back(i);
  }
  s->worker = std::thread(run_worker, s);
  *out = s;
  return DV_OK;
}

int dv_streamer_push(dv_streamer* s, void* compute_stream, int32_t l0, int32_t l1,
                     const int32_t* t0, const int32_t* t1, uint64_t staging_offset,
                     uint64_t dst_offset, uint64_t* out_bytes) {
  if (!s || !t1) return DV_ERR_INVALID;
  uint64_t bytes = 0;
  int rc = dv_packed_bytes(&s->src, l0, l1, t0, t1, &bytes);
  if (rc != DV_OK) return rc;
  if (out_bytes) *out_bytes = bytes;
  if (staging_offset % 16 != 0 || dst_offset % 16 != 0) return DV_ERR_INVALID;
  if (staging_offset > s->staging_cap || bytes > s->staging_cap - staging_offset ||
      dst_offset > s->dst_cap || bytes > s->dst_cap - dst_offset)
    return DV_ERR_SPACE;
  // The worker waits on the host for the event recorded below; under graph
  // capture that record is only a graph node, so the push is refused.
  hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(static_cast<hipStream_t>(compute_stream), &capture) != hipSuccess)
    return DV_ERR_HIP;
  if (capture != hipStreamCaptureStatusNone) return DV_ERR_INVALID;
  Request r;
  r.l0 = l0;
  r.l1 = l1;
  const int32_t B = s->src.batch;
  r.t0.assign(B, 0);
  if (t0) r.t0.assign(t0, t0 + B);
  r.t1.assign(t1, t1 + B);
  r.staging_off = staging_offset;
  r.dst_off = dst_offset;
  r.bytes = bytes;
  r.side = dv::pick_side(compute_stream, s->side[0], s->side[1]);
  {
    std::unique_lock<std::mutex> lk(s->m);
    if (s->error != DV_OK) return s->error;
    s->cv.wait(lk, [s] { return !s->free_events.empty(); });
    r.event = s->free_events.back();
    s->free_events.pop_back();
  }
  if (hipEventRecord(s->events[r.event], static_cast<hipStream_t>(compute_stream)) !=
      hipSuccess) {
    std::lock_guard<std::mutex> lk(s->m);
    s->free_events.push_back(r.event);
    return DV_ERR_HIP;
  }
  {
    std::lock_guard<std::mutex> lk(s->m);
    s->queue.push_back(std::move(r));
  }
  s->cv.notify_all();
  return DV_OK;
}

int dv_streamer_flush(dv_streamer* s) {
  if (!s) return DV_ERR_INVALID;
  {
    std::unique_lock<std::mutex> lk(s->m);
    s->cv.wait(lk, [s] { return s->queue.empty() && s->busy == 0; });
  }
  for (hipStream_t x : s->side)
    if (hipStreamSynchronize(x) != hipSuccess) return DV_ERR_HIP;
  std::lock_guard<std::mutex> lk(s->m);
  return s->error;
}

int dv_streamer_destroy(dv_streamer* s) {
  if (!s) return DV_ERR_INVALID;
  release(s);
  return DV_OK;
}

}  // extern "C"
