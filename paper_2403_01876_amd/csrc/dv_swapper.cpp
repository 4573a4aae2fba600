// Microbatch swap scheduler: the round-robin protocol of the paper's
// microbatch swapping (Sec. 4.2.2, Figure "swapping").  All microbatches'
// caches live in pinned host memory; two device slots hold the microbatch
// being processed and the next one.  Before microbatch x's step the
// scheduler has prefetched x into a slot (swap-in on its input stream);
// after the step it swaps out only the part the step updated (swap-out on
// its output stream), which also frees the slot for the microbatch after
// next.  Data movement goes through dv_swap_in / dv_swap_out.
//
// The calls keep the slot bookkeeping and hand the swaps to a worker thread,
// which waits on the host for what each swap depends on (the step before a
// swap-out, the slot's previous swap-out before a swap-in) and then issues
// it.  Only the compute stream waits on the GPU, for residency.  A stream
// waiting on the GPU behind a copy on the SDMA engines stretched that copy
// (about 0.46 ms per waiting stream on an 82 ms swap-in), and the protocol
// had two to three such waiters per swap-in.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <condition_variable>
#include <deque>
#include <mutex>
#include <new>
#include <thread>
#include <utility>
#include <vector>

#include "../../include/dv.h"
#include "dv_host.h"

namespace {

constexpr int kStepEvents = 8;

struct Swap {
  bool in;            // swap-in (prefetch) or swap-out (update)
  int32_t mb, slot;
  std::vector<int32_t> t0, t1;
  int step_event;     // swap-out: index of the step's event, waited for first
  bool own_queue;     // which form of the side streams to use
};

}  // namespace

struct dv_swapper {
  dv_cache dev, host;
  std::vector<void*> dev_base, host_base;
  // Input and output streams, each in two forms (see create_side_streams):
  // [0] on HIP's shared hardware queues, [1] on a hardware queue of its own.
  // own_queue picks between them: the form for the compute stream of the
  // latest begin_step / end_step (shared queues until one has been seen).
  hipStream_t s_in[2] = {}, s_out[2] = {};
  bool own_queue = false;
  hipEvent_t resident[2] = {nullptr, nullptr};  // swap-in into the slot done
  hipEvent_t freed[2] = {nullptr, nullptr};     // slot's last occupant swapped out
  bool freed_recorded[2] = {false, false};
  hipEvent_t step_events[kStepEvents] = {};
  // Bookkeeping of the calls (host thread).
  int next_slot = 0;
  std::vector<int> slot_of;  // per host microbatch: slot it is in, or -1
  int occupant[2] = {-1, -1};
  // A slot may be refilled only after its occupant's step has ended (its
  // update is then queued for swap-out and `freed` orders the refill).
  bool done[2] = {true, true};
  // Worker state, under m.
  std::mutex m;
  std::condition_variable cv;
  std::deque<Swap> queue;
  std::vector<int> free_step_events;
  std::vector<uint64_t> issued;  // per host microbatch: swap-ins issued so far
  std::vector<uint64_t> asked;   // per host microbatch: swap-ins queued so far
  int busy = 0;
  int error = DV_OK;
  bool stop = false;
  int device = 0;
  std::thread worker;
};

namespace {

int hip_ok(hipError_t e) { return e == hipSuccess ? DV_OK : DV_ERR_HIP; }

void run_worker(dv_swapper* s) {
  (void)hipSetDevice(s->device);
  for (;;) {
    Swap w;
    {
      std::unique_lock<std::mutex> lk(s->m);
      s->cv.wait(lk, [s] { return s->stop || !s->queue.empty(); });
      if (s->queue.empty()) return;
      w = std::move(s->queue.front());
      s->queue.pop_front();
      ++s->busy;
    }
    int rc = DV_OK;
    if (w.in) {
      const hipStream_t in = s->s_in[w.own_queue ? 1 : 0];
      // The slot is refilled only after its previous occupant's update has
      // left; the worker recorded that swap-out, so the event is current.
      if (s->freed_recorded[w.slot] && hipEventSynchronize(s->freed[w.slot]) != hipSuccess)
        rc = DV_ERR_HIP;
      if (rc == DV_OK)
        rc = dv_swap_in(&s->host, w.mb, &s->dev, w.slot, 0, s->host.num_layers, nullptr,
                        w.t1.data(), in);
      if (rc == DV_OK) rc = hip_ok(hipEventRecord(s->resident[w.slot], in));
    } else {
      const hipStream_t out = s->s_out[w.own_queue ? 1 : 0];
      if (hipEventSynchronize(s->step_events[w.step_event]) != hipSuccess) rc = DV_ERR_HIP;
      {
        std::lock_guard<std::mutex> lk(s->m);
        s->free_step_events.push_back(w.step_event);
      }
      if (rc == DV_OK)
        rc = dv_swap_out(&s->dev, w.slot, &s->host, w.mb, 0, s->host.num_layers, w.t0.data(),
                         w.t1.data(), out);
      if (rc == DV_OK) rc = hip_ok(hipEventRecord(s->freed[w.slot], out));
      if (rc == DV_OK) s->freed_recorded[w.slot] = true;
    }
    {
      std::lock_guard<std::mutex> lk(s->m);
      if (rc != DV_OK && s->error == DV_OK) s->error = rc;
      if (w.in) ++s->issued[w.mb];
      --s->busy;
    }
    s->cv.notify_all();
  }
}

void release(dv_swapper* s) {
  if (s->worker.joinable()) {
    {
      std::lock_guard<std::mutex> lk(s->m);
      s->stop = true;
    }
    s->cv.notify_all();
    s->worker.join();
  }
  for (int i = 0; i < 2; ++i) {
    if (s->s_in[i]) (void)hipStreamSynchronize(s->s_in[i]);
    if (s->s_out[i]) (void)hipStreamSynchronize(s->s_out[i]);
  }
  for (int i = 0; i < 2; ++i) {
    if (s->resident[i]) (void)hipEventDestroy(s->resident[i]);
    if (s->freed[i]) (void)hipEventDestroy(s->freed[i]);
  }
  for (hipEvent_t e : s->step_events)
    if (e) (void)hipEventDestroy(e);
  for (int i = 0; i < 2; ++i) {
    if (s->s_in[i]) (void)hipStreamDestroy(s->s_in[i]);
    if (s->s_out[i]) (void)hipStreamDestroy(s->s_out[i]);
  }
  delete s;
}

void enqueue(dv_swapper* s, Swap&& w) {
  {
    std::lock_guard<std::mutex> lk(s->m);
    if (w.in) ++s->asked[w.mb];
    s->queue.push_back(std::move(w));
  }
  s->cv.notify_all();
}

// The ranges [t0, t1) fit both the device slots and the host mirrors, so
// the swap calls of a step can only fail in the runtime.
int check_ranges(const dv_swapper* s, const int32_t* t0, const int32_t* t1) {
  int rc = dv_packed_bytes(&s->dev, 0, s->dev.num_layers, t0, t1, nullptr);
  if (rc == DV_OK) rc = dv_packed_bytes(&s->host, 0, s->host.num_layers, t0, t1, nullptr);
  return rc;
}

// Whether the n regions [base[i], base[i] + bytes) are non-null, 16-byte
// aligned and pairwise disjoint.
bool disjoint_regions(void* const* base, int64_t n, uint64_t bytes) {
  std::vector<uintptr_t> a;
  a.reserve(n);
  for (int64_t i = 0; i < n; ++i) {
    const uintptr_t p = reinterpret_cast<uintptr_t>(base[i]);
    if (p == 0 || (p & 15u) != 0) return false;
    a.push_back(p);
  }
  std::sort(a.begin(), a.end());
  for (size_t i = 1; i < a.size(); ++i)
    if (a[i] - a[i - 1] < bytes) return false;
  return true;
}

// The scheduler orders its streams against the caller's with events; a
// compute stream under graph capture would turn those into graph nodes the
// scheduler's own streams cannot wait for, so such calls are refused.
int refuse_capture(void* stream, int* rc) {
  hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(static_cast<hipStream_t>(stream), &capture) != hipSuccess)
    return *rc = DV_ERR_HIP;
  return *rc = capture == hipStreamCaptureStatusNone ? DV_OK : DV_ERR_INVALID;
}

}  // namespace

extern "C" {

int dv_swapper_create(const dv_cache* dev_slots, const dv_cache* host, dv_swapper** out) {
  if (!dev_slots || !host || !out || !dev_slots->mb_base || !host->mb_base) return DV_ERR_INVALID;
  if (dev_slots->num_mb < 2 || host->num_mb < 1) return DV_ERR_INVALID;
  if (dev_slots->kind != DV_DENSE || host->kind != DV_DENSE) return DV_ERR_UNSUPPORTED;
  if (dev_slots->mem != DV_MEM_DEVICE || host->mem != DV_MEM_HOST_PINNED) return DV_ERR_INVALID;
  if (dev_slots->num_layers != host->num_layers || dev_slots->num_heads != host->num_heads ||
      dev_slots->head_dim != host->head_dim || dev_slots->batch != host->batch ||
      dev_slots->elem_bytes != host->elem_bytes)
    return DV_ERR_INVALID;
  uint64_t slot_bytes = 0, host_bytes = 0;
  int rc = dv_cache_bytes(dev_slots, &slot_bytes);
  if (rc != DV_OK) return rc;
  rc = dv_cache_bytes(host, &host_bytes);
  if (rc != DV_OK) return rc;
  // A prefetch writes one slot while the step reads the other, and swaps
  // move between mirrors and slots concurrently: the two slots must be
  // disjoint, and so must the host mirrors.
  if (!disjoint_regions(dev_slots->mb_base, 2, slot_bytes) ||
      !disjoint_regions(host->mb_base, host->num_mb, host_bytes))
    return DV_ERR_INVALID;
  dv_swapper* s = new (std::nothrow) dv_swapper();
  if (!s) return DV_ERR_INVALID;
  // Own copies of the base arrays: the caller's may go away after this call.
  s->dev = *dev_slots;
  s->host = *host;
  s->dev_base.assign(dev_slots->mb_base, dev_slots->mb_base + 2);
  s->host_base.assign(host->mb_base, host->mb_base + host->num_mb);
  s->dev.num_mb = 2;
  s->dev.mb_base = s->dev_base.data();
  s->host.mb_base = s->host_base.data();
  s->dev.block_table = s->host.block_table = nullptr;  // dense: never read
  s->dev.block_owner = s->host.block_owner = nullptr;
  s->slot_of.assign(host->num_mb, -1);
  s->issued.assign(host->num_mb, 0);
  s->asked.assign(host->num_mb, 0);
  // Streams at the default priority.
  if (hipGetDevice(&s->device) != hipSuccess ||
      dv::create_side_streams(&s->s_in[0], &s->s_in[1]) != hipSuccess ||
      dv::create_side_streams(&s->s_out[0], &s->s_out[1]) != hipSuccess) {
    release(s);
    return DV_ERR_HIP;
  }
  for (int i = 0; i < 2; ++i) {
    if (hipEventCreateWithFlags(&s->resident[i], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&s->freed[i], hipEventDisableTiming | hipEventBlockingSync) !=
            hipSuccess) {
      release(s);
      return DV_ERR_HIP;
    }
  }
  for (int i = 0; i < kStepEvents; ++i) {
    if (hipEventCreateWithFlags(&s->step_events[i],
                                hipEventDisableTiming | hipEventBlockingSync) != hipSuccess) {
      release(s);
      return DV_ERR_HIP;
    }
    s->free_step_events.push_back(i);
  }
  s->worker = std::thread(run_worker, s);
  *out = s;
  return DV_OK;
}

int dv_swapper_destroy(dv_swapper* s) {
  if (!s) return DV_ERR_INVALID;
  release(s);
  return DV_OK;
}

int dv_swapper_prefetch(dv_swapper* s, int32_t mb, const int32_t* len) {
  if (!s || !len) return DV_ERR_INVALID;
  if (mb < 0 || mb >= s->host.num_mb) return DV_ERR_RANGE;
  if (s->slot_of[mb] >= 0) return DV_OK;  // already resident or on its way
  const int slot = s->next_slot;
  const int prev = s->occupant[slot];
  if (!s->done[slot]) return DV_ERR_INVALID;  // occupant's step has not ended
  int rc = check_ranges(s, nullptr, len);
  if (rc != DV_OK) return rc;
  {
    std::lock_guard<std::mutex> lk(s->m);
    if (s->error != DV_OK) return s->error;
  }
  Swap w;
  w.in = true;
  w.mb = mb;
  w.slot = slot;
  w.t1.assign(len, len + s->host.batch);
  w.step_event = -1;
  w.own_queue = s->own_queue;
  enqueue(s, std::move(w));
  if (prev >= 0) s->slot_of[prev] = -1;
  s->occupant[slot] = mb;
  s->slot_of[mb] = slot;
  s->done[slot] = false;
  s->next_slot ^= 1;
  return DV_OK;
}

int dv_swapper_begin_step(dv_swapper* s, int32_t mb, void* compute_stream, int32_t* slot_out) {
  if (!s || !slot_out) return DV_ERR_INVALID;
  if (mb < 0 || mb >= s->host.num_mb) return DV_ERR_RANGE;
  const int slot = s->slot_of[mb];
  if (slot < 0) return DV_ERR_RANGE;  // not prefetched
  int rc = DV_OK;
  if (refuse_capture(compute_stream, &rc) != DV_OK) return rc;
  {
    // The swap-in must have been issued before its event can be waited for.
    std::unique_lock<std::mutex> lk(s->m);
    s->cv.wait(lk, [s, mb] { return s->issued[mb] == s->asked[mb] || s->error != DV_OK; });
    if (s->error != DV_OK) return s->error;
  }
  if (hipStreamWaitEvent(static_cast<hipStream_t>(compute_stream), s->resident[slot], 0) !=
      hipSuccess)
    return DV_ERR_HIP;
  s->own_queue = dv::pick_side(compute_stream, s->s_in[0], s->s_in[1]) == s->s_in[1];
  *slot_out = slot;
  return DV_OK;
}

int dv_swapper_end_step(dv_swapper* s, int32_t mb, void* compute_stream, const int32_t* t0,
                        const int32_t* t1) {
  if (!s || !t1) return DV_ERR_INVALID;
  if (mb < 0 || mb >= s->host.num_mb) return DV_ERR_RANGE;
  const int slot = s->slot_of[mb];
  if (slot < 0) return DV_ERR_RANGE;
  int rc = check_ranges(s, t0, t1);
  if (rc != DV_OK) return rc;
  if (refuse_capture(compute_stream, &rc) != DV_OK) return rc;
  int ev = -1;
  {
    std::unique_lock<std::mutex> lk(s->m);
    if (s->error != DV_OK) return s->error;
    s->cv.wait(lk, [s] { return !s->free_step_events.empty(); });
    ev = s->free_step_events.back();
    s->free_step_events.pop_back();
  }
  if (hipEventRecord(s->step_events[ev], static_cast<hipStream_t>(compute_stream)) !=
      hipSuccess) {
    std::lock_guard<std::mutex> lk(s->m);
    s->free_step_events.push_back(ev);
    return DV_ERR_HIP;
  }
  s->own_queue = dv::pick_side(compute_stream, s->s_out[0], s->s_out[1]) == s->s_out[1];
  Swap w;
  w.in = false;
  w.mb = mb;
  w.slot = slot;
  w.t0.assign(s->host.batch, 0);
  if (t0) w.t0.assign(t0, t0 + s->host.batch);
  w.t1.assign(t1, t1 + s->host.batch);
  w.step_event = ev;
  w.own_queue = s->own_queue;
  enqueue(s, std::move(w));
  s->done[slot] = true;
  return DV_OK;
}

int dv_swapper_sync(dv_swapper* s) {
  if (!s) return DV_ERR_INVALID;
  {
    std::unique_lock<std::mutex> lk(s->m);
    s->cv.wait(lk, [s] { return s->queue.empty() && s->busy == 0; });
  }
  for (int i = 0; i < 2; ++i)
    if (hipStreamSynchronize(s->s_in[i]) != hipSuccess ||
        hipStreamSynchronize(s->s_out[i]) != hipSuccess)
      return DV_ERR_HIP;
  std::lock_guard<std::mutex> lk(s->m);
  return s->error;
}

}  // extern "C"
