// Host-side helpers shared by the C-ABI entry points, the swap scheduler and
// the streamer (no kernels here).
#pragma once

#include <hip/hip_runtime.h>

namespace dv {

// Side streams of the swap scheduler and the streamer.  HIP deals ordinary
// streams onto a pool of GPU_MAX_HW_QUEUES hardware queues, and two streams
// on one queue run in order: a side stream there serialises with the compute
// stream it should overlap (measured on MI355X: one creation in four, after
// the process has made a few dozen streams).  A stream with a CU mask gets a
// hardware queue of its own, but HIP creates it blocking, so it waits for the
// legacy null stream and the null stream for it.  create_side_streams makes one
// of each; pick_side() takes the own-queue stream unless the compute stream is
// the legacy null stream.
hipError_t create_side_streams(hipStream_t* shared_queue, hipStream_t* own_queue);
inline hipStream_t pick_side(void* compute_stream, hipStream_t shared_queue,
                             hipStream_t own_queue) {
  const hipStream_t c = static_cast<hipStream_t>(compute_stream);
  return (c == nullptr || c == hipStreamLegacy) ? shared_queue : own_queue;
}

}  // namespace dv
