// Device twin of synth.fill_bytes: fills a buffer with the SplitMix64
// counter-mode stream (Steele, Lea and Flood, OOPSLA 2014).  64-bit word k of
// a buffer filled with seed s is mix(s + (k + 1) * GOLDEN).  Input generation
// only: nothing here knows about KV-cache layouts.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// One 16-byte unit (two words) per thread per iteration, grid-stride.
__global__ void __launch_bounds__(256) fill_kernel(ulonglong2* __restrict__ out, uint64_t units,
                                                   uint64_t seed, uint64_t first_word) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t u = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; u < units; u += stride) {
    const uint64_t k = first_word + 2 * u;
    ulonglong2 v;
    v.x = mix(seed + (k + 1) * kGolden);
    v.y = mix(seed + (k + 2) * kGolden);
    out[u] = v;
  }
}

}  // namespace

extern "C" __attribute__((visibility("default"))) int dvsynth_fill(void* dev, uint64_t nbytes,
                                                                 uint64_t seed,
                                                                 uint64_t first_byte,
                                                                 void* stream) {
  if (dev == nullptr || (nbytes % 16) != 0 || (first_byte % 16) != 0 ||
      (reinterpret_cast<uintptr_t>(dev) % 16) != 0)
    return -1;
  if (nbytes == 0) return 0;
  const uint64_t units = nbytes / 16;
  uint64_t blocks = (units + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                     (ulonglong2*)dev, units, seed, first_byte / 8);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}
