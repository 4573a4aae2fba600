/* Host twin of synth.fill_bytes (SplitMix64 counter mode, Steele, Lea and
 * Flood, OOPSLA 2014): 64-bit word k of a buffer filled with seed s is
 * mix(s + (k + 1) * GOLDEN).  Input generation only. */
#include <stdint.h>
#include <string.h>

static uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* Fill `nbytes` bytes starting at stream byte `first_byte`. */
void dvsynth_host_fill(void* out, uint64_t nbytes, uint64_t seed, uint64_t first_byte) {
  uint8_t* p = (uint8_t*)out;
  uint64_t j = first_byte;
  const uint64_t end = first_byte + nbytes;
  while (j < end && (j & 7)) { /* leading partial word */
    const uint64_t w = mix(seed + (j / 8 + 1) * 0x9E3779B97F4A7C15ull);
    *p++ = (uint8_t)(w >> (8 * (j & 7)));
    ++j;
  }
  for (; j + 8 <= end; j += 8, p += 8) {
    const uint64_t w = mix(seed + (j / 8 + 1) * 0x9E3779B97F4A7C15ull);
    memcpy(p, &w, 8);
  }
  if (j < end) { /* trailing partial word */
    const uint64_t w = mix(seed + (j / 8 + 1) * 0x9E3779B97F4A7C15ull);
    for (int i = 0; j < end; ++i, ++j) *p++ = (uint8_t)(w >> (8 * i));
  }
}
