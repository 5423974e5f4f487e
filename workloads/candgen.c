/*
 * Seeded candidate generator: route choices and 32-bit priorities.
 *
 * Shared input code: it feeds both the CPU oracle and the GPU evaluator and
 * holds none of the evaluation's arithmetic. It only draws numbers.
 *
 * Every value is the output of SplitMix64 (Steele, Lea and Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014) for a counter:
 *   r(key) = mix(seed + (key + 1) * 0x9e3779b97f4a7c15)
 * with mix the SplitMix64 output function, i.e. the (key+1)-th output of a
 * SplitMix64 stream seeded with `seed`. The counter of value j of candidate i
 * in stream t (1 = routes, 2 = priorities) is key = t<<60 | i<<28 | j, so any
 * candidate range can be generated independently of the rest.
 *   route choice = ((r >> 32) * options) >> 32   (Lemire, "Fast random
 *                  integer generation in an interval", TOMACS 2019; the
 *                  multiply-shift map of a 32-bit word onto [0, options))
 *   priority     = r >> 32
 */
#include <stddef.h>
#include <stdint.h>

static inline uint64_t sm64_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

static inline uint64_t draw(uint64_t seed, uint64_t stream, uint64_t i, uint64_t j) {
  uint64_t key = (stream << 60) | (i << 28) | j;
  return sm64_mix(seed + (key + 1) * 0x9e3779b97f4a7c15ull);
}

/* routes[count][route_stride] (options[e] choices for entry e; entries with
 * 0 options get 0) and prio[count][prio_stride], for candidates
 * first .. first+count-1. Returns 0, or -1 on bad arguments. */
int candgen_fill(uint64_t seed, int64_t first, int64_t count, int route_stride,
                 const int32_t *options, int prio_stride, uint8_t *routes, uint32_t *prio) {
  if (first < 0 || count < 0 || route_stride < 0 || prio_stride < 0) return -1;
  if ((uint64_t)(first + count) > (1ull << 32)) return -1;
  if (route_stride >= (1 << 28) || prio_stride >= (1 << 28)) return -1;
  for (int64_t k = 0; k < count; k++) {
    uint64_t i = (uint64_t)(first + k);
    uint8_t *rt = routes + (size_t)k * route_stride;
    uint32_t *pr = prio + (size_t)k * prio_stride;
    for (int e = 0; e < route_stride; e++) {
      uint32_t n = options[e] > 0 ? (uint32_t)options[e] : 0u;
      uint32_t w = (uint32_t)(draw(seed, 1, i, (uint64_t)e) >> 32);
      rt[e] = (uint8_t)(((uint64_t)w * n) >> 32);
    }
    for (int j = 0; j < prio_stride; j++) pr[j] = (uint32_t)(draw(seed, 2, i, (uint64_t)j) >> 32);
  }
  return 0;
}
