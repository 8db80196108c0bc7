// Division of 31-bit unsigned integers by a divisor fixed at launch time:
// one 32x32->64 multiply and a shift (Granlund and Montgomery, "Division by
// invariant integers using multiplication", PLDI 1994, with a numerator
// width of 31 bits): m = ceil(2^(31+l) / d), l = ceil(log2 d), and
// x / d = (x * m) >> (31 + l) for every 0 <= x < 2^31.
#ifndef TOPOEP_FASTDIV_H
#define TOPOEP_FASTDIV_H

#include <stdint.h>

#ifdef __HIPCC__
#define TOPOEP_HD __host__ __device__
#else
#define TOPOEP_HD
#endif

typedef struct FastDiv {
  uint32_t m;
  uint32_t sh;
} FastDiv;

// d >= 1
TOPOEP_HD inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < (uint64_t)d) ++l;
  FastDiv f;
  f.m = (uint32_t)((((uint64_t)1 << (31 + l)) + d - 1) / d);
  f.sh = 31 + l;
  return f;
}

// x < 2^31
TOPOEP_HD inline uint32_t fdiv(uint32_t x, FastDiv f) { return (uint32_t)(((uint64_t)x * f.m) >> f.sh); }

#endif
