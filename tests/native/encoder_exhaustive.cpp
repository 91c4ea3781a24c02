// Exhaustive check of the library's E4M3 / E2M1 encoders (the __host__
// __device__ functions the quantize kernels use) against the CPU oracle's
// encoders, over every one of the 2^32 fp32 bit patterns. Built for the
// host only; prints the mismatch counts and the first mismatches.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "common.hpp"

extern "C" uint8_t qo_e4m3_encode(float v);
extern "C" uint8_t qo_e2m1_encode(float v);

int main() {
  unsigned long long bad8 = 0, bad4 = 0;
#pragma omp parallel for schedule(static) reduction(+ : bad8, bad4)
  for (long long i = 0; i < (1LL << 32); ++i) {
    const uint32_t u = (uint32_t)i;
    float f;
    memcpy(&f, &u, 4);
    const uint32_t a = qg::enc_e4m3(f), b = qo_e4m3_encode(f);
    const uint32_t c = qg::enc_e2m1(f), d = qo_e2m1_encode(f);
    if (a != b) {
      if (bad8 < 4) printf("e4m3 mismatch 0x%08x: lib %02x oracle %02x\n", u, a, b);
      ++bad8;
    }
    if (c != d) {
      if (bad4 < 4) printf("e2m1 mismatch 0x%08x: lib %x oracle %x\n", u, c, d);
      ++bad4;
    }
  }
  printf("e4m3_mismatches %llu\ne2m1_mismatches %llu\n", bad8, bad4);
  return (bad8 || bad4) ? 1 : 0;
}
