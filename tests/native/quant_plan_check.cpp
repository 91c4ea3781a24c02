// Invariants of the two-launch dynamic quantizer's plan (quant_plan.hpp),
// checked on the host over many dense tensor sizes: the G code regions
// partition the 16-byte units, start on even units (whole NVFP4 blocks),
// and each holds the P 4-byte slots of the amax workgroups at 4-byte
// aligned offsets inside the code buffer; P is a multiple of 8, so the
// XCD-major slot order is a permutation of 0..P-1; every tensor from the
// small kernel's limit (3072 units of 16) to the plan's own limit gets a plan.
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "quant_plan.hpp"

int main() {
  long long checked = 0, planned = 0, bad = 0;
  const int cbs[2] = {8, 4};
  for (int f = 0; f < 2; ++f) {
    const int cb = cbs[f];
    for (int64_t n = 8; n <= qg::kSlotsMaxElements + 4096; n += (n < 100000 ? 8 : n < 1000000 ? 328 : 4104)) {
      if (cb == 4 && n % 16 != 0) continue;
      const qg::SlotsPlan p = qg::slots_plan(n, cb);
      ++checked;
      if (n > qg::kSlotsMaxElements) {
        if (p.G != 0) { ++bad; printf("plan past the limit: n %lld\n", (long long)n); }
        continue;
      }
      if (p.G == 0) {
        if (n >= 3072 * 16) { ++bad; printf("no plan: n %lld cb %d\n", (long long)n, cb); }
        continue;
      }
      ++planned;
      const int64_t units = n / 8, pairs = units / 2, code_bytes = (cb == 8) ? n : n / 2;
      if (p.P <= 0 || p.P % 8 != 0 || p.P > qg::kSlotsAmaxGroups || p.G > qg::kSlotsQuantGroups) {
        ++bad; printf("bad P/G: n %lld P %lld G %lld\n", (long long)n, (long long)p.P, (long long)p.G);
      }
      int64_t prev = 0;
      for (int64_t j = 0; j < p.G; ++j) {
        const int64_t lo = qg::slot_region_lo(pairs, j, p.G);
        const int64_t hi = (j + 1 == p.G) ? units : qg::slot_region_lo(pairs, j + 1, p.G);
        const bool ok = lo == prev && hi > lo && lo % 2 == 0 && (hi - lo) * cb >= 4 * p.P && (lo * cb) % 4 == 0 &&
                        lo * cb + 4 * p.P <= code_bytes && (cb == 8 || (hi - lo) % 2 == 0);
        if (!ok) {
          if (bad < 8) printf("region %lld of %lld: n %lld cb %d [%lld, %lld)\n", (long long)j, (long long)p.G,
                              (long long)n, cb, (long long)lo, (long long)hi);
          ++bad;
          break;
        }
        prev = hi;
      }
      if (prev != units) { ++bad; printf("regions end at %lld of %lld units\n", (long long)prev, (long long)units); }
      std::vector<char> seen(p.P, 0);
      for (int64_t b = 0; b < p.P; ++b) {
        const int64_t slot = (b % 8) * (p.P / 8) + b / 8;
        if (slot < 0 || slot >= p.P || seen[slot]) { ++bad; break; }
        seen[slot] = 1;
      }
    }
  }
  printf("checked %lld planned %lld violations %lld\n", checked, planned, bad);
  return bad != 0;
}
