// quant_plan.hpp -- the launch plan of the two-launch dynamic quantizer of
// dense tensors (quantize.hip): how many amax workgroups P leave their maxima,
// into how many code regions G, and where region j begins. Host and device
// share it, and a host-only test checks its invariants over many sizes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

namespace qg {

constexpr int kSlotsAmaxLoads = 4;          // 16-byte loads per lane in flight
constexpr int64_t kSlotsAmaxGroups = 1024;  // P, a multiple of 8
constexpr int64_t kSlotsQuantGroups = 2048;
// The P x G scattered 4-byte slot stores grow with the tensor: at 4608 x
// 3072 (P = 1024 or 512, G = 1728 or 1024) the two launches took 17-22 us
// against the chain's 12.4 (GPU time from graph replays); at 256 x 3072 5.7
// against 6.7 us (FP8) and 6.4 against 7.7 (NVFP4), at 512 x 3072 6.2 against
// 7.0 and 6.8 against 7.9, level from 3 Mi elements on (1024 x 4096: 8.2
// against 7.8). Larger tensors take the chain.
constexpr int64_t kSlotsMaxElements = int64_t(3) << 20;

// First 16-byte unit (8 elements) of region j of g over `pairs` unit pairs:
// regions start on even units, so an NVFP4 16-block never straddles two.
__host__ __device__ inline int64_t slot_region_lo(int64_t pairs, int64_t j, int64_t g) { return 2 * (pairs * j / g); }

struct SlotsPlan {
  int64_t P;  // amax workgroups (a multiple of 8), one 4-byte slot each per region
  int64_t G;  // code regions = quantize workgroups; 0: the plan does not apply
};

// Plan for a dense tensor of n elements (n % 8 == 0), code bytes per unit
// cb = 8 (FP8) or 4 (NVFP4): every region's codes must hold the P slots.
inline SlotsPlan slots_plan(int64_t n, int cb) {
  if (n <= 0 || n % 8 != 0 || n > kSlotsMaxElements) return {0, 0};
  const int64_t units = n / 8, pairs = units / 2;
  const int64_t P =
      std::min<int64_t>(kSlotsAmaxGroups, ((units + 256 * kSlotsAmaxLoads - 1) / (256 * kSlotsAmaxLoads) + 7) / 8 * 8);
  const int64_t need = (4 * P + 2 * cb - 1) / (2 * cb);  // unit pairs per region that hold the slots
  const int64_t G = std::min<int64_t>(std::min<int64_t>(kSlotsQuantGroups, (units + 1023) / 1024), pairs / need);
  return {P, G >= 1 ? G : 0};
}

}  // namespace qg
