// pack.hip -- offline weight re-layout into matrix-core operand order.
//
// PTQ weights are quantized once (Sec. 4, quantization paragraph) and then
// laid out so that the GEMM streams them with no index arithmetic. The
// weight [n, k] is cut into panels of 32 rows (n rounded up to 32 with zero
// rows) and each panel into chunks of 128 reduction elements. Inside a chunk
// the 64 lanes of a wavefront each own one row r = l % 32 and one contiguous
// half of the chunk's reduction range, g = l / 32 -- the operand order of the
// 32x32 MFMAs once the reduction index is permuted the same way for both
// operands. A lane's bytes are split into 16-byte pieces h, stored as
// [h][lane][16 B], so that each piece is one contiguous 1 KiB wave access:
//   FP8  : 4096-byte chunk made of two 2048-byte steps of 64 reduction
//          elements; in step t, piece h of lane l = row r, bytes
//          64 t + 32 g + 16 h (each step is one self-contained MFMA operand);
//   NVFP4: 2048-byte code chunk, piece h of lane l = row r, bytes 32 g + 16 h;
//          block scales in their own region, 256 bytes per chunk = [row][8].
//   MXFP4: per 64-wide step t one 1024-byte image [lane][16 B], lane l = row
//          r, elements 64 t + 32 g .. + 31 (bytes 32 t + 16 g): exactly one
//          32-element scale block per lane, the operand of a scaled fp4 MFMA;
//          E8M0 scales in their own region, per 256-wide chunk c one run of
//          4 bytes per lane = the scales of the lane's blocks in steps
//          4c .. 4c + 3 (blocks 8c + 2s + g), read as one dword per lane.
//   MXFP8: 2048-byte step images like FP8, but lane half g and register
//          half h hold elements 64 t + 32 h + 16 g .. + 15: the block-scaled
//          fp8 instruction reads scale block h of a row from register half h
//          of both lane halves (its fp8 reduction order), so each of the
//          row's two 32-element scale blocks of the step must sit there; the
//          MXFP4 scale region (lane half g carries the scale of block 2 t + g).
// Chunks of one panel follow each other along k, so a panel is one
// contiguous stream. The header keeps format, n, k and the tensor scale
// (1.0 for the MX formats, which have none).
#include "common.hpp"
#include "kernels.hpp"

namespace qg {

__global__ void k_pack_header(uint8_t* packed, int fmt, int64_t n, int64_t k, const float* tscale) {
  uint32_t* h = reinterpret_cast<uint32_t*>(packed);
  h[0] = kPackMagic;
  h[1] = kPackVersion;
  h[2] = (uint32_t)fmt;
  h[3] = 0u;
  reinterpret_cast<int64_t*>(packed)[2] = n;
  reinterpret_cast<int64_t*>(packed)[3] = k;
  reinterpret_cast<float*>(packed + kPackScaleOffset)[0] = tscale ? *tscale : 1.0f;
}

__global__ void k_unpack_header(const uint8_t* packed, float* tscale) {
  if (tscale) *tscale = reinterpret_cast<const float*>(packed + kPackScaleOffset)[0];
}

// Canonical [n, row_bytes] byte offset of the 16-byte piece that packed
// piece `p` holds, or -1 for a padding row (see the layout above).
__device__ inline int64_t canon_piece(int fmt, int64_t p, int64_t n, int64_t k) {
  if (fmt == 3) {
    const int64_t steps = k / 64;
    const int64_t sc = p >> 6, l = p & 63;
    const int64_t panel = sc / steps, t = sc - panel * steps;
    const int64_t row = panel * 32 + (l & 31);
    if (row >= n) return -1;
    return row * (k / 2) + t * 32 + 16 * (l >> 5);
  }
  const int64_t kc_n = k / 128;
  const int per = (fmt == 1 || fmt == 4) ? 256 : 128;  // pieces per chunk
  const int64_t chunk = p / per, s = p - chunk * per;
  const int64_t panel = chunk / kc_n, kc = chunk - panel * kc_n;
  const int64_t h = s >> 6, l = s & 63;
  const int64_t row = panel * 32 + (l & 31);
  if (row >= n) return -1;
  if (fmt == 1) return row * k + kc * 128 + 64 * (h >> 1) + 32 * (l >> 5) + 16 * (h & 1);
  if (fmt == 4) return row * k + kc * 128 + 64 * (h >> 1) + 32 * (h & 1) + 16 * (l >> 5);
  return row * (k / 2) + kc * 64 + 32 * (l >> 5) + 16 * h;
}

// Canonical [n, k/16] offset of the 8-byte scale run that packed run `p`
// holds (run = one row of one chunk), or -1 for a padding row.
__device__ inline int64_t canon_scale_run(int64_t p, int64_t n, int64_t k) {
  const int64_t kc_n = k / 128;
  const int64_t chunk = p >> 5, r = p & 31;
  const int64_t panel = chunk / kc_n, kc = chunk - panel * kc_n;
  const int64_t row = panel * 32 + r;
  if (row >= n) return -1;
  return row * (k / 16) + kc * 8;
}

template <bool PACK>
__global__ void __launch_bounds__(256) k_pack_codes(int fmt, uint8_t* canon, uint8_t* packed_codes,
                                                    int64_t npieces, int64_t n, int64_t k) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= npieces) return;
  const int64_t c = canon_piece(fmt, p, n, k);
  if (PACK)
    reinterpret_cast<uint4*>(packed_codes)[p] =
        (c < 0) ? make_uint4(0u, 0u, 0u, 0u) : *reinterpret_cast<const uint4*>(canon + c);
  else if (c >= 0)
    *reinterpret_cast<uint4*>(canon + c) = reinterpret_cast<const uint4*>(packed_codes)[p];
}

template <bool PACK>
__global__ void __launch_bounds__(256) k_pack_scales(uint8_t* canon, uint8_t* packed_scales,
                                                     int64_t nruns, int64_t n, int64_t k) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= nruns) return;
  const int64_t c = canon_scale_run(p, n, k);
  if (PACK)
    reinterpret_cast<uint2*>(packed_scales)[p] =
        (c < 0) ? make_uint2(0u, 0u) : *reinterpret_cast<const uint2*>(canon + c);
  else if (c >= 0)
    *reinterpret_cast<uint2*>(canon + c) = reinterpret_cast<const uint2*>(packed_scales)[p];
}

// MXFP4 scale runs: run p = (panel, 256-wide chunk c, lane l); byte s of
// the run is the E8M0 scale of block 8c + 2s + g of row panel * 32 + r.
template <bool PACK>
__global__ void __launch_bounds__(256) k_pack_mx_scales(uint8_t* canon, uint8_t* packed_scales,
                                                        int64_t nruns, int64_t n, int64_t k) {
  const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (p >= nruns) return;
  const int64_t cn = k / 256;
  const int64_t pc = p >> 6, l = p & 63;
  const int64_t panel = pc / cn, c = pc - panel * cn;
  const int64_t row = panel * 32 + (l & 31), g = l >> 5;
  uint8_t* run = packed_scales + 4 * p;
  if (PACK) {
    uint32_t w = 0;
    if (row < n)
      for (int s = 0; s < 4; ++s) w |= (uint32_t)canon[row * (k / 32) + 8 * c + 2 * s + g] << (8 * s);
    *reinterpret_cast<uint32_t*>(run) = w;
  } else if (row < n) {
    const uint32_t w = *reinterpret_cast<const uint32_t*>(run);
    for (int s = 0; s < 4; ++s) canon[row * (k / 32) + 8 * c + 2 * s + g] = (uint8_t)(w >> (8 * s));
  }
}

static inline unsigned blocks_for(int64_t t) { return (unsigned)((t + 255) / 256); }

hipError_t launch_pack(int fmt, const uint8_t* codes, const uint8_t* bscale, const float* tscale,
                       int64_t n, int64_t k, uint8_t* packed, hipStream_t st) {
  hipLaunchKernelGGL(k_pack_header, dim3(1), dim3(1), 0, st, packed, fmt, n, k, tscale);
  const int64_t cb = packed_codes_bytes(fmt, n, k);
  if (cb == 0) return hipGetLastError();
  uint8_t* pc = packed + kPackHeader;
  const int64_t npieces = cb / 16;
  hipLaunchKernelGGL(k_pack_codes<true>, dim3(blocks_for(npieces)), dim3(256), 0, st, fmt,
                     const_cast<uint8_t*>(codes), pc, npieces, n, k);
  if (fmt == 3 || fmt == 4) {
    const int64_t nruns = padded_rows(n) * k / 128;
    hipLaunchKernelGGL(k_pack_mx_scales<true>, dim3(blocks_for(nruns)), dim3(256), 0, st,
                       const_cast<uint8_t*>(bscale), pc + cb, nruns, n, k);
  }
  if (fmt == 2) {
    const int64_t nruns = padded_rows(n) * k / 128;
    hipLaunchKernelGGL(k_pack_scales<true>, dim3(blocks_for(nruns)), dim3(256), 0, st,
                       const_cast<uint8_t*>(bscale), pc + cb, nruns, n, k);
  }
  return hipGetLastError();
}

hipError_t launch_unpack(int fmt, const uint8_t* packed, int64_t n, int64_t k, uint8_t* codes,
                         uint8_t* bscale, float* tscale, hipStream_t st) {
  hipLaunchKernelGGL(k_unpack_header, dim3(1), dim3(1), 0, st, packed, tscale);
  const int64_t cb = packed_codes_bytes(fmt, n, k);
  if (cb == 0) return hipGetLastError();
  uint8_t* pc = const_cast<uint8_t*>(packed) + kPackHeader;
  const int64_t npieces = cb / 16;
  hipLaunchKernelGGL(k_pack_codes<false>, dim3(blocks_for(npieces)), dim3(256), 0, st, fmt, codes,
                     pc, npieces, n, k);
  if (fmt == 3 || fmt == 4) {
    const int64_t nruns = padded_rows(n) * k / 128;
    hipLaunchKernelGGL(k_pack_mx_scales<false>, dim3(blocks_for(nruns)), dim3(256), 0, st, bscale,
                       pc + cb, nruns, n, k);
  }
  if (fmt == 2) {
    const int64_t nruns = padded_rows(n) * k / 128;
    hipLaunchKernelGGL(k_pack_scales<false>, dim3(blocks_for(nruns)), dim3(256), 0, st, bscale,
                       pc + cb, nruns, n, k);
  }
  return hipGetLastError();
}

}  // namespace qg
