// gemm.hip -- quantized linear layers on gfx950 matrix cores.
//
// Y[m, n] = s_a * s_w * sum_k deq'(A)[m, k] * deq'(W)[n, k], the low-bit
// linears of the paper's denoising transformer (Sec. 4, quantization
// paragraph; Table 2) and of its small text encoder (weight-only).
//
// Three operand modes:
//   W8A8  (FP8 x FP8)    : codes go straight into v_mfma_f32_32x32x64_f8f6f4
//                          (OCP E4M3 operands; v_mfma_f32_16x16x128_f8f6f4 in
//                          the 288 x 192 tile kernel); tensor scales in the
//                          epilogue. Kernels: k_gemm_fp8_t288 and
//                          k_gemm_fp8_direct for large token counts, k_gemm_fp8
//                          for mid-size ones, the split-K k_gemm_splitk for few
//                          tokens (also from a bf16 activation quantized in the
//                          kernel: qg_linear_fp8).
//   W4A4  (NVFP4 x NVFP4): the E4M3 block scale changes every 16 reduction
//                          elements and is not a power of two, so it cannot
//                          ride in the hardware's per-32 power-of-two operand
//                          scale. An E2M1 code times its E4M3 block scale is
//                          exact in fp16 (<= 6 significant bits, magnitudes in
//                          [2^-10, 2688]), so both operands are expanded to
//                          fp16 in registers (v_cvt_scalef32_pk_f16_fp4 then
//                          v_pk_mul_f16) and fed to v_mfma_f32_32x32x16_f16.
//                          Kernels: k_gemm_nvfp4_direct for large token
//                          counts, the split-K k_gemm_splitk below that.
//   W4A16 (bf16 x NVFP4) : the weight is expanded the same way to bf16
//                          (exact) for v_mfma_f32_32x32x16_bf16.
//
// Reduction order. Both operands of a 32x32 MFMA are read in the same
// permuted reduction order, so each lane's operand bytes are contiguous runs
// (the order of the sum changes, its terms do not). Lane l covers row l % 32
// and half g = l / 32:
//   FP8  : in 64-wide step s of a 128-wide chunk, elements
//          [64 s + 32 g, 64 s + 32 g + 32) of its row (one 2 KiB operand
//          image per 32-row panel and step);
//   NVFP4, W4A16: elements [64 g, 64 g + 64) of its row over the chunk's
//          eight 16-wide steps.
//
// Tiling of the large-M W4A16 kernel (k_gemm): a workgroup of WM x WN
// wavefronts owns a (32 TM WM) x (32 TN WN) output tile; each wave owns
// TM x TN tiles of 32 x 32. Chunks of 128 are staged in LDS in the packed
// weight's lane-major order, so every LDS read is one contiguous 1 KiB wave
// access. Global loads run one chunk ahead; LDS is double buffered with one
// barrier per chunk.
//
// MFMA orientation: the weight panel is the MFMA A operand and the
// activation panel the B operand, so a lane ends with runs of 4 consecutive
// output columns of one output row.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace qg {

enum { MODE_FP8 = 1, MODE_NVFP4 = 2, MODE_W4A16 = 3 };

typedef float v16f __attribute__((ext_vector_type(16)));

struct GemmArgs {
  const uint8_t* a;         // FP8/NVFP4 codes or bf16 activations
  const uint8_t* a_bscale;  // NVFP4 block scales [m, k/16]
  const float* a_tscale;    // tensor scale of A (quantized modes)
  int64_t lda;              // elements between rows of A
  const uint8_t* w_codes;   // packed weight codes (after the header)
  const uint8_t* w_scales;  // packed block scales (NVFP4)
  const float* w_tscale;    // tensor scale of W (in the packed header)
  int m, n, k;
  void* y;
  int64_t ldy;
  int out_mode;             // OUT_BF16, OUT_F32, OUT_FP8 or OUT_NVFP4 (static output scale)
  const float* y_scale;     // decode scale of the FP8 output / tensor scale of the NVFP4 output
  uint8_t* y_bscale;        // NVFP4 output: E4M3 block scales [m, ldy / 16]
  int tiles_m, tiles_n;
};

constexpr int OUT_BF16 = 0, OUT_F32 = 1, OUT_FP8 = 2, OUT_NVFP4 = 3;

// Cache-policy operand of a buffer load: non-temporal, for data that one call
// reads exactly once (a streamed weight pool).
constexpr int kNT = 2;

// Reciprocal of the FP8 output's decode scale (the static quantizer's r).
__device__ __attribute__((always_inline)) inline float out_rscale(const GemmArgs& g) {
  if (g.out_mode != OUT_FP8) return 0.0f;
  const float s = *g.y_scale;
  return (s > 0.0f) ? __fdiv_rn(1.0f, s) : 0.0f;
}

// Two fp32 values to a pair of bf16 (low half = a), round to nearest even
// (one v_cvt_pk_bf16_f32).
__device__ __attribute__((always_inline)) inline uint32_t pk_bf16(float a, float b) {
  typedef float v2f_t __attribute__((ext_vector_type(2)));
  typedef __bf16 v2bf_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((v2f_t){a, b}, v2bf_t));
}

// Four consecutive outputs y[m][n .. n+3] (n % 4 == 0) in the output format:
// bf16 (RNE), fp32, or E4M3 codes of fl(y * r) (round to nearest even,
// saturating: the element step of the static quantizer, on the fp32 value).
// vec: the row pitch and base allow one aligned store.
__device__ __attribute__((always_inline)) inline void store4(const GemmArgs& g, int m, int n, float v0, float v1,
                                                             float v2, float v3, bool vec, float r) {
  if (g.out_mode == OUT_F32) {
    float* o = reinterpret_cast<float*>(g.y) + (int64_t)m * g.ldy + n;
    if (vec) *reinterpret_cast<float4*>(o) = make_float4(v0, v1, v2, v3);
    else { o[0] = v0; o[1] = v1; o[2] = v2; o[3] = v3; }
  } else if (g.out_mode == OUT_FP8) {
    const float y[4] = {__fmul_rn(v0, r), __fmul_rn(v1, r), __fmul_rn(v2, r), __fmul_rn(v3, r)};
    const uint32_t w = hw_e4m3x4(y);
    uint8_t* o = reinterpret_cast<uint8_t*>(g.y) + (int64_t)m * g.ldy + n;
    if (vec) *reinterpret_cast<uint32_t*>(o) = w;
    else { o[0] = (uint8_t)w; o[1] = (uint8_t)(w >> 8); o[2] = (uint8_t)(w >> 16); o[3] = (uint8_t)(w >> 24); }
  } else {
    uint16_t* o = reinterpret_cast<uint16_t*>(g.y) + (int64_t)m * g.ldy + n;
    const uint32_t w0 = pk_bf16(v0, v1), w1 = pk_bf16(v2, v3);
    if (vec) *reinterpret_cast<uint2*>(o) = make_uint2(w0, w1);
    else { o[0] = (uint16_t)w0; o[1] = (uint16_t)(w0 >> 16); o[2] = (uint16_t)w1; o[3] = (uint16_t)(w1 >> 16); }
  }
}

// Whether store4 may use one aligned store for every row of this output.
__device__ __attribute__((always_inline)) inline bool out_vec(const GemmArgs& g) {
  const int esz = g.out_mode == OUT_F32 ? 4 : g.out_mode == OUT_FP8 ? 1 : 2;
  return ((reinterpret_cast<uintptr_t>(g.y) & (4 * esz - 1)) == 0) && ((g.ldy & 3) == 0);
}

// NVFP4 output (qg_gemm_quant_nvfp4): the static NVFP4 quantizer's steps on
// the fp32 output values y (the values store4 would round), with the
// output's tensor decode scale s_t: d = fl(6 s_t); per 16-block of a row
// v = d > 0 ? fl(max|y| / d) : 0, s_b = E4M3(v) (saturating at 448),
// S = fl(e4m3(s_b) s_t), r = S > 0 ? fl(1/S) : 0, q = E2M1(fl(y r)). Codes
// two per byte (element 2i in the low nibble), rows of ldy / 2 bytes; block
// scales one byte per block, rows of ldy / 16 bytes.
__device__ __attribute__((always_inline)) inline float nv_out_d(const GemmArgs& g) {
  return g.out_mode == OUT_NVFP4 ? __fmul_rn(6.0f, *g.y_scale) : 0.0f;
}

// E4M3 block scale of a block whose largest |y| has the bit pattern amax,
// and the reciprocal r its elements are multiplied by.
__device__ __attribute__((always_inline)) inline uint32_t nv_block(uint32_t amax, float st, float d, float& r) {
  const float vb = (d > 0.0f) ? __fdiv_rn(u2f(amax), d) : 0.0f;
  const uint32_t sb = enc_e4m3(vb);
  const float S = __fmul_rn(dec_e4m3(sb), st);
  r = (S > 0.0f) ? __fdiv_rn(1.0f, S) : 0.0f;
  return sb;
}

// One 16-block of row m held by a lane pair in the MFMA output layout: lane
// half g holds columns n16 + 4 g + [0, 4) in v[0..3] and n16 + 8 + 4 g +
// [0, 4) in v[4..7]. Both lanes of the pair (l, l ^ 32) call this together.
// Lane half 0 stores bytes 0..3 of the block's codes, half 1 bytes 4..7.
__device__ __attribute__((always_inline)) inline void store_nv_pair(const GemmArgs& g, int m, int n16,
                                                                    const float (&v)[8], int gq, float st,
                                                                    float d) {
  uint32_t am = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) am = max(am, f2u(v[j]) & 0x7FFFFFFFu);
  am = max(am, (uint32_t)__shfl_xor((int)am, 32));
  float r;
  const uint32_t sb = nv_block(am, st, d, r);
  float y[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) y[j] = __fmul_rn(v[j], r);
  // half 0 holds the bytes of elements 0-3 and 8-11 ([b0 b1 b4 b5]), half 1
  // those of 4-7 and 12-15 ([b2 b3 b6 b7]); one exchange makes them runs
  const uint32_t w = hw_e2m1x8(y);
  const uint32_t x = (uint32_t)__shfl_xor((int)w, 32);
  const uint32_t out = gq ? ((x >> 16) | (w & 0xFFFF0000u)) : ((w & 0xFFFFu) | (x << 16));
  uint8_t* row = reinterpret_cast<uint8_t*>(g.y) + (int64_t)m * (g.ldy >> 1);
  *reinterpret_cast<uint32_t*>(row + (n16 >> 1) + 4 * gq) = out;
  if (gq == 0) g.y_bscale[(int64_t)m * (g.ldy >> 4) + (n16 >> 4)] = (uint8_t)sb;
}

// One 16-block of row m held by four consecutive lanes, lane n / 4 % 4
// holding columns n .. n + 3 in v (the split-K kernels' reduction layout).
// All four lanes call this together.
__device__ __attribute__((always_inline)) inline void store_nv_quad(const GemmArgs& g, int m, int n,
                                                                    const float (&v)[4], float st, float d) {
  uint32_t am = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) am = max(am, f2u(v[j]) & 0x7FFFFFFFu);
  am = max(am, (uint32_t)__shfl_xor((int)am, 1));
  am = max(am, (uint32_t)__shfl_xor((int)am, 2));
  float r;
  const uint32_t sb = nv_block(am, st, d, r);
  uint32_t w = 0;
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, __fmul_rn(v[0], r), __fmul_rn(v[1], r), 1.0f, 0);
  w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, __fmul_rn(v[2], r), __fmul_rn(v[3], r), 1.0f, 1);
  uint8_t* row = reinterpret_cast<uint8_t*>(g.y) + (int64_t)m * (g.ldy >> 1);
  *reinterpret_cast<uint16_t*>(row + (n >> 1)) = (uint16_t)w;
  if ((n & 15) == 0) g.y_bscale[(int64_t)m * (g.ldy >> 4) + (n >> 4)] = (uint8_t)sb;
}

// LDS bytes per 32-row panel per 128-chunk of the large-M W4A16 kernel:
// bf16 activations (A), weight codes (B) and decoded weight block scales.
template <int MODE> struct Lds;
template <> struct Lds<MODE_W4A16> { static constexpr int A = 8192, B = 2048, AS = 0, BS = 1024; };

// 8 E2M1 codes (one dword) times an fp16 block scale -> 8 fp16 (exact).
__device__ inline v8h dequant8_f16(uint32_t w, _Float16 sc) {
  const v2h s2 = {sc, sc};
  const v2h p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 0) * s2;
  const v2h p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 1) * s2;
  const v2h p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 2) * s2;
  const v2h p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 1.0f, 3) * s2;
  return (v8h){p0.x, p0.y, p1.x, p1.y, p2.x, p2.y, p3.x, p3.y};
}

// 8 E2M1 codes times an fp32 block scale -> 8 bf16 (exact, so the top half
// of the fp32 product is already the bf16 value): one conversion, two
// multiplies and one byte permute per pair.
__device__ inline v4i dequant8_bf16(uint32_t w, float sc) {
  const auto t0 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 0);
  const auto t1 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 1);
  const auto t2 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 2);
  const auto t3 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 3);
  v4i o;
  o[0] = (int)__builtin_amdgcn_perm(f2u(t0[1] * sc), f2u(t0[0] * sc), 0x07060302u);
  o[1] = (int)__builtin_amdgcn_perm(f2u(t1[1] * sc), f2u(t1[0] * sc), 0x07060302u);
  o[2] = (int)__builtin_amdgcn_perm(f2u(t2[1] * sc), f2u(t2[0] * sc), 0x07060302u);
  o[3] = (int)__builtin_amdgcn_perm(f2u(t3[1] * sc), f2u(t3[0] * sc), 0x07060302u);
  return o;
}

// Output tile order: consecutive workgroups are dealt round-robin to the 8
// XCDs (each with its own L2), so the linear id is remapped to give every XCD
// a contiguous band of tiles, walked in groups of GROUP_M tile rows so that
// concurrently running tiles share activation rows and weight panels.
__device__ inline void tile_coords(int id, int tiles_m, int tiles_n, int& bm, int& bn) {
  const int total = tiles_m * tiles_n;
  int t = id;
  if (total % 8 == 0) t = (id & 7) * (total >> 3) + (id >> 3);
  constexpr int GROUP_M = 4;
  const int per_group = GROUP_M * tiles_n;
  const int grp = t / per_group;
  const int first_m = grp * GROUP_M;
  const int rows = min(GROUP_M, tiles_m - first_m);
  const int in = t - grp * per_group;
  bm = first_m + in % rows;
  bn = in / rows;
}

template <int MODE, int WM, int WN, int TM, int TN, int DEPTH>
__global__ void __launch_bounds__(64 * WM * WN) k_gemm(GemmArgs g) {
  static_assert(MODE == MODE_W4A16, "W8A8 and W4A4 have kernels of their own");
  constexpr int NT = 64 * WM * WN;
  constexpr int PA = TM * WM, PB = TN * WN;  // 32-row panels per tile
  constexpr int BM = 32 * PA, BN = 32 * PB;
  constexpr int A_BYTES = PA * Lds<MODE>::A, B_BYTES = PB * Lds<MODE>::B;
  constexpr int AS_BYTES = PA * Lds<MODE>::AS, BS_BYTES = PB * Lds<MODE>::BS;
  constexpr int STAGE = A_BYTES + B_BYTES + AS_BYTES + BS_BYTES;
  // 16-byte pieces per stage of each operand; one 8-byte scale run per weight row
  constexpr int NPA = A_BYTES / 16, NPB = B_BYTES / 16;
  static_assert(NPA % NT == 0 && NPB % NT == 0, "piece count must divide the thread count");
  constexpr int RA = NPA / NT, RB = NPB / NT;
  constexpr int NSB = BN;
  constexpr int RSB = (NSB + NT - 1) / NT;
  constexpr int PIECES_A = Lds<MODE>::A / 16, PIECES_B = Lds<MODE>::B / 16;  // per panel chunk

  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  int bm, bn;
  tile_coords(blockIdx.x, g.tiles_m, g.tiles_n, bm, bn);
  const int m0 = bm * BM, n0 = bn * BN;
  const int kcn = g.k >> 7;
  const int npanels_w = (g.n + 31) >> 5;

  // Global reads go through buffer descriptors (base + byte count in SGPRs):
  // each piece a thread copies is one 32-bit offset, the chunk advance is the
  // scalar offset, and rows or panels past the end fall outside the buffer's
  // range, which the hardware turns into zeros -- no branches, no clamping.
  const int64_t a_row_bytes = 2 * g.lda;
  const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a), 0, (int)((int64_t)g.m * a_row_bytes), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * kcn * Lds<MODE>::B), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_sb = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, (int)((int64_t)npanels_w * kcn * 256), 0x00020000);

  // Activation pieces are read row-contiguously (CPR 16-byte pieces cover a
  // row's chunk bytes, so 64 lanes read 64 / CPR whole row runs) and written
  // to the lane-major LDS image through an XOR swizzle: piece c of row r
  // belongs to lane (r, g = c / HALF) as its piece h = c % HALF and lands in
  // slot ((r + 32 g) ^ c) of LDS block h. The lanes of one row then hit
  // distinct LDS banks, and the operand read of lane l (slot l ^ (h + HALF g))
  // stays a conflict-free 1 KiB access.
  constexpr int CPR = 16;
  constexpr int HALF = CPR / 2;
  uint32_t oa[RA];
  uint32_t la[RA];
#pragma unroll
  for (int it = 0; it < RA; ++it) {
    const int q = it * NT + tid;
    const int p = q / (32 * CPR), rr = (q / CPR) % 32, c = q % CPR;
    const uint32_t row = (uint32_t)(m0 + 32 * p + rr);
    oa[it] = (row < (uint32_t)g.m) ? row * (uint32_t)a_row_bytes + 16u * c : 0x80000000u;
    const int gg = c / HALF, h = c % HALF;
    la[it] = (uint32_t)(p * Lds<MODE>::A + h * 1024 + (((rr + 32 * gg) ^ c) * 16));
  }
  uint32_t ob[RB];
#pragma unroll
  for (int it = 0; it < RB; ++it) {
    const int q = it * NT + tid;
    const int p = q / PIECES_B, s = q - p * PIECES_B;
    const uint32_t panel = (uint32_t)((n0 >> 5) + p);
    ob[it] = (panel < (uint32_t)npanels_w) ? panel * (uint32_t)(kcn * Lds<MODE>::B) + 16u * s : 0x80000000u;
  }
  uint32_t osb[RSB > 0 ? RSB : 1];
#pragma unroll
  for (int it = 0; it < RSB; ++it) {
    const int q = it * NT + tid;
    const uint32_t panel = (uint32_t)((n0 >> 5) + (q >> 5));
    osb[it] = (q < NSB && panel < (uint32_t)npanels_w) ? panel * (uint32_t)(kcn * 256) + 8u * (q & 31) : 0x80000000u;
  }

  struct Regs {
    v4i a[RA > 0 ? RA : 1];
    v4i b[RB > 0 ? RB : 1];
    v2i sb[RSB > 0 ? RSB : 1];
  };

  // ---- global -> registers for chunk kc
  auto load_chunk = [&](Regs& R, int kc) {
    const int sa_off = kc * 256;
#pragma unroll
    for (int it = 0; it < RA; ++it) R.a[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[it], sa_off, 0);
#pragma unroll
    for (int it = 0; it < RB; ++it) R.b[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[it], kc * Lds<MODE>::B, 0);
#pragma unroll
    for (int it = 0; it < RSB; ++it) R.sb[it] = __builtin_amdgcn_raw_buffer_load_b64(rs_sb, osb[it], kc * 256, 0);
  };

  // ---- registers -> LDS stage (block scales expanded once per workgroup)
  auto store_chunk = [&](const Regs& R, uint8_t* st) {
    uint8_t* sa = st;
    uint8_t* sb = st + A_BYTES;
    uint8_t* ssb = st + A_BYTES + B_BYTES + AS_BYTES;
#pragma unroll
    for (int it = 0; it < RA; ++it) *reinterpret_cast<v4i*>(sa + la[it]) = R.a[it];
#pragma unroll
    for (int it = 0; it < RB; ++it) reinterpret_cast<v4i*>(sb)[it * NT + tid] = R.b[it];
#pragma unroll
    for (int it = 0; it < RSB; ++it) {
      const int q = it * NT + tid;
      if (q < NSB) {
        const uint32_t w[2] = {(uint32_t)R.sb[it].x, (uint32_t)R.sb[it].y};
        float f[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = dec_e4m3((w[j >> 2] >> (8 * (j & 3))) & 0xFFu);
        reinterpret_cast<float4*>(ssb)[2 * q] = make_float4(f[0], f[1], f[2], f[3]);
        reinterpret_cast<float4*>(ssb)[2 * q + 1] = make_float4(f[4], f[5], f[6], f[7]);
      }
    }
  };

  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  // ---- MFMAs over one staged chunk
  auto compute_chunk = [&](const uint8_t* st) {
    const uint8_t* sa = st;
    const uint8_t* sb = st + A_BYTES;
    const uint8_t* ssb = st + A_BYTES + B_BYTES + AS_BYTES;
    const int r = lane & 31, gq = lane >> 5;
    {
      uint4 cb[TN][2];
      float4 scb[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int p = wn * TN + j;
        cb[j][0] = *reinterpret_cast<const uint4*>(sb + p * 2048 + lane * 16);
        cb[j][1] = *reinterpret_cast<const uint4*>(sb + p * 2048 + 1024 + lane * 16);
        scb[j] = *reinterpret_cast<const float4*>(ssb + p * 1024 + r * 32 + 16 * gq);
      }
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        v8bf fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          fa[i] = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4i*>(sa + (wm * TM + i) * 8192 + s * 1024 + ((lane ^ (s + 8 * gq)) * 16)));
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const uint4 c = cb[j][s >> 2];
          const uint32_t w = ((s & 3) == 0) ? c.x : ((s & 3) == 1) ? c.y : ((s & 3) == 2) ? c.z : c.w;
          const float sc = ((s >> 1) == 0) ? scb[j].x : ((s >> 1) == 1) ? scb[j].y : ((s >> 1) == 2) ? scb[j].z : scb[j].w;
          fb[j] = __builtin_bit_cast(v8bf, dequant8_bf16(w, sc));
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
      }
    }
  };

  // ---- main loop. DEPTH 2: chunk kc+2 loads while chunk kc multiplies and
  // chunk kc+1's registers (loaded one iteration earlier) go to the free LDS
  // buffer. DEPTH 1: chunk kc+1 loads while chunk kc multiplies.
  if (kcn > 0) {
    if (DEPTH == 2) {
      Regs R0, R1;
      load_chunk(R0, 0);
      if (kcn > 1) load_chunk(R1, 1);
      store_chunk(R0, smem);
      __syncthreads();
      int kc = 0;
      for (; kc + 1 < kcn; kc += 2) {
        if (kc + 2 < kcn) load_chunk(R0, kc + 2);
        compute_chunk(smem);
        store_chunk(R1, smem + STAGE);
        __syncthreads();
        if (kc + 3 < kcn) load_chunk(R1, kc + 3);
        compute_chunk(smem + STAGE);
        if (kc + 2 < kcn) store_chunk(R0, smem);
        __syncthreads();
      }
      if (kc < kcn) compute_chunk(smem);  // odd chunk count: the last one sits in buffer 0
    } else {
      Regs R;
      load_chunk(R, 0);
      store_chunk(R, smem);
      __syncthreads();
      for (int kc = 0; kc < kcn; ++kc) {
        const bool more = kc + 1 < kcn;
        if (more) load_chunk(R, kc + 1);
        compute_chunk(smem + (kc & 1) * STAGE);
        if (more) store_chunk(R, smem + ((kc + 1) & 1) * STAGE);
        __syncthreads();
      }
    }
  }

  // ---- epilogue: scale, round, store. Lane holds Y[m][n + 8 q .. +3] for q = 0..3.
  float c = *g.w_tscale;
  const bool vec = out_vec(g);
  const float ry = out_rscale(g);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + (wm * TM + i) * 32 + (lane & 31);
    if (m >= g.m) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int n = n0 + (wn * TN + j) * 32 + 8 * qd + 4 * (lane >> 5);
        if (n >= g.n) continue;
        store4(g, m, n, acc[i][j][4 * qd] * c, acc[i][j][4 * qd + 1] * c, acc[i][j][4 * qd + 2] * c,
               acc[i][j][4 * qd + 3] * c, vec, ry);
      }
    }
  }
}

// Buffer descriptor of the activation codes: exactly the bytes a caller must
// provide, (m - 1) * lda + k, so reads past the last row's k bytes are out of
// range and return zeros. All offsets go in the per-lane offset, which is what
// the hardware range-checks.
__device__ __attribute__((always_inline)) inline __amdgpu_buffer_rsrc_t rsrc_a_fp8(const GemmArgs& g) {
  const int64_t bytes = (g.m > 0) ? (int64_t)(g.m - 1) * g.lda + g.k : 0;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(g.a), 0, (int)bytes, 0x00020000);
}

// Epilogue shared by the MFMA-layout kernels: a wave's TM x TN accumulator tiles,
// first output row mw and column nw, scaled by c and rounded to the output
// type. Lane l holds Y[mw + 32 i + l % 32][nw + 32 j + 8 q + 4 (l / 32) + e].
template <int TM, int TN>
__device__ __attribute__((always_inline)) inline void store_tiles(const GemmArgs& g, const v16f (&acc)[TM][TN],
                                                                  int mw, int nw, int lane, float c) {
  if (g.out_mode == OUT_NVFP4) {
    const float st = *g.y_scale, d = nv_out_d(g);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = mw + 32 * i + (lane & 31);
      if (m >= g.m) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int n16 = nw + 32 * j + 16 * b;
          if (n16 >= g.n) continue;
          float v[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = acc[i][j][8 * b + e] * c;
          store_nv_pair(g, m, n16, v, lane >> 5, st, d);
        }
    }
    return;
  }
  const bool vec = out_vec(g);
  const float ry = out_rscale(g);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = mw + 32 * i + (lane & 31);
    if (m >= g.m) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int n = nw + 32 * j + 8 * qd + 4 * (lane >> 5);
        if (n >= g.n) continue;
        store4(g, m, n, acc[i][j][4 * qd] * c, acc[i][j][4 * qd + 1] * c, acc[i][j][4 * qd + 2] * c,
               acc[i][j][4 * qd + 3] * c, vec, ry);
      }
    }
  }
}

// ---------------------------------------------------------------- FP8 (W8A8), few tokens
// Four wavefronts (one per SIMD) on a (64 TM) x (64 TN) tile, each owning
// TM x TN MFMA tiles of 32 x 32 (used with TM = 1, TN = 2: 64 x 128 tiles,
// so that a short activation still spreads over many workgroups). The
// reduction advances in steps of 64 --
// one v_mfma_f32_32x32x64_f8f6f4 per tile and step -- through three LDS
// stages, so that LDS traffic is spread evenly over every step instead of
// bursting after a barrier:
//   during step t: the MFMAs of step t run on fragments already in registers,
//   interleaved with the LDS reads of step t+1's fragments (stage (t+1) % 3,
//   written during step t-1), the LDS writes of step t+2 (registers loaded
//   two steps ago) and the global loads of step t+4; one barrier per step.
// A stage is rewritten two steps after it was last read, so one barrier per
// step separates every write from the reads before and after it. The loop
// body has no branches: loads past the last step get an out-of-range offset
// and read zeros, and LDS traffic past the end lands in stages nobody reads
// again. The packed weight keeps each 64-wide step of a 32-row
// panel as one contiguous 2 KiB operand image; activation rows are read
// row-contiguously and stored through the XOR swizzle of k_gemm.
template <int TM, int TN>
__global__ void __launch_bounds__(256) k_gemm_fp8(GemmArgs g) {
  constexpr int NT = 256;
  constexpr int PA = 2 * TM, PB = 2 * TN;                 // 32-row panels per tile
  constexpr int BM = 32 * PA, BN = 32 * PB;
  constexpr int A_BYTES = PA * 2048, B_BYTES = PB * 2048, STAGE = A_BYTES + B_BYTES;
  constexpr int NPA = A_BYTES / 16, NPB = B_BYTES / 16;   // 16-byte pieces per step
  static_assert(NPA % NT == 0 && NPB % NT == 0, "every thread copies whole pieces: no guards in the loop");
  constexpr int RA = NPA / NT, RB = NPB / NT;
  constexpr int NS = 3;                                   // LDS stages
  __shared__ __attribute__((aligned(16))) uint8_t smem[NS * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int gq = lane >> 5;
  int bm, bn;
  tile_coords(blockIdx.x, g.tiles_m, g.tiles_n, bm, bn);
  const int m0 = bm * BM, n0 = bn * BN;
  const int steps = g.k >> 6;
  const int npanels_w = (g.n + 31) >> 5;
  const __amdgpu_buffer_rsrc_t rs_a = rsrc_a_fp8(g);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * steps * 2048), 0x00020000);

  // activation piece c (0..3) of row rr: bytes [16 c, 16 c + 16) of the step,
  // lane half g = c / 2, piece h = c % 2, swizzled slot (rr + 32 g) ^ c
  uint32_t oa[RA], la[RA], ob[RB], lb[RB];
#pragma unroll
  for (int it = 0; it < RA; ++it) {
    const int q = it * NT + tid;
    const int p = q >> 7, rr = (q >> 2) & 31, c = q & 3;
    const uint32_t row = (uint32_t)(m0 + 32 * p + rr);
    oa[it] = (row < (uint32_t)g.m) ? row * (uint32_t)g.lda + 16u * c : 0x80000000u;
    la[it] = (uint32_t)(p * 2048 + (c & 1) * 1024 + (((rr + 32 * (c >> 1)) ^ c) * 16));
  }
#pragma unroll
  for (int it = 0; it < RB; ++it) {
    const int q = it * NT + tid;
    const uint32_t panel = (uint32_t)((n0 >> 5) + (q >> 7));
    ob[it] = (panel < (uint32_t)npanels_w) ? panel * (uint32_t)(steps * 2048) + 16u * (q & 127) : 0x80000000u;
    lb[it] = (uint32_t)(A_BYTES + 16 * q);
  }

  v4i ra[2][RA], rb[2][RB];
  // offsets of steps past the last one get the top bit: out of range for any base
  auto gload = [&](int set, int t) __attribute__((always_inline)) {
    const uint32_t hi = t < steps ? 0u : 0x80000000u;
#pragma unroll
    for (int it = 0; it < RA; ++it) ra[set][it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, (oa[it] + t * 64) | hi, 0, 0);
#pragma unroll
    for (int it = 0; it < RB; ++it) rb[set][it] = __builtin_amdgcn_raw_buffer_load_b128(rs_b, (ob[it] + t * 2048) | hi, 0, 0);
  };
  auto lds_write = [&](int set, uint8_t* st) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < RA; ++it) *reinterpret_cast<v4i*>(st + la[it]) = ra[set][it];
#pragma unroll
    for (int it = 0; it < RB; ++it) *reinterpret_cast<v4i*>(st + lb[it]) = rb[set][it];
  };
  v8i fa[2][TM], fb[2][TN];
  auto frag_read = [&](int set, const uint8_t* st) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const uint8_t* p = st + (wm * TM + i) * 2048;
      const v4i lo = *reinterpret_cast<const v4i*>(p + ((lane ^ (2 * gq)) * 16));
      const v4i hi = *reinterpret_cast<const v4i*>(p + 1024 + ((lane ^ (1 + 2 * gq)) * 16));
      fa[set][i] = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const uint8_t* p = st + A_BYTES + (wn * TN + j) * 2048 + lane * 16;
      const v4i lo = *reinterpret_cast<const v4i*>(p), hi = *reinterpret_cast<const v4i*>(p + 1024);
      fb[set][j] = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    }
  };
  v16f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  constexpr int NMF = TM * TN, NRD = 2 * (TM + TN), NWR = RA + RB, NLD = RA + RB;
  auto step_body = [&](int set, int t) __attribute__((always_inline)) {
    // t = current step; fragments of t are in fa/fb[set]
    uint8_t* rd = smem + ((t + 1) % NS) * STAGE;
    uint8_t* wr = smem + ((t + 2) % NS) * STAGE;
    frag_read(set ^ 1, rd);
    lds_write(set, wr);   // set == t % 2: the register set holding step t + 2
    gload(set, t + 4);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fb[set][j], fa[set][i], acc[i][j], 0, 0, 0, 0, 0, 0);
    // interleave: each MFMA followed by its share of LDS reads, writes and loads
#pragma unroll
    for (int t2 = 0; t2 < NMF; ++t2) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (t2 < NRD) __builtin_amdgcn_sched_group_barrier(0x100, (NRD + NMF - 1) / NMF, 0);
      if (t2 < NWR) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
      if (t2 < NLD) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
  };

  if (steps > 0) {
    // prologue: stages 0 and 1 filled, registers hold steps 2 and 3
    gload(0, 0);
    gload(1, 1);
    lds_write(0, smem);
    lds_write(1, smem + STAGE);
    __syncthreads();
    gload(0, 2);
    gload(1, 3);
    frag_read(0, smem);
    // steps = k / 64 is even (k % 128 == 0): two steps per iteration, one per register set
    for (int t = 0; t < steps; t += 2) {
      step_body(0, t);
      step_body(1, t + 1);
    }
  }

  store_tiles<TM, TN>(g, acc, m0 + wm * TM * 32, n0 + wn * TN * 32, lane, *g.w_tscale * *g.a_tscale);
}

template <int TM, int TN>
static hipError_t run_fp8(GemmArgs g, hipStream_t st) {
  g.tiles_m = (g.m + 64 * TM - 1) / (64 * TM);
  g.tiles_n = (g.n + 64 * TN - 1) / (64 * TN);
  hipLaunchKernelGGL((k_gemm_fp8<TM, TN>), dim3(g.tiles_m * g.tiles_n), dim3(256), 0, st, g);
  return hipGetLastError();
}

// ---------------------------------------------------------------- W8A8 / W4A4, few tokens: split K
// A workgroup owns a (32 MT) x (32 NP) output tile; its NW wavefronts split
// the reduction dimension (128-wide chunk kc goes to wave kc % NW), each
// wave accumulates the whole tile over its chunks, and the NW partial tiles
// are summed through LDS at the end. So a tile costs a few chunks of one
// wave, not K / 128 chunks in a row, and a short activation still keeps
// every CU busy. Both operands go straight from memory into registers in
// matrix-core operand order (no LDS staging, no barrier in the K loop):
//   weights     : the packed image, one 16-byte piece per lane and register
//                 half (plus, for NVFP4, one dword of four E4M3 block scales);
//   activations : lane (r, g) reads row r's bytes of the permuted reduction
//                 order directly: FP8 bytes [64 s + 32 g, +32) of step s,
//                 NVFP4 bytes [32 g, 32 g + 32) of the chunk's 64 (elements
//                 [64 g, 64 g + 64)) and its four block scales as one dword.
// Every wave keeps D chunks in flight in a ring of register sets: the loads
// of its chunk t + D are issued as soon as chunk t has been multiplied.
// NVFP4 expands both operands to fp16 in registers (exact, as in k_gemm);
// FP8 feeds the codes to the fp8 MFMA as they are.
// Partial tiles go to LDS as row-major fp32 (row pitch 32 NP + 4 words, so
// the 32 rows a store instruction touches spread over the banks), then
// every thread sums four consecutive outputs of a row over the waves in a
// fixed order (deterministic) and stores them: row-contiguous output writes.
// When NW tiles do not fit in the LDS, waves NW/2.. first add theirs into
// waves 0..NW/2-1 through it.
// Tiles are dealt so that each XCD owns a contiguous range of weight panel
// groups (its L2 then holds 1/8 of the weight and the whole activation).
// AQ (FP8 only): A is the bf16 activation itself, quantized in the kernel.
// Every workgroup first reduces the max of the whole activation (a small
// one: the caller bounds it) and derives the decode scale exactly as the
// dynamic quantizer does; each lane then codes the bf16 elements it loads
// for a step into the E4M3 bytes the FP8 path would have loaded, so codes,
// scale and accumulation order are those of quantize-then-GEMM. Workgroup 0
// writes the scale to a_tscale.
template <int MODE, int MT, int NP, int NW, int D, bool AQ = false>
__global__ void __launch_bounds__(64 * NW) k_gemm_splitk(GemmArgs g) {
  static_assert(MODE == MODE_FP8 || MODE == MODE_NVFP4, "W8A8 or W4A4");
  static_assert(!AQ || MODE == MODE_FP8, "in-kernel activation quantization: FP8");
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int BM = 32 * MT, BN = 32 * NP;
  constexpr int LDR = BN + 4;  // fp32 row pitch of a partial tile in LDS
  // partial tiles held in LDS at once: all NW, or NW / 2 when NW of them
  // would not fit (the upper half of the waves then hands its tiles to the
  // lower half first)
  constexpr int NRED = (NW * BM * LDR * 4 <= 160 * 1024) ? NW : NW / 2;
  static_assert(NRED * BM * LDR * 4 <= 160 * 1024, "partial tiles exceed the LDS");
  __shared__ __attribute__((aligned(16))) float red[NRED * BM * LDR];
  // the wave index is uniform across the wave: kept in a scalar register so
  // that the chunk loop's bounds and branches are scalar too (a per-lane
  // value there turns them into exec-masked regions, across which the
  // compiler waits for every outstanding load)
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 31, gq = lane >> 5;
  const int tiles = g.tiles_m * g.tiles_n;
  const int t = (tiles % 8 == 0) ? (int)(blockIdx.x & 7) * (tiles >> 3) + (int)(blockIdx.x >> 3) : (int)blockIdx.x;
  const int bn = t / g.tiles_m, bm = t - bn * g.tiles_m;
  const int m0 = bm * BM, n0 = bn * BN;
  const int kcn = g.k >> 7;
  const int npanels_w = (g.n + 31) >> 5;

  const __amdgpu_buffer_rsrc_t rs_w_ = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * kcn * (MODE == MODE_FP8 ? 4096 : 2048)), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_ws_ = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, MODE == MODE_NVFP4 ? (int)((int64_t)npanels_w * kcn * 256) : 0, 0x00020000);
  // NVFP4 activation rows: lda / 2 code bytes and lda / 16 scale bytes apart,
  // the descriptors ending at the last row's k / 2 and k / 16 bytes
  const int64_t ka = g.lda >> 1, ks = g.lda >> 4;
  const __amdgpu_buffer_rsrc_t rs_a_ = AQ
      ? __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(g.a), 0, (int)(((int64_t)(g.m - 1) * g.lda + g.k) * 2),
                                          0x00020000)
      : (MODE == MODE_FP8)
      ? rsrc_a_fp8(g)
      : __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(g.a), 0, (int)((int64_t)(g.m - 1) * ka + (g.k >> 1)),
                                          0x00020000);
  const __amdgpu_buffer_rsrc_t rs_as_ = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a_bscale), 0, MODE == MODE_NVFP4 ? (int)((int64_t)(g.m - 1) * ks + (g.k >> 4)) : 0,
      0x00020000);

  const __amdgpu_buffer_rsrc_t rs_none = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(g.w_codes), 0, 0, 0x00020000);

  // per-lane base offsets (rows and panels outside the operands: out of range, zeros)
  uint32_t oa[MT], oas[MT], ow[NP], ows[NP];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int row = m0 + 32 * i + r;
    const bool in = row < g.m;
    if (AQ) {  // bf16: two bytes per element
      oa[i] = in ? (uint32_t)(((int64_t)row * g.lda + 32 * gq) * 2) : OOB;
      oas[i] = OOB;
    } else if (MODE == MODE_FP8) {
      oa[i] = in ? (uint32_t)((int64_t)row * g.lda + 32 * gq) : OOB;
      oas[i] = OOB;
    } else {
      oa[i] = in ? (uint32_t)(row * ka + 32 * gq) : OOB;
      oas[i] = in ? (uint32_t)(row * ks + 4 * gq) : OOB;
    }
  }
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    const int pj = (n0 >> 5) + j;
    const bool in = pj < npanels_w;
    ow[j] = in ? (uint32_t)(pj * kcn * (MODE == MODE_FP8 ? 4096 : 2048) + lane * 16) : OOB;
    ows[j] = in ? (uint32_t)(pj * kcn * 256 + r * 8 + 4 * gq) : OOB;
  }

  // AQ: the activation's decode scale and its reciprocal (set below); with
  // a finite r every |x r| stays below 464 (x r <= max|x| r, within a few
  // ulps of 448), where the hardware conversion rounds as the clamped one
  // does, so the clamp is kept only for r = inf (a max below ~2^-119)
  float aq_s = 0.0f, aq_r = 0.0f;
  bool aq_clamp = false;

  // one 128-wide chunk of a lane's operands; FP8: piece 2 s + h = step s,
  // register half h; NVFP4: pieces 0, 1 = the 32 code bytes, sc = 4 scales
  struct Chunk {
    v4i a[MT][AQ ? 8 : (MODE == MODE_FP8 ? 4 : 2)];  // AQ: the bf16 elements of the FP8 pieces
    v4i w[NP][MODE == MODE_FP8 ? 4 : 2];
    uint32_t as[MODE == MODE_NVFP4 ? MT : 1];
    uint32_t ws[MODE == MODE_NVFP4 ? NP : 1];
  };
  auto load = [&](Chunk& C, int kc) __attribute__((always_inline)) {
    // the chunk's byte offset is uniform (the wave index is scalar), so it
    // travels in the loads' scalar offset; loads past the last chunk (never
    // multiplied) go through descriptors of zero bytes, which return zeros
    // without touching memory
    const bool in = kc < kcn;
    const int kq = in ? kc : 0;
    const __amdgpu_buffer_rsrc_t rs_a = in ? rs_a_ : rs_none, rs_as = in ? rs_as_ : rs_none;
    const __amdgpu_buffer_rsrc_t rs_w = in ? rs_w_ : rs_none, rs_ws = in ? rs_ws_ : rs_none;
    if (MODE == MODE_FP8) {
#pragma unroll
      for (int p = 0; p < 4; ++p) {  // step p / 2, register half p % 2
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          if (AQ) {  // the 16 elements of piece p as bf16: two 16-byte loads
            C.a[i][2 * p] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[i] + (p >> 1) * 128 + (p & 1) * 32, kq * 256, 0);
            C.a[i][2 * p + 1] =
                __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[i] + (p >> 1) * 128 + (p & 1) * 32 + 16, kq * 256, 0);
          } else {
            C.a[i][p] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[i] + (p >> 1) * 64 + (p & 1) * 16, kq * 128, 0);
          }
        }
#pragma unroll
        for (int j = 0; j < NP; ++j)
          C.w[j][p] = __builtin_amdgcn_raw_buffer_load_b128(rs_w, ow[j] + p * 1024, kq * 4096, 0);
      }
    } else {
      // in the order of use: block scales, then code halves 0 (steps 0..3)
      // and 1 (steps 4..7), so each step waits only for what it reads
#pragma unroll
      for (int i = 0; i < MT; ++i) C.as[i] = __builtin_amdgcn_raw_buffer_load_b32(rs_as, oas[i], kq * 8, 0);
#pragma unroll
      for (int j = 0; j < NP; ++j) C.ws[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_ws, ows[j], kq * 256, 0);
#pragma unroll
      for (int p = 0; p < 2; ++p) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
          C.a[i][p] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[i] + 16 * p, kq * 64, 0);
#pragma unroll
        for (int j = 0; j < NP; ++j)
          C.w[j][p] = __builtin_amdgcn_raw_buffer_load_b128(rs_w, ow[j] + 1024 * p, kq * 2048, 0);
      }
    }
    // keep each chunk's loads together and in this order: the waits before
    // a chunk's MFMAs then leave the later chunks' loads in flight
    __builtin_amdgcn_sched_barrier(0);
  };

  v16f acc[MT][NP];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NP; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  auto compute = [&](const Chunk& C) __attribute__((always_inline)) {
    if (MODE == MODE_FP8) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        v8i fa[MT], fb[NP];
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          if (AQ) {
            // E4M3(fl(x r)), four elements per dword: the dynamic
            // quantizer's element step
            int q[8];
            if (aq_clamp) {
#pragma unroll
              for (int d = 0; d < 8; ++d) {
                const v4i v = C.a[i][4 * s + (d >> 1)];
                const uint32_t w0 = (uint32_t)((d & 1) ? v.z : v.x), w1 = (uint32_t)((d & 1) ? v.w : v.y);
                const float y[4] = {__fmul_rn(bf16_lo(w0), aq_r), __fmul_rn(bf16_hi(w0), aq_r),
                                    __fmul_rn(bf16_lo(w1), aq_r), __fmul_rn(bf16_hi(w1), aq_r)};
                q[d] = (int)hw_e4m3x4(y);
              }
            } else {
#pragma unroll
              for (int d = 0; d < 8; ++d) {
                const v4i v = C.a[i][4 * s + (d >> 1)];
                const uint32_t w0 = (uint32_t)((d & 1) ? v.z : v.x), w1 = (uint32_t)((d & 1) ? v.w : v.y);
                typedef short v2s __attribute__((ext_vector_type(2)));
                v2s c = {0, 0};
                c = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(c, __fmul_rn(bf16_lo(w0), aq_r),
                                                             __fmul_rn(bf16_hi(w0), aq_r), 1.0f, false);
                c = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(c, __fmul_rn(bf16_lo(w1), aq_r),
                                                             __fmul_rn(bf16_hi(w1), aq_r), 1.0f, true);
                q[d] = __builtin_bit_cast(int, c);
              }
            }
            fa[i] = (v8i){q[0], q[1], q[2], q[3], q[4], q[5], q[6], q[7]};
          } else {
            const v4i lo = C.a[i][2 * s], hi = C.a[i][2 * s + 1];
            fa[i] = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
          }
        }
#pragma unroll
        for (int j = 0; j < NP; ++j) {
          const v4i lo = C.w[j][2 * s], hi = C.w[j][2 * s + 1];
          fb[j] = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        }
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int j = 0; j < NP; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fb[j], fa[i], acc[i][j], 0, 0, 0, 0, 0, 0);
      }
    } else {
      // the lane's four block scales as fp16 (the multiplies take the one
      // they need from its register half)
      uint2 sa[MT], sw[NP];
#pragma unroll
      for (int i = 0; i < MT; ++i) sa[i] = e4m3x4_to_f16x4(C.as[i]);
#pragma unroll
      for (int j = 0; j < NP; ++j) sw[j] = e4m3x4_to_f16x4(C.ws[j]);
      // step s: elements [64 g + 8 s, +8) of the chunk, block 4 g + s / 2;
      // the expansion of step s + 1 is issued between the MFMAs of step s
      v8h fa[2][MT], fb[2][NP];
      auto expand = [&](int s, int set) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          const v4i c = C.a[i][s >> 2];
          const uint32_t w = (uint32_t)((s & 3) == 0 ? c.x : (s & 3) == 1 ? c.y : (s & 3) == 2 ? c.z : c.w);
          fa[set][i] = dequant8_f16(w, scale_f16(sa[i], s >> 1));
        }
#pragma unroll
        for (int j = 0; j < NP; ++j) {
          const v4i c = C.w[j][s >> 2];
          const uint32_t w = (uint32_t)((s & 3) == 0 ? c.x : (s & 3) == 1 ? c.y : (s & 3) == 2 ? c.z : c.w);
          fb[set][j] = dequant8_f16(w, scale_f16(sw[j], s >> 1));
        }
      };
      expand(0, 0);
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        if (s < 7) expand(s + 1, (s + 1) & 1);
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int j = 0; j < NP; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fb[s & 1][j], fa[s & 1][i], acc[i][j], 0, 0, 0);
        if (s < 7) {
          // each MFMA followed by its share of the next step's 8 (MT + NP)
          // conversions and multiplies
#pragma unroll
          for (int t = 0; t < MT * NP; ++t) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, (8 * (MT + NP) + MT * NP - 1) / (MT * NP), 0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  // this wave's chunks: kc = wave + NW t, t = 0 .. nt - 1
  const int nt = (kcn - wave + NW - 1) / NW;
  Chunk C[D];
#pragma unroll
  for (int d = 0; d < D; ++d) load(C[d], wave + NW * d);
  if constexpr (AQ) {
    // max |x| over the whole activation (bf16 magnitude bits, as the
    // quantizer reduces them), eight 16-byte units per thread in flight
    // (sixteen were no faster at 128 x 256 and slower at 1 x 1024 .. 16 x 1024)
    __shared__ uint32_t aq_part[NW];
    const int upr = g.k >> 3, units = g.m * upr;
    uint32_t mx = 0;
    for (int u0 = (int)threadIdx.x; u0 < units; u0 += 8 * 64 * NW) {
      uint4 v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int u = u0 + e * 64 * NW;
        const int row = u / upr;
        v[e] = (u < units) ? *reinterpret_cast<const uint4*>(g.a + ((int64_t)row * g.lda + 8 * (u - row * upr)) * 2)
                           : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t w[4] = {v[e].x, v[e].y, v[e].z, v[e].w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t t2 = w[j] & 0x7FFF7FFFu;
          mx = max(mx, max(t2 & 0xFFFFu, t2 >> 16));
        }
      }
    }
    for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
    if (lane == 0) aq_part[wave] = mx;
    __syncthreads();
    uint32_t a = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) a = max(a, aq_part[w]);
    a <<= 16;
    aq_s = (a >= 0x7F800000u) ? __builtin_nanf("") : __fdiv_rn(u2f(a), 448.0f);
    aq_r = (aq_s > 0.0f) ? __fdiv_rn(1.0f, aq_s) : 0.0f;
    aq_clamp = !(aq_r <= 3.40282347e38f);
    if (blockIdx.x == 0 && threadIdx.x == 0) *const_cast<float*>(g.a_tscale) = aq_s;
  }
  for (int t0 = 0; t0 < nt; t0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      if (t0 + d < nt) compute(C[d]);
      load(C[d], wave + NW * (t0 + d + D));
    }
  }

  // partial tiles -> LDS (row-major fp32), then the sum over the waves
  auto put = [&](float* part) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < NP; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<float4*>(part + (32 * i + r) * LDR + 32 * j + 8 * q + 4 * gq) =
              make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
  };
  if (NRED < NW) {
    // waves NRED.. pass their tiles to waves 0..NRED-1 (wave w + NRED -> w)
    if (wave >= NRED) put(red + (wave - NRED) * (BM * LDR));
    __syncthreads();
    if (wave < NRED) {
      const float* part = red + wave * (BM * LDR);
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NP; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float4 v = *reinterpret_cast<const float4*>(part + (32 * i + r) * LDR + 32 * j + 8 * q + 4 * gq);
            acc[i][j][4 * q] += v.x; acc[i][j][4 * q + 1] += v.y; acc[i][j][4 * q + 2] += v.z; acc[i][j][4 * q + 3] += v.w;
          }
    }
    __syncthreads();
  }
  if (wave < NRED) put(red + wave * (BM * LDR));
  __syncthreads();
  const float c = *g.w_tscale * (AQ ? aq_s : *g.a_tscale);
  const bool vec = out_vec(g);
  const float ry = out_rscale(g);
  const bool nv = g.out_mode == OUT_NVFP4;
  const float st = nv ? *g.y_scale : 0.0f, d = nv_out_d(g);
  // the four lanes of a 16-block are consecutive (BN / 4 is a multiple of 8)
  for (int u = threadIdx.x; u < BM * (BN / 4); u += 64 * NW) {
    const int row = u / (BN / 4), c4 = u - row * (BN / 4);
    const int m = m0 + row, n = n0 + 4 * c4;
    if (m >= g.m || n >= g.n) continue;
    float4 sum = *reinterpret_cast<const float4*>(red + row * LDR + 4 * c4);
#pragma unroll
    for (int w = 1; w < NRED; ++w) {
      const float4 v = *reinterpret_cast<const float4*>(red + w * (BM * LDR) + row * LDR + 4 * c4);
      sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
    }
    if (nv) {
      const float v[4] = {sum.x * c, sum.y * c, sum.z * c, sum.w * c};
      store_nv_quad(g, m, n, v, st, d);
    } else {
      store4(g, m, n, sum.x * c, sum.y * c, sum.z * c, sum.w * c, vec, ry);
    }
  }
}

template <int MODE, int MT, int NP, int NW, int D, bool AQ = false>
static hipError_t run_splitk(GemmArgs g, hipStream_t st) {
  g.tiles_m = (g.m + 32 * MT - 1) / (32 * MT);
  g.tiles_n = (g.n + 32 * NP - 1) / (32 * NP);
  hipLaunchKernelGGL((k_gemm_splitk<MODE, MT, NP, NW, D, AQ>), dim3(g.tiles_m * g.tiles_n), dim3(64 * NW), 0, st, g);
  return hipGetLastError();
}

// ---------------------------------------------------------------- FP8, 256 x 256 tiles
// Epilogue fast path: bf16 output, whole tile inside the output, 16-byte
// aligned rows. Stored straight from the MFMA layout, every store
// instruction would scatter 8-byte pieces over 32 rows, which the memory
// pipeline takes one cache line at a time; here each 32-row block of the
// wave's tile is converted into the wave's private LDS area in the MFMA
// layout (row pitch padded by 16 bytes so the 32 rows spread over all
// banks) and read back 16 bytes per lane in row order, so that every store
// instruction writes four whole 256-byte row segments. Each wave reads back
// only what it wrote, so no barrier is needed; all addresses are one base
// register plus immediate offsets. `stage` holds 32 * (64 TN + 16) bytes.
template <int TM, int TN>
__device__ __attribute__((always_inline)) inline void store_tiles_fast(const GemmArgs& g, const v16f (&acc)[TM][TN],
                                                                       uint8_t* stage, int mw, int nw, int lane,
                                                                       float c) {
  constexpr int RB = 64 * TN, PITCH = RB + 16, PPR = RB / 16, ROWS_PER_IT = 64 / PPR;
  static_assert(64 % PPR == 0, "a wave reads whole rows per instruction");
  uint8_t* wr = stage + (lane & 31) * PITCH + 8 * (lane >> 5);
  const uint8_t* rd = stage + (lane / PPR) * PITCH + 16 * (lane % PPR);
  uint8_t* out = reinterpret_cast<uint8_t*>(g.y) + ((int64_t)(mw + lane / PPR) * g.ldy + nw + 8 * (lane % PPR)) * 2;
  const int64_t it_stride = (int64_t)ROWS_PER_IT * g.ldy * 2;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd)
        *reinterpret_cast<uint2*>(wr + (32 * j + 8 * qd) * 2) =
            make_uint2(pk_bf16(acc[i][j][4 * qd] * c, acc[i][j][4 * qd + 1] * c),
                       pk_bf16(acc[i][j][4 * qd + 2] * c, acc[i][j][4 * qd + 3] * c));
    uint8_t* o = out + (int64_t)i * 32 * 2 * g.ldy;
#pragma unroll
    for (int it = 0; it < 32 / ROWS_PER_IT; ++it)
      *reinterpret_cast<uint4*>(o + it * it_stride) = *reinterpret_cast<const uint4*>(rd + it * ROWS_PER_IT * PITCH);
  }
}

// Activation staging shared by the 256 x 256 FP8 kernels: 256 rows x one
// 128-byte chunk, read row-contiguously (8 lanes per row) and stored in LDS
// as 8 panels of 4 KiB. Piece c (bytes 16c .. 16c+15 of the row's chunk)
// belongs to step s = c / 4, lane half g = (c / 2) % 2 and register half
// h = c % 2 of the MFMA operand, so it lands in 1 KiB block 2s + h of its
// panel at slot (r + 32 g) ^ (c + 8 h): the eight lanes of a row, and the
// sixteen lanes of two rows, fall into distinct bank groups (32 or 64
// banks), and the operand read of lane l (slot l ^ (4s + 2g + 9h)) is a
// permutation of one contiguous 1 KiB block -- conflict free.
//
// MX8 (MXFP8): the block-scaled fp8 instruction reads a row's scale block h
// from register half h of both lane halves, so there piece c belongs to
// step s = c / 4, register half h = (c / 2) % 2 and lane half g = c % 2; the
// slot XOR is the same function of (s, g, h), so read_a_frag serves both.
struct AStage256 {
  static constexpr int RA = 8;  // pieces per thread per chunk
  uint32_t oa[RA], la[RA];
  template <bool MX8 = false>
  __device__ __attribute__((always_inline)) inline void init(const GemmArgs& g, int m0, int tid) {
#pragma unroll
    for (int it = 0; it < RA; ++it) {
      const int q = it * 256 + tid;
      const int p = q >> 8, rr = (q >> 3) & 31, c = q & 7;
      const int s = c >> 2, gg = MX8 ? (c & 1) : ((c >> 1) & 1), h = MX8 ? ((c >> 1) & 1) : (c & 1);
      const uint32_t row = (uint32_t)(m0 + 32 * p + rr);
      oa[it] = (row < (uint32_t)g.m) ? row * (uint32_t)g.lda + 16u * c : 0x80000000u;
      la[it] = (uint32_t)(p * 4096 + (2 * s + h) * 1024 + (((rr + 32 * gg) ^ (4 * s + 2 * gg + 9 * h)) * 16));
    }
  }
};

// Operand fragment of activation panel `panel`, step s (0/1) of a staged chunk.
__device__ __attribute__((always_inline)) inline v8i read_a_frag(const uint8_t* st, int panel, int s, int lane) {
  const int x = 4 * s + 2 * (lane >> 5);
  const uint8_t* p = st + panel * 4096 + s * 2048;
  const v4i lo = *reinterpret_cast<const v4i*>(p + ((lane ^ x) * 16));
  const v4i hi = *reinterpret_cast<const v4i*>(p + 1024 + ((lane ^ (x + 9)) * 16));
  return (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
}

// W8A8, weights straight from memory. Same tile and wave layout, but each
// wave loads its weight fragments from the packed buffer directly into
// registers -- the packed layout is already the operand image, one
// contiguous 1 KiB per wave load -- one chunk ahead, in two register sets.
// Only the activations pass through LDS, which halves LDS traffic (32 KiB of
// writes and 64 KiB of reads per chunk instead of 64 and 128) at the price
// of each weight chunk being fetched by the two waves that share it (the
// second fetch normally hits the CU's L1). Activation fragments are read
// just in time, one 32-row panel ahead of the MFMAs that use it.
//
// The grid is persistent (at most one workgroup per CU, each walking the
// tiles blockIdx.x, + gridDim.x, ...), so a workgroup's next tile starts
// loading while the stores of its previous tile drain. Prefetches that would
// run past the last chunk of a tile are turned into out-of-range loads,
// which return zeros without touching memory.
__global__ void __launch_bounds__(256) k_gemm_fp8_direct(GemmArgs g) {
  constexpr int A_STAGE = 8 * 4096;
  constexpr int RA = AStage256::RA;
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int OUT_STAGE = 32 * (64 * 4 + 16);  // per wave: 32 rows of 128 bf16 + pad
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * A_STAGE];
  __shared__ __attribute__((aligned(16))) uint8_t sout[4 * OUT_STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int kcn = g.k >> 7;
  const int npanels_w = (g.n + 31) >> 5;
  const int total = g.tiles_m * g.tiles_n;
  const float scale = *g.w_tscale * *g.a_tscale;
  const bool fast_out = g.out_mode == OUT_BF16 && ((reinterpret_cast<uintptr_t>(g.y) & 15) == 0) && ((g.ldy & 7) == 0);
  const __amdgpu_buffer_rsrc_t rs_a = rsrc_a_fp8(g);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * kcn * 4096), 0x00020000);

  AStage256 A;
  uint32_t ob[4];
  v4i ga[RA];
  v8i fb[2][2][4];  // [chunk parity][step][weight panel]
  v8i fa[2];
  v16f acc[4][4];

  // The chunk's byte offset is uniform, so it travels in the loads' scalar
  // offset and costs no per-lane arithmetic. Prefetches past the last chunk
  // re-read that chunk (in bounds; their data is never multiplied). Rows and
  // panels outside the operands keep an out-of-range per-lane base.
  auto kcl = [&](int kc) __attribute__((always_inline)) { return kc < kcn ? kc : kcn - 1; };
  auto load_a = [&](int kc) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < RA; ++it)
      ga[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, A.oa[it], kcl(kc) * 128, 0);
  };
  auto write_a = [&](uint8_t* st) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < RA; ++it) *reinterpret_cast<v4i*>(st + A.la[it]) = ga[it];
  };
  // weight fragments of chunk kc into set P: (step, panel) in load order
  auto load_b = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const int so = kcl(kc) * 4096;
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const v4i lo = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[j] + s * 2048, so, 0);
        const v4i hi = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[j] + s * 2048 + 1024, so, 0);
        fb[P][s][j] = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      }
  };
  // MFMA group f = (step f / 4, activation panel f % 4) on fragment fa[f % 2]
  auto mgroup = [&](auto Pc, int f) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc[f & 3][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fb[P][f >> 2][j], fa[f & 1], acc[f & 3][j], 0, 0, 0, 0, 0, 0);
  };
  auto chunk = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const uint8_t* cur = smem + P * A_STAGE;
    uint8_t* nxt = smem + (P ^ 1) * A_STAGE;
    // step 0: weight loads of chunk kc + 1, activation fragments 1..4
    load_b(std::integral_constant<int, P ^ 1>(), kc + 1);
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      fa[(f + 1) & 1] = read_a_frag(cur, wm * 4 + ((f + 1) & 3), (f + 1) >> 2, lane);
      mgroup(Pc, f);
    }
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS read: next fragment
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (weights)
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    // step 1, groups 4..6: stage activations of chunk kc + 1, load kc + 2.
    // The LDS writes sit between the fragment reads in program order (the
    // compiler cannot tell the two stages apart, so it keeps LDS accesses in
    // that order); each activation load follows the write of its register.
    const int a_so = kcl(kc + 2) * 128;
#pragma unroll
    for (int f = 4; f < 7; ++f) {
      fa[(f + 1) & 1] = read_a_frag(cur, wm * 4 + ((f + 1) & 3), (f + 1) >> 2, lane);
#pragma unroll
      for (int it = 3 * (f - 4); it < 3 * (f - 3) && it < RA; ++it)
        *reinterpret_cast<v4i*>(nxt + A.la[it]) = ga[it];
      mgroup(Pc, f);
#pragma unroll
      for (int it = 3 * (f - 4); it < 3 * (f - 3) && it < RA; ++it)
        ga[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, A.oa[it], a_so, 0);
    }
#pragma unroll
    for (int f = 4; f < 7; ++f) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS read: next fragment
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        if (t < 3 && 3 * (f - 4) + t < RA) {
          __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // DS write
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (activations)
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    // group 7 covers the read of the next chunk's first fragment
    fa[0] = read_a_frag(nxt, wm * 4, 0, lane);
    mgroup(Pc, 7);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    int bm, bn;
    tile_coords(tile, g.tiles_m, g.tiles_n, bm, bn);
    const int m0 = bm * 256, n0 = bn * 256;
    A.init(g, m0, tid);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t panel = (uint32_t)((n0 >> 5) + wn * 4 + j);
      ob[j] = (panel < (uint32_t)npanels_w) ? panel * (uint32_t)(kcn * 4096) + 16u * lane : OOB;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // An odd chunk count takes its first chunk unpipelined, so that the
    // pipelined loop always runs whole pairs of chunks (register set 0, then
    // 1) and nothing follows it.
    int kc = 0;
    if (kcn & 1) {
      load_a(0);
      write_a(smem);
      load_b(std::integral_constant<int, 0>(), 0);
      __syncthreads();
#pragma unroll
      for (int f = 0; f < 8; ++f) {
        fa[f & 1] = read_a_frag(smem, wm * 4 + (f & 3), f >> 2, lane);
        mgroup(std::integral_constant<int, 0>(), f);
      }
      __syncthreads();
      kc = 1;
    }
    if (kc < kcn) {
      load_a(kc);
      write_a(smem);
      __syncthreads();
      // weights of chunk kc before activations of kc + 1: the order the loop
      // issues them in, so that the loop head's waits count the same loads
      load_b(std::integral_constant<int, 0>(), kc);
      load_a(kc + 1);
      fa[0] = read_a_frag(smem, wm * 4, 0, lane);
      for (; kc < kcn; kc += 2) {
        chunk(std::integral_constant<int, 0>(), kc);
        chunk(std::integral_constant<int, 1>(), kc + 1);
      }
    }
    // Every operand write of this tile happened before its last barrier; the
    // next tile's first write to stage 0 can only race with the discarded
    // fragment read after that barrier.
    if (fast_out && m0 + 256 <= g.m && n0 + 256 <= g.n)
      store_tiles_fast<4, 4>(g, acc, sout + wave * OUT_STAGE, m0 + wm * 128, n0 + wn * 128, lane, scale);
    else
      store_tiles<4, 4>(g, acc, m0 + wm * 128, n0 + wn * 128, lane, scale);
  }
}

// ---------------------------------------------------------------- FP8, 288 x 192 tiles
// At the transformer shapes (M = 4608, N = 3072 or 9216) 256 x 256 tiles
// number 216 or 648 on 256 CUs, so one round of tiles in every three (or the
// only round) runs 16-47% empty, and the kernel's time follows the number of
// rounds (measured: 1.0, 2.0 and 3.0 rounds' time at 0.84, 1.97 and 2.53
// rounds of tiles). 288 x 192 tiles give exactly 256 or 768 tiles there.
// Four waves in 2 x 2, each 144 x 96 = 9 x 6 blocks of
// v_mfma_f32_16x16x128_f8f6f4, which runs at the 32x32x64 instruction's rate
// (4.69 PFLOP/s with 54 independent accumulators, one wave per SIMD), so the
// tile needs no 32-row granularity in M.
//   weights     : fragment (16 rows x 128 K) of lane l = row l % 16, bytes
//                 32 (l / 16) .. + 31 of the row's chunk; in the packed FP8
//                 image those are pieces h = 0, 1 of step t = l / 32, lane
//                 half g = (l / 16) % 2, so each 16-byte wave load reads four
//                 contiguous 256-byte runs. Loaded straight into registers one
//                 chunk ahead, two register sets.
//   activations : staged in LDS per chunk as 18 blocks of 16 rows x 128 B;
//                 piece c (16 B) of row i of a block sits in slot
//                 8 i + (c ^ f(i)), f(i) = (i & 7) ^ (i >> 3): the eight
//                 lanes that stage one row, and the fragment reads (lane l:
//                 row l % 16, pieces 2 (l / 16) and 2 (l / 16) + 1), hit
//                 distinct bank groups for 32 and for 64 banks (checked on the
//                 CPU).
// Output: lane l of block (i, j) holds Y[m0 + 16 i + l % 16][n0 + 16 j +
// 4 (l / 16) + e], four consecutive outputs of a row. bf16, fp32 and FP8
// outputs; the NVFP4 output keeps the 256 x 256 kernel.
struct AStage288 {
  static constexpr int RA = 9;  // 16-byte pieces per thread per chunk
  uint32_t oa[RA], la[RA];
  __device__ __attribute__((always_inline)) inline void init(const GemmArgs& g, int m0, int tid) {
#pragma unroll
    for (int it = 0; it < RA; ++it) {
      const int q = it * 256 + tid;
      const int row = q >> 3, c = q & 7, i = row & 15;
      const uint32_t grow = (uint32_t)(m0 + row);
      oa[it] = (grow < (uint32_t)g.m) ? grow * (uint32_t)g.lda + 16u * c : 0x80000000u;
      la[it] = (uint32_t)((row >> 4) * 2048 + i * 128 + ((c ^ ((i & 7) ^ (i >> 3))) * 16));
    }
  }
};

__device__ __attribute__((always_inline)) inline v8i read_a16(const uint8_t* st, int blk, int lane) {
  const int i = lane & 15, q = lane >> 4, f = (i & 7) ^ (i >> 3);
  const uint8_t* p = st + blk * 2048 + i * 128;
  const v4i lo = *reinterpret_cast<const v4i*>(p + (((2 * q) ^ f) * 16));
  const v4i hi = *reinterpret_cast<const v4i*>(p + (((2 * q + 1) ^ f) * 16));
  return (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
}

__global__ void __launch_bounds__(256) k_gemm_fp8_t288(GemmArgs g) {
  constexpr int A_STAGE = 18 * 2048;
  constexpr int RA = AStage288::RA;
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int OPITCH = 96 * 2 + 16;           // output staging: 16 rows of 96 bf16 + pad
  constexpr int OUT_STAGE = 16 * OPITCH;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * A_STAGE];
  __shared__ __attribute__((aligned(16))) uint8_t sout[4 * OUT_STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int kcn = g.k >> 7;
  const int npanels_w = (g.n + 31) >> 5;
  const int total = g.tiles_m * g.tiles_n;
  const float scale = *g.w_tscale * *g.a_tscale;
  const bool fast_out = g.out_mode == OUT_BF16 && ((reinterpret_cast<uintptr_t>(g.y) & 15) == 0) && ((g.ldy & 7) == 0);
  const __amdgpu_buffer_rsrc_t rs_a = rsrc_a_fp8(g);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * kcn * 4096), 0x00020000);
  // lane part of a weight fragment's offset inside a panel's chunk
  const uint32_t lane_b = (uint32_t)((lane >> 5) * 2048 + ((lane & 15) + 32 * ((lane >> 4) & 1)) * 16);

  AStage288 A;
  uint32_t ob[3];
  v4i ga[RA];
  v8i fb[2][6];  // [chunk parity][16-row weight fragment]
  v8i fa[2];
  v4f acc[9][6];

  auto kcl = [&](int kc) __attribute__((always_inline)) { return kc < kcn ? kc : kcn - 1; };
  auto load_a = [&](int kc) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < RA; ++it)
      ga[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, A.oa[it], kcl(kc) * 128, 0);
  };
  auto write_a = [&](uint8_t* st) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < RA; ++it) *reinterpret_cast<v4i*>(st + A.la[it]) = ga[it];
  };
  auto load_b = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const int so = kcl(kc) * 4096;
#pragma unroll
    for (int jj = 0; jj < 6; ++jj) {
      const uint32_t o = ob[jj >> 1] + (jj & 1) * 256;
      const v4i lo = __builtin_amdgcn_raw_buffer_load_b128(rs_b, o, so, 0);
      const v4i hi = __builtin_amdgcn_raw_buffer_load_b128(rs_b, o + 1024, so, 0);
      fb[P][jj] = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    }
  };
  // MFMA group f: activation block f of the wave against its six weight fragments
  auto mgroup = [&](auto Pc, int f, int slot) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
#pragma unroll
    for (int jj = 0; jj < 6; ++jj)
      acc[f][jj] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(fb[P][jj], fa[slot], acc[f][jj], 0, 0, 0, 0, 0, 0);
  };
  auto chunk = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const uint8_t* cur = smem + P * A_STAGE;
    uint8_t* nxt = smem + (P ^ 1) * A_STAGE;
    // groups 0, 1: weight loads of chunk kc + 1 (12 per lane)
    load_b(std::integral_constant<int, P ^ 1>(), kc + 1);
#pragma unroll
    for (int f = 0; f < 3; ++f) {
      fa[(f + 1 + P) & 1] = read_a16(cur, wm * 9 + f + 1, lane);
      mgroup(Pc, f, (f + P) & 1);
    }
#pragma unroll
    for (int f = 0; f < 3; ++f) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS read: next fragment
#pragma unroll
      for (int t = 0; t < 6; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        if (f < 2) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (weights)
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    // groups 3..7: stage the activations of chunk kc + 1 (two pieces per
    // group, the last group one), then load chunk kc + 2 into the same registers
    const int a_so = kcl(kc + 2) * 128;
#pragma unroll
    for (int f = 3; f < 8; ++f) {
      fa[(f + 1 + P) & 1] = read_a16(cur, wm * 9 + f + 1, lane);
#pragma unroll
      for (int it = 2 * (f - 3); it < 2 * (f - 2) && it < RA; ++it)
        *reinterpret_cast<v4i*>(nxt + A.la[it]) = ga[it];
      mgroup(Pc, f, (f + P) & 1);
#pragma unroll
      for (int it = 2 * (f - 3); it < 2 * (f - 2) && it < RA; ++it)
        ga[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, A.oa[it], a_so, 0);
    }
#pragma unroll
    for (int f = 3; f < 8; ++f) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS read: next fragment
#pragma unroll
      for (int t = 0; t < 6; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        if (t < 2 && 2 * (f - 3) + t < RA) {
          __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // DS write
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (activations)
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    // group 8 covers the read of the next chunk's first fragment
    fa[(9 + P) & 1] = read_a16(nxt, wm * 9, lane);
    mgroup(Pc, 8, (8 + P) & 1);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    int bm, bn;
    tile_coords(tile, g.tiles_m, g.tiles_n, bm, bn);
    const int m0 = bm * 288, n0 = bn * 192;
    A.init(g, m0, tid);
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const uint32_t panel = (uint32_t)((n0 >> 5) + wn * 3 + j);
      ob[j] = (panel < (uint32_t)npanels_w) ? panel * (uint32_t)(kcn * 4096) + lane_b : OOB;
    }
#pragma unroll
    for (int i = 0; i < 9; ++i)
#pragma unroll
      for (int j = 0; j < 6; ++j) acc[i][j] = (v4f){0.0f, 0.0f, 0.0f, 0.0f};

    // An odd chunk count takes its first chunk unpipelined, so that the
    // pipelined loop runs whole pairs of chunks (register set 0, then 1).
    int kc = 0;
    if (kcn & 1) {
      load_a(0);
      write_a(smem);
      load_b(std::integral_constant<int, 0>(), 0);
      __syncthreads();
#pragma unroll
      for (int f = 0; f < 9; ++f) {
        fa[f & 1] = read_a16(smem, wm * 9 + f, lane);
        mgroup(std::integral_constant<int, 0>(), f, f & 1);
      }
      __syncthreads();
      kc = 1;
    }
    if (kc < kcn) {
      load_a(kc);
      write_a(smem);
      __syncthreads();
      // weights of chunk kc before activations of kc + 1: the order the loop
      // issues them in, so that the loop head's waits count the same loads
      load_b(std::integral_constant<int, 0>(), kc);
      load_a(kc + 1);
      fa[0] = read_a16(smem, wm * 9, lane);
      for (; kc < kcn; kc += 2) {
        chunk(std::integral_constant<int, 0>(), kc);
        chunk(std::integral_constant<int, 1>(), kc + 1);
      }
    }
    const int mw = m0 + wm * 144, nw = n0 + wn * 96;
    if (fast_out && m0 + 288 <= g.m && n0 + 192 <= g.n) {
      // each 16-row block of the wave through its private LDS area, read back
      // in row order so that every store writes whole 192-byte row segments
      uint8_t* st = sout + wave * OUT_STAGE;
      uint8_t* wr = st + (lane & 15) * OPITCH + 8 * (lane >> 4);
#pragma unroll
      for (int i = 0; i < 9; ++i) {
#pragma unroll
        for (int jj = 0; jj < 6; ++jj)
          *reinterpret_cast<uint2*>(wr + 32 * jj) =
              make_uint2(pk_bf16(acc[i][jj][0] * scale, acc[i][jj][1] * scale),
                         pk_bf16(acc[i][jj][2] * scale, acc[i][jj][3] * scale));
#pragma unroll
        for (int it = 0; it < 3; ++it) {
          const int idx = it * 64 + lane, row = idx / 12, pc = idx - 12 * (idx / 12);
          const uint4 v = *reinterpret_cast<const uint4*>(st + row * OPITCH + pc * 16);
          *reinterpret_cast<uint4*>(reinterpret_cast<uint8_t*>(g.y) +
                                    ((int64_t)(mw + 16 * i + row) * g.ldy + nw + 8 * pc) * 2) = v;
        }
      }
    } else {
      const bool vec = out_vec(g);
      const float ry = out_rscale(g);
#pragma unroll
      for (int i = 0; i < 9; ++i) {
        const int m = mw + 16 * i + (lane & 15);
        if (m >= g.m) continue;
#pragma unroll
        for (int jj = 0; jj < 6; ++jj) {
          const int n = nw + 16 * jj + 4 * (lane >> 4);
          if (n >= g.n) continue;
          store4(g, m, n, acc[i][jj][0] * scale, acc[i][jj][1] * scale, acc[i][jj][2] * scale,
                 acc[i][jj][3] * scale, vec, ry);
        }
      }
    }
  }
}

// ---------------------------------------------------------------- MXFP8 (W8A8, MX block scaling)
// OCP MXFP8 x MXFP8: the W8A8 kernel above with the E8M0 block scales handed
// to the block-scaled matrix instruction. With fp8 operands that instruction
// takes a row's 32-element scale block h from register half h of both lane
// halves (elements 32 h + 16 g of the step in lane half g), and the scale of
// block h from lane half h, so weights and activations are laid out that way
// (MXFP8 packing, AStage256<MX8>):
//   weights     : the FP8 packed images, plus one dword per panel, 256-wide
//                 group and lane holding the lane's scales of its four steps
//                 (the MXFP4 scale layout); chunk kc uses bytes 2 (kc % 2) + s;
//   activations : codes staged as in the W8A8 kernel; the row's 4 scales of a
//                 128-wide chunk staged beside them, re-ordered to
//                 [half 0: steps 0, 1][half 1: steps 0, 1], one 16-bit read per
//                 lane and panel.
// K must be a multiple of 256 (whole chunk pairs, no odd first chunk); no
// tensor scales.
__global__ void __launch_bounds__(256) k_gemm_mxfp8_direct(GemmArgs g) {
  constexpr int A_CODES = 8 * 4096;
  constexpr int A_STAGE = A_CODES + 256 * 4;
  constexpr int RA = AStage256::RA;
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int OUT_STAGE = 32 * (64 * 4 + 16);
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * A_STAGE];
  __shared__ __attribute__((aligned(16))) uint8_t sout[4 * OUT_STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r = lane & 31, gq = lane >> 5;
  const int kcn = g.k >> 7;
  const int npanels_w = (g.n + 31) >> 5;
  const int total = g.tiles_m * g.tiles_n;
  const bool fast_out = g.out_mode == OUT_BF16 && ((reinterpret_cast<uintptr_t>(g.y) & 15) == 0) && ((g.ldy & 7) == 0);
  const uint32_t ks = (uint32_t)(g.k >> 5);  // A scale bytes per row
  const __amdgpu_buffer_rsrc_t rs_a = rsrc_a_fp8(g);
  const __amdgpu_buffer_rsrc_t rs_as = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a_bscale), 0, (int)((int64_t)g.m * ks), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * kcn * 4096), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_bs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, (int)((int64_t)npanels_w * (kcn >> 1) * 256), 0x00020000);

  AStage256 A;
  uint32_t ob[4], osb[4], osa;
  v4i ga[RA];
  uint32_t gs;         // staged activation scales of the thread's row (4 blocks of a chunk)
  v8i fb[2][2][4];     // [chunk parity][step][weight panel]
  uint32_t bsc[4];     // weight scales of the current chunk pair [panel]: byte 2 (kc % 2) + s
  uint32_t bsn[4];     // ... of the next pair
  uint32_t asc[4];     // activation scales of the current chunk [panel]: byte s (low half)
  v8i fa[2];
  v16f acc[4][4];

  // Chunk offsets are uniform: they travel in the loads' scalar offset,
  // clamped to the last chunk (prefetches past the end re-read it in bounds;
  // their data is never multiplied). Rows and panels outside the operands
  // keep an out-of-range per-lane base.
  auto kcl = [&](int kc) __attribute__((always_inline)) { return kc < kcn ? kc : kcn - 1; };
  auto load_a = [&](int kc) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < RA; ++it)
      ga[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, A.oa[it], kcl(kc) * 128, 0);
    gs = __builtin_amdgcn_raw_buffer_load_b32(rs_as, osa, kcl(kc) * 4, 0);
  };
  // blocks 0..3 of the chunk -> [half 0: 0 2][half 1: 1 3]
  auto write_a_scales = [&](uint8_t* st) __attribute__((always_inline)) {
    *reinterpret_cast<uint32_t*>(st + A_CODES + tid * 4) = __builtin_amdgcn_perm(0u, gs, 0x03010200u);
  };
  auto write_a = [&](uint8_t* st) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < RA; ++it) *reinterpret_cast<v4i*>(st + A.la[it]) = ga[it];
    write_a_scales(st);
  };
  auto read_asc = [&](const uint8_t* st) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      asc[i] = *reinterpret_cast<const uint16_t*>(st + A_CODES + ((wm * 4 + i) * 32 + r) * 4 + 2 * gq);
  };
  auto load_b = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const int so = kcl(kc) * 4096;
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const v4i lo = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[j] + s * 2048, so, 0);
        const v4i hi2 = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[j] + s * 2048 + 1024, so, 0);
        fb[P][s][j] = (v8i){lo.x, lo.y, lo.z, lo.w, hi2.x, hi2.y, hi2.z, hi2.w};
      }
  };
  // the weight scale dwords of the chunk pair starting at chunk kc (even)
  auto load_bs = [&](int kc) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 4; ++j) bsn[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_bs, osb[j], (kcl(kc) >> 1) * 256, 0);
  };
  // MFMA group f = (step f / 4, activation panel f % 4); chunk parity P
  auto mgroup = [&](auto Pc, auto Fc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value, f = decltype(Fc)::value;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      acc[f & 3][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fb[P][f >> 2][j], fa[f & 1], acc[f & 3][j], 0, 0,
                                                                       2 * P + (f >> 2), (int)bsc[j], f >> 2,
                                                                       (int)asc[f & 3]);
  };
  auto chunk = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const uint8_t* cur = smem + P * A_STAGE;
    uint8_t* nxt = smem + (P ^ 1) * A_STAGE;
    // step 0: weight loads of chunk kc + 1 (and, in the first chunk of a
    // pair, the scale dwords of the next pair), activation fragments 1..4
    load_b(std::integral_constant<int, P ^ 1>(), kc + 1);
    if (P == 0) load_bs(kc + 2);
    [&]<int... F>(std::integer_sequence<int, F...>) {
      ((fa[(F + 1) & 1] = read_a_frag(cur, wm * 4 + ((F + 1) & 3), (F + 1) >> 2, lane),
        mgroup(Pc, std::integral_constant<int, F>())), ...);
    }(std::make_integer_sequence<int, 4>());
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS read: next fragment
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (weights)
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    // step 1, groups 4..6: stage activations of chunk kc + 1, load kc + 2
    const int a_so = kcl(kc + 2);
    [&]<int... F>(std::integer_sequence<int, F...>) {
      ((fa[(F + 5) & 1] = read_a_frag(cur, wm * 4 + ((F + 5) & 3), (F + 5) >> 2, lane),
        [&] {
#pragma unroll
          for (int it = 3 * F; it < 3 * F + 3 && it < RA; ++it) *reinterpret_cast<v4i*>(nxt + A.la[it]) = ga[it];
          if (F == 2) write_a_scales(nxt);
        }(),
        mgroup(Pc, std::integral_constant<int, F + 4>()),
        [&] {
#pragma unroll
          for (int it = 3 * F; it < 3 * F + 3 && it < RA; ++it)
            ga[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, A.oa[it], a_so * 128, 0);
          if (F == 2) gs = __builtin_amdgcn_raw_buffer_load_b32(rs_as, osa, a_so * 4, 0);
        }()), ...);
    }(std::make_integer_sequence<int, 3>());
#pragma unroll
    for (int f = 4; f < 7; ++f) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // DS read: next fragment
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        if (t < 3 && 3 * (f - 4) + t < RA) {
          __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // DS write
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (activations)
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    // group 7 covers the reads of the next chunk's first fragment and scales
    fa[0] = read_a_frag(nxt, wm * 4, 0, lane);
    mgroup(Pc, std::integral_constant<int, 7>());
    read_asc(nxt);
    if (P == 1) {
#pragma unroll
      for (int j = 0; j < 4; ++j) bsc[j] = bsn[j];
    }
    __builtin_amdgcn_sched_barrier(0);
  };

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    int bm, bn;
    tile_coords(tile, g.tiles_m, g.tiles_n, bm, bn);
    const int m0 = bm * 256, n0 = bn * 256;
    A.init<true>(g, m0, tid);
    {
      const uint32_t row = (uint32_t)(m0 + tid);
      osa = (row < (uint32_t)g.m) ? row * ks : OOB;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t panel = (uint32_t)((n0 >> 5) + wn * 4 + j);
      const bool in = panel < (uint32_t)npanels_w;
      ob[j] = in ? panel * (uint32_t)(kcn * 4096) + 16u * lane : OOB;
      osb[j] = in ? panel * (uint32_t)((kcn >> 1) * 256) + 4u * lane : OOB;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    load_a(0);
    write_a(smem);
    load_bs(0);
    __syncthreads();
    load_a(1);
    load_b(std::integral_constant<int, 0>(), 0);
    fa[0] = read_a_frag(smem, wm * 4, 0, lane);
    read_asc(smem);
#pragma unroll
    for (int j = 0; j < 4; ++j) bsc[j] = bsn[j];
    for (int kc = 0; kc < kcn; kc += 2) {
      chunk(std::integral_constant<int, 0>(), kc);
      chunk(std::integral_constant<int, 1>(), kc + 1);
    }
    if (fast_out && m0 + 256 <= g.m && n0 + 256 <= g.n)
      store_tiles_fast<4, 4>(g, acc, sout + wave * OUT_STAGE, m0 + wm * 128, n0 + wn * 128, lane, 1.0f);
    else
      store_tiles<4, 4>(g, acc, m0 + wm * 128, n0 + wn * 128, lane, 1.0f);
  }
}

// ---------------------------------------------------------------- W4A4 (NVFP4), large token counts

// W4A4 on 256 x 256 tiles, four wavefronts (one per SIMD) of 128 x 128 =
// 4 x 4 MFMA tiles of 32 x 32 -- the largest wave tile, which minimises the
// operand expansion per MFMA: each lane expands 8 fragments of 8 elements per
// 16-wide step for 16 MFMAs. Per 128-wide chunk: 128 v_mfma_f32_32x32x16_f16
// (4096 MFMA cycles) against ~600 VALU operations of expansion.
//   weights     : codes (2 x 1 KiB wave loads per panel) and E4M3 block scales
//                 (one dword per lane) straight from the packed buffer into
//                 registers, one chunk ahead, two register sets;
//   activations : codes and block scales staged in LDS per chunk (scales
//                 converted to fp16 once per workgroup while staging);
//   expansion   : software-pipelined one step ahead of the MFMAs that use it,
//                 into two sets of fp16 fragments.
// One barrier per chunk, after step 5 (the next chunk's staging writes are
// issued at steps 4 and 5); step 6 reads the next chunk's first activation
// code half and scales, a whole step before step 7 expands them (read one
// MFMA before their use, their latency stalled the wave). Persistent grid and
// staged epilogue as in k_gemm_fp8_direct.
__global__ void __launch_bounds__(256) k_gemm_nvfp4_direct(GemmArgs g) {
  constexpr int A_CODES = 8 * 2048;              // 256 rows x 64 B of codes
  constexpr int A_STAGE = A_CODES + 256 * 16;    // + 256 rows x 8 fp16 scales
  constexpr int OUT_STAGE = 32 * (64 * 4 + 16);
  constexpr uint32_t OOB = 0x80000000u;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * A_STAGE];
  __shared__ __attribute__((aligned(16))) uint8_t sout[4 * OUT_STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r = lane & 31, gq = lane >> 5;
  const int kcn = g.k >> 7;
  const int npanels_w = (g.n + 31) >> 5;
  const int total = g.tiles_m * g.tiles_n;
  const float scale = *g.w_tscale * *g.a_tscale;
  const bool fast_out = g.out_mode == OUT_BF16 && ((reinterpret_cast<uintptr_t>(g.y) & 15) == 0) && ((g.ldy & 7) == 0);
  // A rows: lda / 2 code bytes and lda / 16 scale bytes apart; the
  // descriptors end at the last row's k / 2 and k / 16 bytes
  const uint32_t ka = (uint32_t)(g.lda >> 1), ks = (uint32_t)(g.lda >> 4);
  const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a), 0, (int)((int64_t)(g.m - 1) * ka + (g.k >> 1)), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_as = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a_bscale), 0, (int)((int64_t)(g.m - 1) * ks + (g.k >> 4)), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * kcn * 2048), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_bs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, (int)((int64_t)npanels_w * kcn * 256), 0x00020000);

  uint32_t oa[4], la[4], osa, ob[4], osb[4];
  v4i ga[4];        // staged activation codes of a chunk
  v2i gs;           // staged activation scales (one row per thread)
  v4i bc[2][4][2];  // weight codes [chunk parity][panel][half]
  uint32_t bs[2][4];  // weight E4M3 scales [chunk parity][panel]
  uint2 bf[4];      // weight fp16 scales of the current chunk
  v4i ac[2][4];     // activation codes [half][panel] of the current chunk
  uint2 af[4];      // activation fp16 scales of the current chunk
  v8h fa[2][4], fb[2][4];  // expanded fragments, two steps
  v16f acc[4][4];

  // Chunk offsets are uniform: they travel in the loads' scalar offset,
  // clamped to the last chunk (prefetches past the end re-read it in bounds;
  // their data is never multiplied). Rows and panels outside the operands
  // keep an out-of-range per-lane base.
  auto kcl = [&](int kc) __attribute__((always_inline)) { return kc < kcn ? kc : kcn - 1; };
  auto load_a = [&](int kc) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < 4; ++it) ga[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[it], kcl(kc) * 64, 0);
    gs = __builtin_amdgcn_raw_buffer_load_b64(rs_as, osa, kcl(kc) * 8, 0);
  };
  auto write_a_codes = [&](uint8_t* st, int from, int to) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < 4; ++it)
      if (it >= from && it < to) *reinterpret_cast<v4i*>(st + la[it]) = ga[it];
  };
  auto write_a_scales = [&](uint8_t* st) __attribute__((always_inline)) {
    const uint2 lo = e4m3x4_to_f16x4((uint32_t)gs.x), hi = e4m3x4_to_f16x4((uint32_t)gs.y);
    *reinterpret_cast<uint4*>(st + A_CODES + tid * 16) = make_uint4(lo.x, lo.y, hi.x, hi.y);
  };
  auto load_b = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const int kq = kcl(kc);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      bc[P][j][0] = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[j], kq * 2048, 0);
      bc[P][j][1] = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[j] + 1024, kq * 2048, 0);
      bs[P][j] = __builtin_amdgcn_raw_buffer_load_b32(rs_bs, osb[j], kq * 256, 0);
    }
  };
  auto read_a_half = [&](const uint8_t* st, int h) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      ac[h][i] = *reinterpret_cast<const v4i*>(st + (wm * 4 + i) * 2048 + h * 1024 + ((lane ^ (4 * h + 10 * gq)) * 16));
  };
  auto read_a_scales = [&](const uint8_t* st) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const uint2*>(st + A_CODES + ((wm * 4 + i) * 32 + r) * 16 + 8 * gq);
  };
  auto convert_b_scales = [&](auto Pc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
#pragma unroll
    for (int j = 0; j < 4; ++j) bf[j] = e4m3x4_to_f16x4(bs[P][j]);
  };
  // expand step s (0..7) of the chunk held in ac / af and bc[P] / bf into set D
  auto expand = [&](auto Pc, int s, int D) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const v4i c = ac[s >> 2][i];
      const uint32_t w = (uint32_t)((s & 3) == 0 ? c.x : (s & 3) == 1 ? c.y : (s & 3) == 2 ? c.z : c.w);
      fa[D][i] = dequant8_f16(w, scale_f16(af[i], s >> 1));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const v4i c = bc[P][j][s >> 2];
      const uint32_t w = (uint32_t)((s & 3) == 0 ? c.x : (s & 3) == 1 ? c.y : (s & 3) == 2 ? c.z : c.w);
      fb[D][j] = dequant8_f16(w, scale_f16(bf[j], s >> 1));
    }
  };
  auto mfmas = [&](int D) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fb[D][j], fa[D][i], acc[i][j], 0, 0, 0);
  };
  // 16 MFMAs, each followed by its share of the expansion (64 VALU + scale
  // work); LDS reads in the groups whose bit is set in rmask
  auto interleave = [&](int nvmem, unsigned rmask, int nds_w) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);  // VALU
      if (t < nvmem) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      if ((rmask >> t) & 1) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (t < nds_w) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    }
  };

  auto chunk = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const uint8_t* cur = smem + P * A_STAGE;
    uint8_t* nxt = smem + (P ^ 1) * A_STAGE;
    constexpr std::integral_constant<int, P ^ 1> Q{};
    // steps 0..3: weight loads of chunk kc + 1 (12 per lane), second code half
    // of the activations read during step 2
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s == 0) load_b(Q, kc + 1);
      if (s == 2) read_a_half(cur, 1);
      mfmas(s & 1);
      expand(Pc, s + 1, (s + 1) & 1);
      interleave(s == 0 ? 12 : 0, s == 2 ? 0xFu : 0u, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // steps 4, 5: stage the activations of chunk kc + 1, then load kc + 2
#pragma unroll
    for (int s = 4; s < 6; ++s) {
      if (s == 4) write_a_codes(nxt, 0, 2);
      else { write_a_codes(nxt, 2, 4); write_a_scales(nxt); }
      if (s == 5) load_a(kc + 2);
      mfmas(s & 1);
      expand(Pc, s + 1, (s + 1) & 1);
      interleave(s == 5 ? 5 : 0, 0u, s == 4 ? 2 : 3);
      __builtin_amdgcn_sched_barrier(0);
    }
    // the barrier that publishes chunk kc + 1 (its last writes were issued at
    // the start of step 5)
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    // step 6 reads the next chunk's first code half (its ac[0] was last
    // expanded in step 2) and, once this step's expansion has used the
    // current scales, the next chunk's scales: a step of MFMAs hides their
    // latency before step 7 expands them
    read_a_half(nxt, 0);
    mfmas(0);
    expand(Pc, 7, 1);
    read_a_scales(nxt);
    interleave(0, 0x0F0Fu, 0);
    __builtin_amdgcn_sched_barrier(0);
    // step 7: the next chunk's step-0 expansion
    convert_b_scales(Q);
    mfmas(1);
    expand(Q, 0, 0);
    interleave(0, 0u, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    int bm, bn;
    tile_coords(tile, g.tiles_m, g.tiles_n, bm, bn);
    const int m0 = bm * 256, n0 = bn * 256;
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int q = it * 256 + tid;
      const int p = q >> 7, rr = (q >> 2) & 31, c = q & 3;
      const uint32_t row = (uint32_t)(m0 + 32 * p + rr);
      oa[it] = (row < (uint32_t)g.m) ? row * ka + 16u * c : OOB;
      // slot XOR 4 h + 10 g: the 4 pieces of a row and 2 or 4 neighbouring
      // rows fall into distinct bank groups (checked on the CPU)
      la[it] = (uint32_t)(p * 2048 + (c & 1) * 1024 + (((rr + 32 * (c >> 1)) ^ (4 * (c & 1) + 10 * (c >> 1))) * 16));
    }
    {
      const uint32_t row = (uint32_t)(m0 + tid);
      osa = (row < (uint32_t)g.m) ? row * ks : OOB;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t panel = (uint32_t)((n0 >> 5) + wn * 4 + j);
      const bool in = panel < (uint32_t)npanels_w;
      ob[j] = in ? panel * (uint32_t)(kcn * 2048) + 16u * lane : OOB;
      osb[j] = in ? panel * (uint32_t)(kcn * 256) + 8u * r + 4u * gq : OOB;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // An odd chunk count takes its first chunk unpipelined (see the W8A8 kernel).
    int kc = 0;
    if (kcn & 1) {
      load_a(0);
      load_b(std::integral_constant<int, 0>(), 0);
      write_a_codes(smem, 0, 4);
      write_a_scales(smem);
      __syncthreads();
      read_a_half(smem, 0);
      read_a_half(smem, 1);
      read_a_scales(smem);
      convert_b_scales(std::integral_constant<int, 0>());
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        expand(std::integral_constant<int, 0>(), s, 0);
        mfmas(0);
      }
      __syncthreads();
      kc = 1;
    }
    if (kc < kcn) {
      load_a(kc);
      load_b(std::integral_constant<int, 0>(), kc);
      write_a_codes(smem, 0, 4);
      write_a_scales(smem);
      __syncthreads();
      load_a(kc + 1);
      read_a_half(smem, 0);
      read_a_scales(smem);
      convert_b_scales(std::integral_constant<int, 0>());
      expand(std::integral_constant<int, 0>(), 0, 0);
      for (; kc < kcn; kc += 2) {
        chunk(std::integral_constant<int, 0>(), kc);
        chunk(std::integral_constant<int, 1>(), kc + 1);
      }
    }
    if (fast_out && m0 + 256 <= g.m && n0 + 256 <= g.n)
      store_tiles_fast<4, 4>(g, acc, sout + wave * OUT_STAGE, m0 + wm * 128, n0 + wn * 128, lane, scale);
    else
      store_tiles<4, 4>(g, acc, m0 + wm * 128, n0 + wn * 128, lane, scale);
  }
}

// ---------------------------------------------------------------- MXFP4 (W4A4, MX block scaling)
// OCP MXFP4 x MXFP4 on gfx950's block-scaled matrix instruction:
// v_mfma_scale_f32_32x32x64_f8f6f4 with fp4 operands takes, per lane, 32
// E2M1 codes (16 bytes: lanes 0-31 reduction elements 0-31 of the step,
// lanes 32-63 elements 32-63) and one E8M0 scale byte for them -- exactly
// one MX block -- so the format runs at the fp4 matrix rate with no operand
// expansion at all. Same tiles and waves as k_gemm_fp8_direct (256 x 256,
// four waves of 128 x 128, persistent grid, staged epilogue); the reduction
// advances in chunks of 256 (4 MFMA steps of 64, 64 MFMAs of 32 cycles per
// wave per chunk):
//   weights     : one 1 KiB code image per panel and step, loaded straight
//                 into registers three steps ahead (a ring of four steps,
//                 refilled right after each step's last use), plus one dword
//                 per panel and chunk holding the lane's four block scales;
//   activations : 128 bytes per row and chunk staged in LDS (piece c = step
//                 s = c / 2, lane half g = c % 2; the 16-byte slot of lane
//                 32 g + row is XOR-ed with 2 s + 9 g, so that the 8 pieces
//                 of a row, written by 8 neighbouring lanes, and any 16
//                 neighbouring lanes' reads fall into distinct bank groups
//                 for 32 and 64 banks alike), the row's 8 block scales
//                 re-ordered while staging so that a lane reads its 4 as one
//                 dword; the MFMA's byte select picks step s's scale. A group
//                 of 4 fp4 MFMAs lasts about one LDS read latency, so the
//                 fragments are read two groups ahead.
// K must be a multiple of 256 (checked by the caller).
__global__ void __launch_bounds__(256) k_gemm_mxfp4_direct(GemmArgs g) {
  constexpr int A_CODES = 8 * 4096;              // 8 panels x 4 steps x 1 KiB
  constexpr int A_STAGE = A_CODES + 256 * 8;     // + 8 scale bytes per row
  constexpr int OUT_STAGE = 32 * (64 * 4 + 16);
  constexpr uint32_t OOB = 0x80000000u;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * A_STAGE];
  __shared__ __attribute__((aligned(16))) uint8_t sout[4 * OUT_STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r = lane & 31, gq = lane >> 5;
  const int kcn = g.k >> 8;                      // chunks of 256
  const int steps = g.k >> 6;
  const int npanels_w = (g.n + 31) >> 5;
  const int total = g.tiles_m * g.tiles_n;
  const bool fast_out = g.out_mode == OUT_BF16 && ((reinterpret_cast<uintptr_t>(g.y) & 15) == 0) && ((g.ldy & 7) == 0);
  const uint32_t ka = (uint32_t)(g.k >> 1), ks = (uint32_t)(g.k >> 5);  // A code / scale bytes per row
  const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a), 0, (int)((int64_t)g.m * ka), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_as = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a_bscale), 0, (int)((int64_t)g.m * ks), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * steps * 1024), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_bs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, (int)((int64_t)npanels_w * kcn * 256), 0x00020000);

  uint32_t oa[8], la[8], osa, ob[4], osb[4];
  v4i ga[8];           // staged activation codes of a chunk
  uint2 gs;            // staged activation scales of the thread's row
  v4i fb[4][4];        // weight codes, ring over steps: [step % 4][panel]
  uint32_t bsc[2][4];  // weight scales [chunk parity][panel]: byte s = step s
  uint32_t asc[2][4];  // activation scales [chunk parity][panel]: byte s = step s
  v4i fa[4];           // activation fragments, ring over MFMA groups (read two groups ahead)
  v16f acc[4][4];

  // Chunk and step offsets are uniform: they travel in the loads' scalar
  // offset, clamped to the last chunk / step (prefetches past the end re-read
  // it in bounds; their data is never multiplied). Rows and panels outside
  // the operands keep an out-of-range per-lane base.
  auto kcl = [&](int kc) __attribute__((always_inline)) { return kc < kcn ? kc : kcn - 1; };
  auto load_a = [&](int kc) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < 8; ++it) ga[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[it], kcl(kc) * 128, 0);
    const v2i t = __builtin_amdgcn_raw_buffer_load_b64(rs_as, osa, kcl(kc) * 8, 0);
    gs = make_uint2((uint32_t)t.x, (uint32_t)t.y);
  };
  // row scales of the chunk, blocks 0..7 -> [half 0: 0 2 4 6][half 1: 1 3 5 7]
  auto write_a_scales = [&](uint8_t* st) __attribute__((always_inline)) {
    const uint32_t lo = __builtin_amdgcn_perm(gs.y, gs.x, 0x06040200u);
    const uint32_t hi = __builtin_amdgcn_perm(gs.y, gs.x, 0x07050301u);
    *reinterpret_cast<uint2*>(st + A_CODES + tid * 8) = make_uint2(lo, hi);
  };
  // weight codes of global step t (= 4 x chunk + step) into ring slot S
  auto load_b = [&](auto Sc, int t) __attribute__((always_inline)) {
    constexpr int S = decltype(Sc)::value;
    const int so = (t < steps ? t : steps - 1) * 1024;
#pragma unroll
    for (int j = 0; j < 4; ++j) fb[S][j] = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[j], so, 0);
  };
  auto load_bs = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
#pragma unroll
    for (int j = 0; j < 4; ++j) bsc[P][j] = __builtin_amdgcn_raw_buffer_load_b32(rs_bs, osb[j], kcl(kc) * 256, 0);
  };
  auto read_fa = [&](const uint8_t* st, int s, int i) __attribute__((always_inline)) {
    return *reinterpret_cast<const v4i*>(st + (wm * 4 + i) * 4096 + s * 1024 + ((lane ^ (2 * s + 9 * gq)) * 16));
  };
  auto read_asc = [&](auto Pc, const uint8_t* st) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      asc[P][i] = *reinterpret_cast<const uint32_t*>(st + A_CODES + ((wm * 4 + i) * 32 + r) * 8 + 4 * gq);
  };
  // MFMA group f = (step f / 4, activation panel f % 4) on fragment fa[f % 4]
  auto mgroup = [&](auto Pc, auto Fc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value, f = decltype(Fc)::value;
    const v4i xa = fa[f & 3];
    const v8i xv = (v8i){xa.x, xa.y, xa.z, xa.w, 0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const v4i wa = fb[f >> 2][j];
      const v8i wv = (v8i){wa.x, wa.y, wa.z, wa.w, 0, 0, 0, 0};
      acc[f & 3][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wv, xv, acc[f & 3][j], 4, 4, f >> 2, (int)bsc[P][j],
                                                                       f >> 2, (int)asc[P][f & 3]);
    }
  };
  // one region: groups 4s .. 4s + NG - 1, each a fragment read for the next
  // group and 4 MFMAs; NV global loads and NW LDS writes spread over the slots
  auto pattern = [&](auto NGc, auto NVc, auto NWc) __attribute__((always_inline)) {
    constexpr int NG = decltype(NGc)::value, NV = decltype(NVc)::value, NW = decltype(NWc)::value;
#pragma unroll
    for (int f = 0; f < NG; ++f) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        if (4 * f + t < NW) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // DS write
        if (4 * f + t < NV) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // fragment reads run two groups ahead of their MFMAs: group f reads the
  // fragment of group f + 2 (for f = 14, 15: groups 0, 1 of the next chunk,
  // after the barrier that publishes it)
  auto chunk = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    using I = std::integral_constant<int, 0>;
    const uint8_t* cur = smem + P * A_STAGE;
    uint8_t* nxt = smem + (P ^ 1) * A_STAGE;
    const int t0 = 4 * kc;
    // step 0: refill slot 3 (step 3 of this chunk)
    load_b(std::integral_constant<int, 3>(), t0 + 3);
    [&]<int... F>(std::integer_sequence<int, F...>) {
      ((fa[(F + 2) & 3] = read_fa(cur, (F + 2) >> 2, (F + 2) & 3), mgroup(Pc, std::integral_constant<int, F>())), ...);
    }(std::make_integer_sequence<int, 4>());
    pattern(std::integral_constant<int, 4>(), std::integral_constant<int, 4>(), I());
    // step 1: slot 0 <- step 0 of the next chunk; next chunk's weight scales
    load_b(std::integral_constant<int, 0>(), t0 + 4);
    load_bs(std::integral_constant<int, P ^ 1>(), kc + 1);
    [&]<int... F>(std::integer_sequence<int, F...>) {
      ((fa[(F + 6) & 3] = read_fa(cur, (F + 6) >> 2, (F + 6) & 3), mgroup(Pc, std::integral_constant<int, F + 4>())), ...);
    }(std::make_integer_sequence<int, 4>());
    pattern(std::integral_constant<int, 4>(), std::integral_constant<int, 8>(), I());
    // step 2: slot 1 refill; stage the activations of chunk kc + 1 (written
    // between the fragment reads in program order), then load those of kc + 2
    const int a_so = kcl(kc + 2) * 128;
    load_b(std::integral_constant<int, 1>(), t0 + 5);
    [&]<int... F>(std::integer_sequence<int, F...>) {
      ((fa[(F + 10) & 3] = read_fa(cur, (F + 10) >> 2, (F + 10) & 3),
        *reinterpret_cast<v4i*>(nxt + la[2 * F]) = ga[2 * F],
        *reinterpret_cast<v4i*>(nxt + la[2 * F + 1]) = ga[2 * F + 1],
        mgroup(Pc, std::integral_constant<int, F + 8>()),
        ga[2 * F] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[2 * F], a_so, 0),
        ga[2 * F + 1] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[2 * F + 1], a_so, 0)), ...);
    }(std::make_integer_sequence<int, 4>());
    pattern(std::integral_constant<int, 4>(), std::integral_constant<int, 12>(), std::integral_constant<int, 8>());
    // step 3, first half: slot 2 refill, the row scales of chunk kc + 1
    load_b(std::integral_constant<int, 2>(), t0 + 6);
    write_a_scales(nxt);
    {
      const v2i t = __builtin_amdgcn_raw_buffer_load_b64(rs_as, osa, kcl(kc + 2) * 8, 0);
      gs = make_uint2((uint32_t)t.x, (uint32_t)t.y);
    }
    [&]<int... F>(std::integer_sequence<int, F...>) {
      ((fa[(F + 14) & 3] = read_fa(cur, 3, (F + 2) & 3), mgroup(Pc, std::integral_constant<int, F + 12>())), ...);
    }(std::make_integer_sequence<int, 2>());
    pattern(std::integral_constant<int, 2>(), std::integral_constant<int, 5>(), std::integral_constant<int, 1>());
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    // step 3, second half: the next chunk's first two fragments and its scales
    fa[0] = read_fa(nxt, 0, 0);
    mgroup(Pc, std::integral_constant<int, 14>());
    fa[1] = read_fa(nxt, 0, 1);
    read_asc(std::integral_constant<int, P ^ 1>(), nxt);
    mgroup(Pc, std::integral_constant<int, 15>());
    __builtin_amdgcn_sched_barrier(0);
  };

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    int bm, bn;
    tile_coords(tile, g.tiles_m, g.tiles_n, bm, bn);
    const int m0 = bm * 256, n0 = bn * 256;
#pragma unroll
    for (int it = 0; it < 8; ++it) {
      const int q = it * 256 + tid;
      const int p = q >> 8, rr = (q >> 3) & 31, c = q & 7;
      const uint32_t row = (uint32_t)(m0 + 32 * p + rr);
      oa[it] = (row < (uint32_t)g.m) ? row * ka + 16u * c : OOB;
      la[it] = (uint32_t)(p * 4096 + (c >> 1) * 1024 + (((rr + 32 * (c & 1)) ^ (2 * (c >> 1) + 9 * (c & 1))) * 16));
    }
    {
      const uint32_t row = (uint32_t)(m0 + tid);
      osa = (row < (uint32_t)g.m) ? row * ks : OOB;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t panel = (uint32_t)((n0 >> 5) + wn * 4 + j);
      const bool in = panel < (uint32_t)npanels_w;
      ob[j] = in ? panel * (uint32_t)(steps * 1024) + 16u * lane : OOB;
      osb[j] = in ? panel * (uint32_t)(kcn * 256) + 4u * lane : OOB;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    int kc = 0;
    if (kcn & 1) {  // odd chunk count: first chunk unpipelined
      load_a(0);
      load_b(std::integral_constant<int, 0>(), 0);
      load_b(std::integral_constant<int, 1>(), 1);
      load_b(std::integral_constant<int, 2>(), 2);
      load_b(std::integral_constant<int, 3>(), 3);
      load_bs(std::integral_constant<int, 0>(), 0);
#pragma unroll
      for (int it = 0; it < 8; ++it) *reinterpret_cast<v4i*>(smem + la[it]) = ga[it];
      write_a_scales(smem);
      __syncthreads();
      read_asc(std::integral_constant<int, 0>(), smem);
      [&]<int... F>(std::integer_sequence<int, F...>) {
        ((fa[F & 3] = read_fa(smem, F >> 2, F & 3), mgroup(std::integral_constant<int, 0>(), std::integral_constant<int, F>())), ...);
      }(std::make_integer_sequence<int, 16>());
      __syncthreads();
      kc = 1;
    }
    if (kc < kcn) {
      load_a(kc);
#pragma unroll
      for (int it = 0; it < 8; ++it) *reinterpret_cast<v4i*>(smem + la[it]) = ga[it];
      write_a_scales(smem);
      __syncthreads();
      load_a(kc + 1);
      load_b(std::integral_constant<int, 0>(), 4 * kc);
      load_b(std::integral_constant<int, 1>(), 4 * kc + 1);
      load_b(std::integral_constant<int, 2>(), 4 * kc + 2);
      load_bs(std::integral_constant<int, 0>(), kc);
      fa[0] = read_fa(smem, 0, 0);
      fa[1] = read_fa(smem, 0, 1);
      read_asc(std::integral_constant<int, 0>(), smem);
      for (; kc < kcn; kc += 2) {
        chunk(std::integral_constant<int, 0>(), kc);
        chunk(std::integral_constant<int, 1>(), kc + 1);
      }
    }
    // no tensor scales in MX: the block scales are applied inside the MFMAs
    if (fast_out && m0 + 256 <= g.m && n0 + 256 <= g.n)
      store_tiles_fast<4, 4>(g, acc, sout + wave * OUT_STAGE, m0 + wm * 128, n0 + wn * 128, lane, 1.0f);
    else
      store_tiles<4, 4>(g, acc, m0 + wm * 128, n0 + wn * 128, lane, 1.0f);
  }
}

// ---------------------------------------------------------------- W4A16, large token counts
// W4A16 (bf16 activations, NVFP4 weights) past the ridge point: the tile and
// wave layout of the W4A4 kernel (256 x 256 tiles, four waves of 128 x 128,
// persistent grid), on v_mfma_f32_32x32x16_bf16.
//   weights     : codes and E4M3 block scales straight from the packed buffer
//                 into registers one chunk ahead (as in k_gemm_nvfp4_direct);
//                 each 8-code step fragment is expanded to bf16 with its block
//                 scale (exact: E2M1 x E4M3 has at most 6 significant bits):
//                 4 conversions to fp32, 8 multiplies, 4 byte permutes (gfx950
//                 has no packed bf16 multiply);
//   activations : bf16 rows staged in LDS per chunk (256 rows x 256 B). The
//                 reduction order is the weights' permuted one: step s, lane
//                 half g holds k = 64 g + 8 s + [0, 8), the 16-byte piece
//                 c = 8 g + s of the row's chunk. Piece c of row r of a panel
//                 sits in 1 KiB step block s at slot (r + 32 g) ^ (s + 8 g): the
//                 16 lanes that stage one row and the fragment reads of any 8
//                 or 16 neighbouring lanes fall into distinct bank groups (32
//                 or 64 banks; checked on the CPU). Staged through registers
//                 in four quarters of four pieces per thread per chunk, two
//                 register sets, stored at steps 2, 3, 5 and 6.
// One barrier per chunk, after step 6; step 7 reads the next chunk's first
// fragments. The bf16 output staging of the epilogue reuses activation
// stage 1, which no wave reads after the last chunk's barrier (a tile's
// chunks run in pairs, stage 0 then 1), and the next tile writes it only
// after its first barrier.
__global__ void __launch_bounds__(256) k_gemm_w4a16_direct(GemmArgs g) {
  constexpr int A_STAGE = 8 * 8192;              // 256 rows x 128 bf16
  constexpr int OUT_STAGE = 32 * (64 * 4 + 16);
  constexpr uint32_t OOB = 0x80000000u;
  static_assert(4 * OUT_STAGE <= A_STAGE, "the output staging fits in one activation stage");
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * A_STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r = lane & 31, gq = lane >> 5;
  const int kcn = g.k >> 7;
  const int npanels_w = (g.n + 31) >> 5;
  const int total = g.tiles_m * g.tiles_n;
  const float scale = *g.w_tscale;
  const bool fast_out = g.out_mode == OUT_BF16 && ((reinterpret_cast<uintptr_t>(g.y) & 15) == 0) && ((g.ldy & 7) == 0);
  const uint32_t lda2 = (uint32_t)(g.lda * 2);
  const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a), 0, (int)((int64_t)(g.m - 1) * lda2 + g.k * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * kcn * 2048), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_bs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, (int)((int64_t)npanels_w * kcn * 256), 0x00020000);
  // staging: thread tid copies piece c = tid % 16 of rows 16 i + tid / 16,
  // i = 0 .. 15; its LDS slots depend only on i % 2 (and i / 2 through the
  // panel, a constant offset)
  const int cpc = tid & 15, s_c = cpc & 7, g_c = cpc >> 3, rlo = tid >> 4;
  uint32_t la_pair[2];
#pragma unroll
  for (int h = 0; h < 2; ++h)
    la_pair[h] = (uint32_t)(s_c * 1024 + ((((16 * h + rlo) + 32 * g_c) ^ (s_c + 8 * g_c)) * 16));

  uint32_t oa[16], ob[4], osb[4];
  v4i ga[8];            // two staging quarters (register sets 0 and 1)
  v4i bc[2][4][2];      // weight codes [chunk parity][panel][half]
  uint32_t bs[2][4];    // weight E4M3 scales [chunk parity][panel]
  float sw[4][4];       // weight block scales of the current chunk, fp32 [panel][block]
  v8bf fa[2][4], fb[2][4];
  v16f acc[4][4];

  auto kcl = [&](int kc) __attribute__((always_inline)) { return kc < kcn ? kc : kcn - 1; };
  // quarter q of the thread's 16 pieces (rows 16 i + tid / 16, i = 4 q ..
  // 4 q + 3) through register set q % 2
  auto load_a = [&](int kc, int q) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < 4; ++it)
      ga[4 * (q & 1) + it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[4 * q + it], kcl(kc) * 256, 0);
  };
  auto write_a = [&](uint8_t* st, int q) __attribute__((always_inline)) {
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int i = 4 * q + it;
      *reinterpret_cast<v4i*>(st + (i >> 1) * 8192 + la_pair[i & 1]) = ga[4 * (q & 1) + it];
    }
  };
  auto load_b = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const int kq = kcl(kc);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      bc[P][j][0] = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[j], kq * 2048, 0);
      bc[P][j][1] = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[j] + 1024, kq * 2048, 0);
      bs[P][j] = __builtin_amdgcn_raw_buffer_load_b32(rs_bs, osb[j], kq * 256, 0);
    }
  };
  auto read_a = [&](const uint8_t* st, int s, int D) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      fa[D][i] = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4i*>(
          st + (wm * 4 + i) * 8192 + s * 1024 + ((lane ^ (s + 8 * gq)) * 16)));
  };
  // the lane's four E4M3 block scales of each panel, exactly (never negative or NaN)
  auto convert_b_scales = [&](auto Pc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const v2f lo = __builtin_amdgcn_cvt_pk_f32_fp8((int)bs[P][j], false);
      const v2f hi = __builtin_amdgcn_cvt_pk_f32_fp8((int)bs[P][j], true);
      sw[j][0] = lo[0]; sw[j][1] = lo[1]; sw[j][2] = hi[0]; sw[j][3] = hi[1];
    }
  };
  auto expand = [&](auto Pc, int s, int D) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const v4i c = bc[P][j][s >> 2];
      const uint32_t w = (uint32_t)((s & 3) == 0 ? c.x : (s & 3) == 1 ? c.y : (s & 3) == 2 ? c.z : c.w);
      fb[D][j] = __builtin_bit_cast(v8bf, dequant8_bf16(w, sw[j][s >> 1]));
    }
  };
  auto mfmas = [&](int D) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[D][j], fa[D][i], acc[i][j], 0, 0, 0);
  };
  // 16 MFMAs, each followed by its share of the next step's expansion (64 VALU)
  auto interleave = [&](int nvmem, int nds_r, int nds_w) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < 16; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);  // VALU
      if (t < nvmem) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      if (t < nds_r) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if (t < nds_w) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    }
  };

  auto chunk = [&](auto Pc, int kc) __attribute__((always_inline)) {
    constexpr int P = decltype(Pc)::value;
    const uint8_t* cur = smem + P * A_STAGE;
    uint8_t* nxt = smem + (P ^ 1) * A_STAGE;
    constexpr std::integral_constant<int, P ^ 1> Q{};
#pragma unroll
    for (int s = 0; s < 7; ++s) {
      // the activations of chunk kc + 1 in quarters of four pieces through
      // two register sets: quarters 0 and 1 loaded in step 0, stored in steps
      // 2 and 3, where quarters 2 and 3 are loaded into the freed sets and
      // stored in steps 5 and 6 (two or three steps for each load); at most
      // four stores and four loads per step keep the compiler on the
      // MFMA / expansion interleave
      if (s == 0) { load_b(Q, kc + 1); load_a(kc + 1, 0); load_a(kc + 1, 1); }
      if (s == 2) { write_a(nxt, 0); load_a(kc + 1, 2); }
      if (s == 3) { write_a(nxt, 1); load_a(kc + 1, 3); }
      if (s == 5) write_a(nxt, 2);
      if (s == 6) write_a(nxt, 3);
      read_a(cur, s + 1, (s + 1) & 1);
      mfmas(s & 1);
      expand(Pc, s + 1, (s + 1) & 1);
      interleave(s == 0 ? 20 : (s == 2 || s == 3) ? 4 : 0, 4, (s == 2 || s == 3 || s >= 5) ? 4 : 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    // step 7 covers the next chunk's first reads and its step-0 expansion
    read_a(nxt, 0, 0);
    convert_b_scales(Q);
    mfmas(1);
    expand(Q, 0, 0);
    interleave(0, 4, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
    int bm, bn;
    tile_coords(tile, g.tiles_m, g.tiles_n, bm, bn);
    const int m0 = bm * 256, n0 = bn * 256;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t row = (uint32_t)(m0 + 16 * i + rlo);
      oa[i] = (row < (uint32_t)g.m) ? row * lda2 + 16u * cpc : OOB;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t panel = (uint32_t)((n0 >> 5) + wn * 4 + j);
      const bool in = panel < (uint32_t)npanels_w;
      ob[j] = in ? panel * (uint32_t)(kcn * 2048) + 16u * lane : OOB;
      osb[j] = in ? panel * (uint32_t)(kcn * 256) + 8u * r + 4u * gq : OOB;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    // An odd chunk count takes its first chunk unpipelined.
    int kc = 0;
    if (kcn & 1) {
      load_b(std::integral_constant<int, 0>(), 0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        load_a(0, q);
        write_a(smem, q);
      }
      __syncthreads();
      convert_b_scales(std::integral_constant<int, 0>());
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        read_a(smem, s, 0);
        expand(std::integral_constant<int, 0>(), s, 0);
        mfmas(0);
      }
      __syncthreads();
      kc = 1;
    }
    if (kc < kcn) {
      load_b(std::integral_constant<int, 0>(), kc);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        load_a(kc, q);
        write_a(smem, q);
      }
      __syncthreads();
      read_a(smem, 0, 0);
      convert_b_scales(std::integral_constant<int, 0>());
      expand(std::integral_constant<int, 0>(), 0, 0);
      for (; kc < kcn; kc += 2) {
        chunk(std::integral_constant<int, 0>(), kc);
        chunk(std::integral_constant<int, 1>(), kc + 1);
      }
    }
    if (fast_out && m0 + 256 <= g.m && n0 + 256 <= g.n)
      store_tiles_fast<4, 4>(g, acc, smem + A_STAGE + wave * OUT_STAGE, m0 + wm * 128, n0 + wn * 128, lane, scale);
    else
      store_tiles<4, 4>(g, acc, m0 + wm * 128, n0 + wn * 128, lane, scale);
  }
}

// ---------------------------------------------------------------- W4A16, up to 1024 tokens
// bf16 activations against NVFP4 weights when the output is too small to
// fill the chip with large tiles (the text-encoder linears). A workgroup
// owns NP 32-row weight panels (32 NP output columns) and one block of 32 MT
// activation rows; its NW wavefronts split the reduction dimension (chunk kc
// goes to wave kc % NW) and their partial accumulators are summed through
// LDS at the end, so a workgroup's latency is a few chunks, not K / 128 of
// them. Every workgroup re-reads its activation rows, so NP sets how often
// the activations cross L2 (M K 2 bytes per 32 NP output columns). Each wave
// reads the packed weight straight from memory in operand order (32 B of
// codes + 4 B of scales per lane, panel and chunk). Activations are
// read row-contiguously (16 lanes per 256-byte row run of a chunk: 8 cache
// lines per load instruction instead of the 64 that loading the MFMA
// fragments directly would touch) into a wave-private LDS area, stored in
// fragment order [step][lane][16 B] with the lane slot XOR-ed by 4 * step
// (conflict-free writes and reads; LDS operations of one wave complete in
// order, so no barrier is needed). With XLDS false (a few activation rows,
// where nearly all lanes of such a load would be out of range anyway) each
// lane loads its fragments directly. Offsets past the last chunk or row get
// the top bit set and read zeros.
template <int MT, int NP, int NW, int D, bool XLDS>
__global__ void __launch_bounds__(64 * NW) k_w4a16_splitk(GemmArgs g) {
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int XS = 8192;  // one 32-row block of one chunk: 32 rows x 256 B
  constexpr int RED = NW * MT * 4096;  // one panel's partial tiles of all waves
  constexpr int STG = XLDS ? NW * MT * XS : 0;
  __shared__ __attribute__((aligned(16))) uint8_t smem[STG > RED ? STG : RED];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int panel = blockIdx.x;
  const int mb = blockIdx.y * 32 * MT;
  const int kcn = g.k >> 7;
  const int r = lane & 31, gq = lane >> 5;
  const int npanels_w = (g.n + 31) >> 5;
  const __amdgpu_buffer_rsrc_t rs_w = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * kcn * 2048), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_ws = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, (int)((int64_t)npanels_w * kcn * 256), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_x = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a), 0, (int)(((int64_t)(g.m - 1) * g.lda + g.k) * 2), 0x00020000);
  uint32_t ow[NP], ows[NP];
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    const int pj = panel * NP + j;
    const bool in = pj < npanels_w;
    ow[j] = in ? (uint32_t)(pj * kcn * 2048 + lane * 16) : OOB;
    ows[j] = in ? (uint32_t)(pj * kcn * 256 + r * 8 + 4 * gq) : OOB;
  }
  // row-contiguous activation pieces: load it covers rows 4 it .. 4 it + 3 of
  // the block; lane -> row 4 it + lane / 16, piece c = lane % 16 (elements
  // 8c .. 8c + 7 of the chunk) = step c % 8 of lane half c / 8
  // (direct: lane loads elements [64 g + 8 s, +8) of row r at step s)
  const int prow = XLDS ? (lane >> 4) : r, pc = XLDS ? (lane & 15) : 8 * gq;
  uint32_t ox[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int row = mb + 32 * i + prow;  // + 4 it when staged
    ox[i] = (row < g.m) ? (uint32_t)(((int64_t)row * g.lda + 8 * pc) * 2) : OOB;
  }
  const uint32_t xrow4 = (uint32_t)(4 * g.lda * 2);  // bytes per 4 rows
  const int srow_lim = g.m - mb - prow;               // rows of the block this lane may read: 4 it < srow_lim
  uint8_t* xw = smem + wave * MT * XS;
  // piece (row 4 it + prow, c) belongs to lane slot (row + 32 g) of step
  // s = c % 8, g = c / 8, stored at slot ^ 4s: 4 (it ^ s) + prow + 32 g
  const int ps = pc & 7;
  const int wbase = ps * 1024 + (prow + 32 * (pc >> 3)) * 16;

  struct Chunk {
    v4i c0[NP], c1[NP];  // 64 E2M1 codes of the lane's row of each weight panel
    uint32_t sc[NP];     // their 4 E4M3 block scales
    v4i x[MT][8];        // row-contiguous activation pieces
  };
  auto load = [&](Chunk& C, int kc) __attribute__((always_inline)) {
    const uint32_t hi = kc < kcn ? 0u : OOB;
#pragma unroll
    for (int j = 0; j < NP; ++j) {
      C.c0[j] = __builtin_amdgcn_raw_buffer_load_b128(rs_w, (ow[j] + kc * 2048) | hi, 0, 0);
      C.c1[j] = __builtin_amdgcn_raw_buffer_load_b128(rs_w, (ow[j] + kc * 2048 + 1024) | hi, 0, 0);
      C.sc[j] = __builtin_amdgcn_raw_buffer_load_b32(rs_ws, (ows[j] + kc * 256) | hi, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int it = 0; it < 8; ++it) {
        if (XLDS) {
          const uint32_t rowhi = (4 * it < srow_lim - 32 * i) ? 0u : OOB;
          C.x[i][it] = __builtin_amdgcn_raw_buffer_load_b128(rs_x, (ox[i] + it * xrow4 + kc * 256) | hi | rowhi, 0, 0);
        } else {
          C.x[i][it] = __builtin_amdgcn_raw_buffer_load_b128(rs_x, (ox[i] + it * 16 + kc * 256) | hi, 0, 0);
        }
      }
  };
  v16f acc[NP][MT];
#pragma unroll
  for (int j = 0; j < NP; ++j)
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[j][i][v] = 0.0f;
  auto compute = [&](const Chunk& C) __attribute__((always_inline)) {
    if (XLDS) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int it = 0; it < 8; ++it)
          *reinterpret_cast<v4i*>(xw + i * XS + wbase + 64 * (it ^ ps)) = C.x[i][it];
    }
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      v4i xf[MT];
#pragma unroll
      for (int i = 0; i < MT; ++i)
        xf[i] = XLDS ? *reinterpret_cast<const v4i*>(xw + i * XS + s * 1024 + ((lane ^ (4 * s)) * 16)) : C.x[i][s];
#pragma unroll
      for (int j = 0; j < NP; ++j) {
        const v4i cc = (s < 4) ? C.c0[j] : C.c1[j];
        const uint32_t w = (uint32_t)((s & 3) == 0 ? cc.x : (s & 3) == 1 ? cc.y : (s & 3) == 2 ? cc.z : cc.w);
        const v8bf wb = __builtin_bit_cast(v8bf, dequant8_bf16(w, dec_e4m3_scale(C.sc[j] >> (8 * (s >> 1)))));
#pragma unroll
        for (int i = 0; i < MT; ++i)
          acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wb, __builtin_bit_cast(v8bf, xf[i]), acc[j][i], 0, 0, 0);
      }
    }
  };
  // a wave's chunks kc = wave + NW t are loaded D at a time, all D before any
  // is used, so a short reduction costs one memory latency
  for (int base = wave; base < kcn; base += D * NW) {
    Chunk C[D];
#pragma unroll
    for (int d = 0; d < D; ++d) load(C[d], base + d * NW);
#pragma unroll
    for (int d = 0; d < D; ++d)
      if (base + d * NW < kcn) compute(C[d]);
  }

  // sum the NW partial tiles through LDS (the staging area is reused after a
  // barrier), one panel at a time: thread t owns 4 consecutive outputs
  // (tile i, lane l, quad q) and writes them as one 8-byte bf16 store
  float* red = reinterpret_cast<float*>(smem);  // [NW][MT][64][16]
  const float c = *g.w_tscale;
#pragma unroll
  for (int j = 0; j < NP; ++j) {
    __syncthreads();
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(red + ((wave * MT + i) * 64 + lane) * 16 + 4 * q) =
            make_float4(acc[j][i][4 * q], acc[j][i][4 * q + 1], acc[j][i][4 * q + 2], acc[j][i][4 * q + 3]);
    __syncthreads();
    for (int t = threadIdx.x; t < MT * 256; t += 64 * NW) {
      const int i = t >> 8, l = (t >> 2) & 63, q = t & 3;
      float4 sum = *reinterpret_cast<const float4*>(red + (i * 64 + l) * 16 + 4 * q);
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        const float4 v = *reinterpret_cast<const float4*>(red + ((w * MT + i) * 64 + l) * 16 + 4 * q);
        sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
      }
      const int m = mb + 32 * i + (l & 31);
      const int n = (panel * NP + j) * 32 + 8 * q + 4 * (l >> 5);
      if (m >= g.m || n >= g.n) continue;
      store4(g, m, n, sum.x * c, sum.y * c, sum.z * c, sum.w * c, out_vec(g), out_rscale(g));
    }
  }
}

// W4A16 with very few activation rows (2 .. 16) against a wide weight (a
// weight pool streamed once): HBM-bound, so the weight stream is all that
// matters. A persistent workgroup stages the activation rows in LDS once (row
// pitch padded by 16 bytes, so that the rows of a fragment read fall in
// different banks); each of its waves then owns whole 32-row weight panels
// (no split of the reduction), walking the panel's chunks in groups of D with
// the next group's weight loads issued before the current group's MFMAs, so
// every wave keeps D chunks (D x 2.3 KiB) in flight (D = 4: six chunks
// spill registers at m > 8 and are slower at m <= 8). The weights are read
// once, with non-temporal loads.
//
// Each MFMA step covers exactly one 16-block, so the block scale is applied
// to the step's product instead of to every weight: the packed order gives
// lane (r, g) the codes of k = 64 g + 8 s' + [0, 8) in dword s', and one
// cross-half swap per dword pair (lanes 32..63 of dword 2 j with lanes 0..31
// of dword 2 j + 1) leaves every lane with k = 16 s + 8 g + [0, 8) for step s
// in dword s (j) and s + 4 (j + 4). The codes then decode straight to bf16
// (one instruction per pair, no multiply), the activations are the A operand
// (rows m), the weights the B operand (columns n = panel row r), and the
// step's 32 x 32 product, computed from a zero accumulator, is added to the
// MV useful rows of the running sum with the lane's own block scale (column
// n), one step late, so that the FMAs do not wait on the MFMA just issued:
// MV = 4 for m <= 8, 8 for m <= 16. Lanes of activation rows past m read
// an extra all-zero row. Requires m <= 16 and (m + 1) rows within the LDS
// budget (checked by the launcher).
template <int D, int MV, int NWV = 8>
__global__ void __launch_bounds__(64 * NWV) k_w4a16_stream(GemmArgs g) {
  constexpr uint32_t OOB = 0x80000000u;
  extern __shared__ __attribute__((aligned(16))) uint8_t xl[];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 31, gq = lane >> 5;
  const int kcn = g.k >> 7;
  const int npan = (g.n + 31) >> 5;
  const int pitch = g.k * 2 + 16;
  // stage the activation rows and one zero row (16 bytes per thread and step)
  {
    const int pieces = g.k >> 3;  // 16-byte pieces per row
    for (int t = threadIdx.x; t < (g.m + 1) * pieces; t += 64 * NWV) {
      const int row = t / pieces, c = t - row * pieces;
      *reinterpret_cast<uint4*>(xl + row * pitch + c * 16) =
          (row < g.m) ? *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(g.a) + (int64_t)row * g.lda + 8 * c)
                      : make_uint4(0u, 0u, 0u, 0u);
    }
  }
  __syncthreads();
  const __amdgpu_buffer_rsrc_t rs_w = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npan * kcn * 2048), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_ws = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, (int)((int64_t)npan * kcn * 256), 0x00020000);
  const uint8_t* xrd = xl + min(r, g.m) * pitch + 16 * gq;  // + kc * 256 + s * 32: k = 16 s + 8 g + [0, 8)
  const float c = *g.w_tscale;
  struct W { v4i c0, c1; uint2 sc; };
  W buf[2][D];
  auto load = [&](W (&b)[D], int panel, int kc0) __attribute__((always_inline)) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int kc = kc0 + d;
      const uint32_t o = (kc < kcn && panel < npan) ? (uint32_t)((panel * kcn + kc) * 2048 + lane * 16) : OOB;
      const uint32_t os = (kc < kcn && panel < npan) ? (uint32_t)((panel * kcn + kc) * 256 + r * 8) : OOB;
      b[d].c0 = __builtin_amdgcn_raw_buffer_load_b128(rs_w, o, 0, kNT);
      b[d].c1 = __builtin_amdgcn_raw_buffer_load_b128(rs_w, o + 1024, 0, kNT);
      b[d].sc = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rs_ws, os, 0, kNT));
    }
  };
  float acc[MV];
  auto compute = [&](const W (&b)[D], int kc0) __attribute__((always_inline)) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      if (kc0 + d >= kcn) break;
      const uint32_t dw[8] = {(uint32_t)b[d].c0.x, (uint32_t)b[d].c0.y, (uint32_t)b[d].c0.z, (uint32_t)b[d].c0.w,
                              (uint32_t)b[d].c1.x, (uint32_t)b[d].c1.y, (uint32_t)b[d].c1.z, (uint32_t)b[d].c1.w};
      uint32_t st[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const auto p = __builtin_amdgcn_permlane32_swap(dw[2 * j], dw[2 * j + 1], false, false);
        st[j] = p[0];
        st[j + 4] = p[1];
      }
      // the row's eight block scales (E4M3, never negative or NaN), exactly
      const v2f s01 = __builtin_amdgcn_cvt_pk_f32_fp8((int)b[d].sc.x, false), s23 = __builtin_amdgcn_cvt_pk_f32_fp8((int)b[d].sc.x, true);
      const v2f s45 = __builtin_amdgcn_cvt_pk_f32_fp8((int)b[d].sc.y, false), s67 = __builtin_amdgcn_cvt_pk_f32_fp8((int)b[d].sc.y, true);
      const float sc[8] = {s01[0], s01[1], s23[0], s23[1], s45[0], s45[1], s67[0], s67[1]};
      // step s's product is scaled and summed after step s + 1's MFMA is issued
      v16f t[2];
#pragma unroll
      for (int s = 0; s <= 8; ++s) {
        if (s < 8) {
          const uint4 wq = make_uint4(__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(st[s], 1.0f, 0)),
                                      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(st[s], 1.0f, 1)),
                                      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(st[s], 1.0f, 2)),
                                      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(st[s], 1.0f, 3)));
          const uint4 xv = *reinterpret_cast<const uint4*>(xrd + (kc0 + d) * 256 + s * 32);
          t[s & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, xv), __builtin_bit_cast(v8bf, wq),
                                                             (v16f){}, 0, 0, 0);
        }
        if (s > 0)
#pragma unroll
          for (int v = 0; v < MV; ++v) acc[v] = __builtin_fmaf(t[(s - 1) & 1][v], sc[s - 1], acc[v]);
      }
    }
  };
  const int nw = gridDim.x * NWV;
  int panel = blockIdx.x * NWV + wave;
  int kc0 = 0;
  // one group of D chunks: load the group after it into nb while computing cb;
  // false once the wave has no panel left. The loop below alternates the two
  // register sets in straight-line code (a runtime set index made the
  // compiler copy the loaded sets around every iteration).
  auto group = [&](W (&cb)[D], W (&nb)[D]) __attribute__((always_inline)) {
    // the group after this one: next chunks of this panel, or the next panel
    int np_ = panel, nk = kc0 + D;
    if (nk >= kcn) { np_ = panel + nw; nk = 0; }
    if (kc0 == 0)
#pragma unroll
      for (int v = 0; v < MV; ++v) acc[v] = 0.0f;
    load(nb, np_, nk);
    compute(cb, kc0);
    if (nk == 0) {
      // panel done: lane (r, g) holds column n = 32 panel + r of rows 8 (v / 4) + 4 g + v % 4
      const int n = panel * 32 + r;
      if (n < g.n) {
#pragma unroll
        for (int v = 0; v < MV; ++v) {
          const int m = 8 * (v >> 2) + 4 * gq + (v & 3);
          if (m >= g.m) continue;
          const float y = acc[v] * c;
          if (g.out_mode == OUT_F32) reinterpret_cast<float*>(g.y)[(int64_t)m * g.ldy + n] = y;
          else reinterpret_cast<uint16_t*>(g.y)[(int64_t)m * g.ldy + n] = (uint16_t)pk_bf16(y, 0.0f);
        }
      }
    }
    panel = np_;
    kc0 = nk;
    return panel < npan;
  };
  if (panel < npan) load(buf[0], panel, 0);
  while (panel < npan) {
    if (!group(buf[0], buf[1])) break;
    group(buf[1], buf[0]);
  }
}

// W4A16 with one activation row against a wide weight: a matrix-vector
// product, so no matrix instruction. The panel walk and the double-buffered
// load groups are those of k_w4a16_stream. In the packed order lane (r, g)
// holds, per chunk, the 64 codes of weight row r at k = 64 g + [0, 64): four
// whole 16-blocks (blocks 4 g .. 4 g + 3) with their four scale bytes. The lane decodes two
// codes per instruction to bf16, takes the dot product with the activation
// pairs (one dot2 per pair, fp32 sum, subnormals kept), and multiplies each
// block's partial sum by its E4M3 scale once, instead of scaling every
// element: about 1.1 vector instructions per weight.
// The two lanes of a row are summed at the end of the panel. The weights are
// read once, with non-temporal loads (measured with the caches evicted before
// every call: ~10% faster than ordinary loads). With 3 chunks per group the
// kernel needs ~110 registers, so two workgroups share a CU. Requires m == 1
// and the row within the LDS budget (checked by the launcher).
template <int D>
__global__ void __launch_bounds__(512, 4) k_w4a16_gemv(GemmArgs g) {
  constexpr uint32_t OOB = 0x80000000u;
  extern __shared__ __attribute__((aligned(16))) uint8_t xl[];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 31, gq = lane >> 5;
  const int kcn = g.k >> 7;
  const int npan = (g.n + 31) >> 5;
  for (int t = threadIdx.x; t < (g.k >> 3); t += 512)
    *reinterpret_cast<uint4*>(xl + t * 16) = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(g.a) + 8 * t);
  __syncthreads();
  const __amdgpu_buffer_rsrc_t rs_w = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npan * kcn * 2048), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_ws = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, (int)((int64_t)npan * kcn * 256), 0x00020000);
  const uint8_t* xrd = xl + 128 * gq;  // + kc * 256 + s * 16: activations k = 64 g + 8 s + [0, 8)
  const float c = *g.w_tscale;
  struct W { v4i c0, c1; uint32_t sc; };
  W buf[2][D];
  auto load = [&](W (&b)[D], int panel, int kc0) __attribute__((always_inline)) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int kc = kc0 + d;
      const uint32_t o = (kc < kcn && panel < npan) ? (uint32_t)((panel * kcn + kc) * 2048 + lane * 16) : OOB;
      const uint32_t os = (kc < kcn && panel < npan) ? (uint32_t)((panel * kcn + kc) * 256 + r * 8 + 4 * gq) : OOB;
      b[d].c0 = __builtin_amdgcn_raw_buffer_load_b128(rs_w, o, 0, kNT);
      b[d].c1 = __builtin_amdgcn_raw_buffer_load_b128(rs_w, o + 1024, 0, kNT);
      b[d].sc = __builtin_amdgcn_raw_buffer_load_b32(rs_ws, os, 0, kNT);
    }
  };
  float acc = 0.0f;
  auto compute = [&](const W (&b)[D], int kc0) __attribute__((always_inline)) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      if (kc0 + d >= kcn) break;
      const uint32_t cw[8] = {(uint32_t)b[d].c0.x, (uint32_t)b[d].c0.y, (uint32_t)b[d].c0.z, (uint32_t)b[d].c0.w,
                              (uint32_t)b[d].c1.x, (uint32_t)b[d].c1.y, (uint32_t)b[d].c1.z, (uint32_t)b[d].c1.w};
      // the four block scales (E4M3, never negative or NaN), exactly
      const v2f s01 = __builtin_amdgcn_cvt_pk_f32_fp8((int)b[d].sc, false), s23 = __builtin_amdgcn_cvt_pk_f32_fp8((int)b[d].sc, true);
      const float sc[4] = {s01[0], s01[1], s23[0], s23[1]};
#pragma unroll
      for (int j = 0; j < 4; ++j) {  // block 4 g + j: codes cw[2 j], cw[2 j + 1]
        float p = 0.0f;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int s = 2 * j + h;
          // (pairs taken as uint4 fields: a bit_cast of an int-vector element
          // to v2bf is compiled as element 0 for every index by this compiler)
          const uint4 xv = *reinterpret_cast<const uint4*>(xrd + (kc0 + d) * 256 + s * 16);
          p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw[s], 1.0f, 0),
                                              __builtin_bit_cast(v2bf, xv.x), p, false);
          p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw[s], 1.0f, 1),
                                              __builtin_bit_cast(v2bf, xv.y), p, false);
          p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw[s], 1.0f, 2),
                                              __builtin_bit_cast(v2bf, xv.z), p, false);
          p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(cw[s], 1.0f, 3),
                                              __builtin_bit_cast(v2bf, xv.w), p, false);
        }
        acc = __builtin_fmaf(p, sc[j], acc);
      }
    }
  };
  const int nw = gridDim.x * 8;
  int panel = blockIdx.x * 8 + wave;
  int kc0 = 0, cur = 0;
  if (panel < npan) load(buf[0], panel, 0);
  while (panel < npan) {
    int np_ = panel, nk = kc0 + D;
    if (nk >= kcn) { np_ = panel + nw; nk = 0; }
    if (cur == 0) { load(buf[1], np_, nk); compute(buf[0], kc0); }
    else { load(buf[0], np_, nk); compute(buf[1], kc0); }
    cur ^= 1;
    if (nk == 0) {
      // panel done: row r's two halves sit in lanes r and r + 32
      const float v = (acc + __shfl_xor(acc, 32)) * c;
      acc = 0.0f;
      const int n = panel * 32 + r;
      if (gq == 0 && n < g.n) {
        if (g.out_mode == OUT_F32) reinterpret_cast<float*>(g.y)[n] = v;
        else reinterpret_cast<uint16_t*>(g.y)[n] = (uint16_t)pk_bf16(v, 0.0f);
      }
    }
    panel = np_;
    kc0 = nk;
  }
}

// k = 0: every output is zero (NVFP4: zero codes and zero block scales, one
// thread per code byte).
__global__ void k_zero_rows(void* y, uint8_t* y_bscale, int64_t m, int64_t n, int64_t ldy, int out_mode) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t w = (out_mode == OUT_NVFP4) ? n / 2 : n;  // items per row
  if (t >= m * w) return;
  const int64_t r = t / w, c = t - r * w;
  if (out_mode == OUT_F32) reinterpret_cast<float*>(y)[r * ldy + c] = 0.0f;
  else if (out_mode == OUT_FP8) reinterpret_cast<uint8_t*>(y)[r * ldy + c] = 0;
  else if (out_mode == OUT_NVFP4) {
    reinterpret_cast<uint8_t*>(y)[r * (ldy / 2) + c] = 0;
    if (c % 8 == 0) y_bscale[r * (ldy / 16) + c / 8] = 0;
  } else reinterpret_cast<uint16_t*>(y)[r * ldy + c] = 0;
}

template <int MODE, int WM, int WN, int TM, int TN, int DEPTH = 1>
static hipError_t run(GemmArgs g, hipStream_t st) {
  constexpr int BM = 32 * TM * WM, BN = 32 * TN * WN;
  g.tiles_m = (g.m + BM - 1) / BM;
  g.tiles_n = (g.n + BN - 1) / BN;
  hipLaunchKernelGGL((k_gemm<MODE, WM, WN, TM, TN, DEPTH>), dim3(g.tiles_m * g.tiles_n), dim3(64 * WM * WN), 0, st, g);
  return hipGetLastError();
}



// Compute units of the current device, queried once per device. Persistent
// grids launch at most this many workgroups.
static int device_cus() {
  static int cache[64];  // 0 = not queried yet
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = __atomic_load_n(&cache[dev], __ATOMIC_RELAXED);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    __atomic_store_n(&cache[dev], n, __ATOMIC_RELAXED);
  }
  return n;
}

hipError_t launch_gemm(int a_fmt, const void* a, const uint8_t* a_bscale, const float* a_tscale,
                       int64_t lda, const uint8_t* w_packed, int64_t m, int64_t n, int64_t k,
                       void* y, int64_t ldy, int out_mode, const float* y_scale, uint8_t* y_bscale,
                       hipStream_t st) {
  if (m == 0 || n == 0) return hipSuccess;
  if (k == 0) {
    hipLaunchKernelGGL(k_zero_rows, dim3((unsigned)((m * n + 255) / 256)), dim3(256), 0, st, y, y_bscale, m, n, ldy,
                       out_mode);
    return hipGetLastError();
  }
  const int w_fmt = (a_fmt == 1 || a_fmt == 3 || a_fmt == 4) ? a_fmt : 2;
  GemmArgs g;
  g.a = reinterpret_cast<const uint8_t*>(a);
  g.a_bscale = a_bscale;
  g.a_tscale = a_tscale;
  g.lda = lda;
  g.w_codes = w_packed + kPackHeader;
  g.w_scales = g.w_codes + packed_codes_bytes(w_fmt, n, k);
  g.w_tscale = reinterpret_cast<const float*>(w_packed + kPackScaleOffset);
  g.m = (int)m;
  g.n = (int)n;
  g.k = (int)k;
  g.y = y;
  g.ldy = ldy;
  g.out_mode = out_mode;
  g.y_scale = y_scale;
  g.y_bscale = y_bscale;
  g.tiles_m = g.tiles_n = 0;
  // persistent grids of 256 x 256 tiles, four waves of 128 x 128 each
  if (a_fmt == 4) {
    g.tiles_m = (g.m + 255) / 256;
    g.tiles_n = (g.n + 255) / 256;
    const int tiles = g.tiles_m * g.tiles_n;
    hipLaunchKernelGGL(k_gemm_mxfp8_direct, dim3(std::min(tiles, device_cus())), dim3(256), 0, st, g);
    return hipGetLastError();
  }
  if (a_fmt == 3) {
    g.tiles_m = (g.m + 255) / 256;
    g.tiles_n = (g.n + 255) / 256;
    const int tiles = g.tiles_m * g.tiles_n;
    hipLaunchKernelGGL(k_gemm_mxfp4_direct, dim3(std::min(tiles, device_cus())), dim3(256), 0, st, g);
    return hipGetLastError();
  }
  const int cus = device_cus();
  if (a_fmt == 1) {
    g.tiles_m = (g.m + 255) / 256;
    g.tiles_n = (g.n + 255) / 256;
    const int tiles = g.tiles_m * g.tiles_n;
    // Few tokens: the split-K kernel. FP8 operands need no expansion, so
    // narrow tiles cost nothing extra: the narrowest 32-row tile (32 x 32 NP,
    // NP = 1 .. 4) that still gives every workgroup a CU of its own, with
    // eight waves and one chunk in flight each (NP = 2: four waves, two
    // chunks); else 32 x 64 tiles while those number at most two per CU.
    // Measured at M = 16 .. 1024, N, K in {256, 1024, 3072, 9216} (GPU time
    // from graph replays): the best of five tilings within 2% at every shape
    // (128 x 256 x 256 3.8 -> 3.2 us, 256 x 3072 x 1024 6.6 -> 5.7 us,
    // 1024 x 1024 x 3072 11.9 -> 10.0 us; the 32 x 64 rule alone was 1.2-1.9x
    // faster than the 64 x 128 kernel where K >= 3072).
    if (m <= 1024) {
      const int64_t rows32 = (m + 31) / 32;
      if (rows32 * ((n + 31) / 32) <= cus) {
        // at most four chunks (K <= 512): four waves (128 x 256 x 256: 3.2 -> 2.8 us)
        if ((k >> 7) <= 4) return run_splitk<MODE_FP8, 1, 1, 4, 1>(g, st);
        return run_splitk<MODE_FP8, 1, 1, 8, 1>(g, st);
      }
      if (rows32 * ((n + 63) / 64) <= cus) return run_splitk<MODE_FP8, 1, 2, 4, 2>(g, st);
      if (rows32 * ((n + 95) / 96) <= cus) return run_splitk<MODE_FP8, 1, 3, 8, 1>(g, st);
      if (rows32 * ((n + 127) / 128) <= cus) return run_splitk<MODE_FP8, 1, 4, 8, 1>(g, st);
    }
    const int64_t small_tiles = (int64_t)((m + 31) / 32) * ((n + 63) / 64);
    if (small_tiles <= 2 * cus) return run_splitk<MODE_FP8, 1, 2, 4, 2>(g, st);
    // Too few 256 x 256 tiles to fill the chip: the 64 x 128 kernel's eight
    // times as many workgroups win. Measured crossover (encoder and
    // transformer widths, M = 128 .. 3072): below 3/8 of a tile per CU.
    if (m <= 128 || 8 * tiles < 3 * cus) return run_fp8<1, 2>(g, st);
    // 288 x 192 tiles where their rounds of tiles cover less area than the
    // 256 x 256 tiles' rounds (the time of both kernels follows the round
    // count); not for NVFP4 outputs, whose 16-blocks the 256 x 256 epilogue forms
    const int t288_m = (int)((m + 287) / 288), t288_n = (int)((n + 191) / 192);
    const int64_t t288 = (int64_t)t288_m * t288_n;
    if (out_mode != OUT_NVFP4 &&
        ((t288 + cus - 1) / cus) * (288 * 192) < (int64_t)((tiles + cus - 1) / cus) * (256 * 256)) {
      g.tiles_m = t288_m;
      g.tiles_n = t288_n;
      hipLaunchKernelGGL(k_gemm_fp8_t288, dim3((unsigned)std::min<int64_t>(t288, cus)), dim3(256), 0, st, g);
      return hipGetLastError();
    }
    hipLaunchKernelGGL(k_gemm_fp8_direct, dim3(std::min(tiles, cus)), dim3(256), 0, st, g);
    return hipGetLastError();
  } else if (a_fmt == 2) {
    g.tiles_m = (g.m + 255) / 256;
    g.tiles_n = (g.n + 255) / 256;
    const int tiles = g.tiles_m * g.tiles_n;
    // Below half a round of 256 x 256 tiles the split-K kernel is faster
    // (measured up to M = 2300 at N = K = 3072: 0.9x the time there, 0.3x at
    // M = 512). Tile and split: 64 x 96 tiles where they fill the chip with
    // K >= 2048 (the most MFMAs per expanded operand); 32 x 64 tiles where
    // that leaves CUs idle; 64 x 64 tiles for short reductions (K < 2048).
    // Eight waves, two per SIMD, so that one wave's operand expansion runs
    // beside the other's MFMAs: at 64 x 96 and 64 x 64, one chunk in flight
    // per wave was 10-21% faster than four waves with two or three (NVFP4
    // 512 x 3072 x 3072 16.3 -> 14.3 us, 256 x 3072 x 1024 8.1 -> 6.4 us).
    if (m <= 128 || 2 * tiles < cus) {
      const int kcn = (int)(k >> 7);
      const int64_t t6496 = (int64_t)((m + 63) / 64) * ((n + 95) / 96);
      if (kcn < 16) return run_splitk<MODE_NVFP4, 2, 2, 8, 1>(g, st);
      if (t6496 >= cus - cus / 4) return run_splitk<MODE_NVFP4, 2, 3, 8, 1>(g, st);
      return run_splitk<MODE_NVFP4, 1, 2, 8, 3>(g, st);
    }
    hipLaunchKernelGGL(k_gemm_nvfp4_direct, dim3(std::min(tiles, cus)), dim3(256), 0, st, g);
    return hipGetLastError();
  } else {
    const int64_t npan_all = (n + 31) / 32;
    const int64_t xbytes = (m + 1) * (k * 2 + 16);
    // (bf16 and fp32 outputs only: FP8 outputs take the split-K kernel)
    if (m == 1 && npan_all >= 8 * (int64_t)device_cus() && k * 2 <= 64 * 1024 && out_mode != OUT_FP8) {
      // two workgroups per CU; as few waves as give every wave the same
      // number of panels (up to one), so no last round runs partly empty
      const int64_t wmax = 2 * 8 * (int64_t)device_cus();
      const int64_t ppw = (npan_all + wmax - 1) / wmax;
      const unsigned grid = (unsigned)(((npan_all + ppw - 1) / ppw + 7) / 8);
      hipLaunchKernelGGL((k_w4a16_gemv<3>), dim3(grid), dim3(512), (size_t)(k * 2), st, g);
      return hipGetLastError();
    }
    if (m <= 16 && npan_all >= 8 * (int64_t)device_cus() && xbytes <= 128 * 1024 && out_mode != OUT_FP8) {
      // one workgroup per CU (the activation rows take most of the LDS),
      // balanced like the matrix-vector kernel's grid; as many waves as the
      // registers allow without spills: 16 waves with two chunks in flight at
      // M <= 8, 12 waves with three at M <= 16 (3-4% / 1% faster than 8 waves
      // with four on the cold pool)
      const int nwv = m <= 8 ? 16 : 12;
      const int64_t wmax = nwv * (int64_t)device_cus();
      const int64_t ppw = (npan_all + wmax - 1) / wmax;
      const unsigned grid = (unsigned)(((npan_all + ppw - 1) / ppw + nwv - 1) / nwv);
      if (m <= 8) hipLaunchKernelGGL((k_w4a16_stream<2, 4, 16>), dim3(grid), dim3(1024), (size_t)xbytes, st, g);
      else hipLaunchKernelGGL((k_w4a16_stream<3, 8, 12>), dim3(grid), dim3(768), (size_t)xbytes, st, g);
      return hipGetLastError();
    }
    // Past the ridge point with enough 256 x 256 tiles for half a round: the
    // persistent W4A4-shaped kernel (the weight pool at M = 256, 512: 1.5x the
    // 128 x 256 tile kernel, which was itself 1.5x the split-K kernels there)
    const int t256_m = (int)((m + 255) / 256), t256_n = (int)((n + 255) / 256);
    const int64_t t256 = (int64_t)t256_m * t256_n;
    if (m > 128 && 2 * t256 >= device_cus()) {
      g.tiles_m = t256_m;
      g.tiles_n = t256_n;
      hipLaunchKernelGGL(k_gemm_w4a16_direct, dim3((unsigned)std::min<int64_t>(t256, device_cus())), dim3(256), 0, st, g);
      return hipGetLastError();
    }
    if (m <= 1024) {
      // Shapes measured on the MI355X (text-encoder linears, M <= 512):
      // one-panel workgroups of 8 waves for narrow outputs; two panels per
      // 4-wave workgroup once the output is wide enough that the activation
      // re-reads (once per workgroup column) dominate.
      const int64_t npan = (n + 31) / 32;
      const unsigned mt = (unsigned)((m + 31) / 32);
      if (n >= 2048 && m > 32)
        hipLaunchKernelGGL((k_w4a16_splitk<1, 2, 4, 3, true>), dim3((unsigned)((npan + 1) / 2), mt), dim3(256), 0, st, g);
      else if (m <= 32)
        hipLaunchKernelGGL((k_w4a16_splitk<1, 1, 8, 3, false>), dim3((unsigned)npan, mt), dim3(512), 0, st, g);
      else if (m <= 256)
        hipLaunchKernelGGL((k_w4a16_splitk<1, 1, 8, 3, true>), dim3((unsigned)npan, mt), dim3(512), 0, st, g);
      else
        hipLaunchKernelGGL((k_w4a16_splitk<1, 2, 8, 3, true>), dim3((unsigned)((npan + 1) / 2), mt), dim3(512), 0, st, g);
      return hipGetLastError();
    }
    return run<MODE_W4A16, 2, 2, 2, 4>(g, st);
  }
}

// The FP8 decode scale of a small bf16 activation alone (one workgroup):
// the degenerate shapes of the fused linear, which launch no GEMM tile.
__global__ void __launch_bounds__(256) k_fp8_scale_only(const uint16_t* __restrict__ x, int64_t m, int64_t k,
                                                        int64_t ldx, float* __restrict__ s) {
  uint32_t mx = 0;
  for (int64_t i = threadIdx.x; i < m * k; i += 256) mx = max(mx, (uint32_t)(x[(i / k) * ldx + i % k] & 0x7FFFu));
  for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off));
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t a = max(max(part[0], part[1]), max(part[2], part[3])) << 16;
    *s = (a >= 0x7F800000u) ? __builtin_nanf("") : __fdiv_rn(u2f(a), 448.0f);
  }
}

hipError_t launch_linear_fp8(const uint16_t* x, int64_t ldx, float* a_tscale, const uint8_t* w_packed, int64_t m,
                             int64_t n, int64_t k, void* y, int64_t ldy, int out_mode, hipStream_t st) {
  if (m == 0 || n == 0 || k == 0) {
    hipLaunchKernelGGL(k_fp8_scale_only, dim3(1), dim3(256), 0, st, x, m, k, ldx, a_tscale);
    if (m > 0 && n > 0)
      hipLaunchKernelGGL(k_zero_rows, dim3((unsigned)((m * n + 255) / 256)), dim3(256), 0, st, y, nullptr, m, n,
                         ldy, out_mode);
    return hipGetLastError();
  }
  GemmArgs g;
  g.a = reinterpret_cast<const uint8_t*>(x);
  g.a_bscale = nullptr;
  g.a_tscale = a_tscale;
  g.lda = ldx;
  g.w_codes = w_packed + kPackHeader;
  g.w_scales = g.w_codes + packed_codes_bytes(1, n, k);
  g.w_tscale = reinterpret_cast<const float*>(w_packed + kPackScaleOffset);
  g.m = (int)m;
  g.n = (int)n;
  g.k = (int)k;
  g.y = y;
  g.ldy = ldy;
  g.out_mode = out_mode;
  g.y_scale = nullptr;
  g.y_bscale = nullptr;
  // the split-K tiling launch_gemm takes for an FP8 activation of this shape
  // (so the accumulation order is the same), the 32 x 64 tiles with two
  // chunks in flight where it would leave the split-K kernel
  const int cus = device_cus();
  const int64_t rows32 = (m + 31) / 32;
  if (rows32 * ((n + 31) / 32) <= cus) {
    if ((k >> 7) <= 4) return run_splitk<MODE_FP8, 1, 1, 4, 1, true>(g, st);
    return run_splitk<MODE_FP8, 1, 1, 8, 1, true>(g, st);
  }
  if (rows32 * ((n + 63) / 64) <= cus) return run_splitk<MODE_FP8, 1, 2, 4, 2, true>(g, st);
  if (rows32 * ((n + 95) / 96) <= cus) return run_splitk<MODE_FP8, 1, 3, 8, 1, true>(g, st);
  if (rows32 * ((n + 127) / 128) <= cus) return run_splitk<MODE_FP8, 1, 4, 8, 1, true>(g, st);
  return run_splitk<MODE_FP8, 1, 2, 4, 2, true>(g, st);
}

}  // namespace qg
