// gemm.hip -- quantized linear layers on gfx950 matrix cores.
//
// Y[m, n] = s_a * s_w * sum_k deq'(A)[m, k] * deq'(W)[n, k], the low-bit
// linears of the paper's denoising transformer (Sec. 4, quantization
// paragraph; Table 2) and of its small text encoder (weight-only).
//
// One kernel template, three operand modes, all on 32x32 MFMAs:
//   W8A8  (FP8 x FP8)    : codes go straight into v_mfma_f32_32x32x64_f8f6f4
//                          (OCP E4M3 operands); tensor scales in the epilogue.
//   W4A4  (NVFP4 x NVFP4): the E4M3 block scale changes every 16 reduction
//                          elements and is not a power of two, so it cannot
//                          ride in the hardware's per-32 power-of-two operand
//                          scale. An E2M1 code times its E4M3 block scale is
//                          exact in fp16 (<= 6 significant bits, magnitudes in
//                          [2^-10, 2688]), so both operands are expanded to
//                          fp16 in registers (v_cvt_scalef32_pk_f16_fp4 then
//                          v_pk_mul_f16) and fed to v_mfma_f32_32x32x16_f16.
//   W4A16 (bf16 x NVFP4) : the weight is expanded the same way to bf16
//                          (exact) for v_mfma_f32_32x32x16_bf16.
//
// Reduction order. Both operands of a 32x32 MFMA are read in the same
// permuted reduction order: within a 128-wide chunk, lane l (row l % 32,
// half g = l / 32) feeds the elements [64 g, 64 g + 64) of its row over the
// chunk's MFMA steps, so each lane's operand bytes are one contiguous run
// (the order of the sum changes, its terms do not).
//
// Tiling: a workgroup of WM x WN wavefronts owns a (32 TM WM) x (32 TN WN)
// output tile; each wave owns TM x TN tiles of 32 x 32. Chunks of 128 are
// staged in LDS in the packed weight's lane-major order, so every LDS read
// is one contiguous 1 KiB wave access. Global loads run two chunks ahead in
// two register sets; LDS is double buffered with one barrier per chunk.
//
// MFMA orientation: the weight panel is the MFMA A operand and the
// activation panel the B operand, so a lane ends with runs of 4 consecutive
// output columns of one output row (8-byte bf16 stores).
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
  int f32out;
  int tiles_m, tiles_n;
};

// LDS bytes per 32-row panel per 128-chunk: codes/values of A (activations)
// and B (weights), and expanded block scales of A and B.
template <int MODE> struct Lds;
template <> struct Lds<MODE_FP8> { static constexpr int A = 4096, B = 4096, AS = 0, BS = 0; };
template <> struct Lds<MODE_NVFP4> { static constexpr int A = 2048, B = 2048, AS = 512, BS = 512; };
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
// of the fp32 product is already the bf16 value).
__device__ inline v4i dequant8_bf16(uint32_t w, float sc) {
  v4i o;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    float f0, f1;
    switch (b) {
      case 0: { auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 0); f0 = t[0]; f1 = t[1]; break; }
      case 1: { auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 1); f0 = t[0]; f1 = t[1]; break; }
      case 2: { auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 2); f0 = t[0]; f1 = t[1]; break; }
      default: { auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 3); f0 = t[0]; f1 = t[1]; break; }
    }
    o[b] = (int)((f2u(f0 * sc) >> 16) | (f2u(f1 * sc) & 0xFFFF0000u));
  }
  return o;
}

// 8 E4M3 block scales (two dwords, block j in byte j) -> 8 fp16 (exact).
__device__ inline uint4 e4m3x8_to_f16(uint2 w) {
  uint32_t h[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t d = (j < 2) ? w.x : w.y;
    const uint32_t c0 = (d >> (16 * (j & 1))) & 0xFFu, c1 = (d >> (16 * (j & 1) + 8)) & 0xFFu;
    h[j] = (uint32_t)__builtin_bit_cast(uint16_t, e4m3_to_f16(c0)) |
           ((uint32_t)__builtin_bit_cast(uint16_t, e4m3_to_f16(c1)) << 16);
  }
  return make_uint4(h[0], h[1], h[2], h[3]);
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
  constexpr int NT = 64 * WM * WN;
  constexpr int PA = TM * WM, PB = TN * WN;  // 32-row panels per tile
  constexpr int BM = 32 * PA, BN = 32 * PB;
  constexpr int A_BYTES = PA * Lds<MODE>::A, B_BYTES = PB * Lds<MODE>::B;
  constexpr int AS_BYTES = PA * Lds<MODE>::AS, BS_BYTES = PB * Lds<MODE>::BS;
  constexpr int STAGE = A_BYTES + B_BYTES + AS_BYTES + BS_BYTES;
  // 16-byte pieces per stage of each operand; one 8-byte scale run per row
  constexpr int NPA = A_BYTES / 16, NPB = B_BYTES / 16;
  static_assert(NPA % NT == 0 && NPB % NT == 0, "piece count must divide the thread count");
  constexpr int RA = NPA / NT, RB = NPB / NT;
  constexpr int NSA = (MODE == MODE_NVFP4) ? BM : 0;
  constexpr int NSB = (MODE == MODE_FP8) ? 0 : BN;
  constexpr int RSA = (NSA + NT - 1) / NT, RSB = (NSB + NT - 1) / NT;
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
  const int64_t a_row_bytes = (MODE == MODE_FP8) ? g.lda : (MODE == MODE_NVFP4) ? (int64_t)(g.k >> 1) : 2 * g.lda;
  const __amdgpu_buffer_rsrc_t rs_a = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a), 0, (int)((int64_t)g.m * a_row_bytes), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_b = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_codes), 0, (int)((int64_t)npanels_w * kcn * Lds<MODE>::B), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_sa = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.a_bscale), 0, (MODE == MODE_NVFP4) ? (int)((int64_t)g.m * (g.k >> 4)) : 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t rs_sb = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(g.w_scales), 0, (MODE == MODE_FP8) ? 0 : (int)((int64_t)npanels_w * kcn * 256), 0x00020000);

  // Activation pieces are read row-contiguously (CPR 16-byte pieces cover a
  // row's chunk bytes, so 64 lanes read 64 / CPR whole row runs) and written
  // to the lane-major LDS image through an XOR swizzle: piece c of row r
  // belongs to lane (r, g = c / HALF) as its piece h = c % HALF and lands in
  // slot ((r + 32 g) ^ c) of LDS block h. The lanes of one row then hit
  // distinct LDS banks, and the operand read of lane l (slot l ^ (h + HALF g))
  // stays a conflict-free 1 KiB access.
  constexpr int CPR = (MODE == MODE_FP8) ? 8 : (MODE == MODE_NVFP4) ? 4 : 16;
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
  uint32_t osa[RSA > 0 ? RSA : 1];
#pragma unroll
  for (int it = 0; it < RSA; ++it) {
    const int q = it * NT + tid;
    const uint32_t row = (uint32_t)(m0 + q);
    osa[it] = (q < NSA && row < (uint32_t)g.m) ? row * (uint32_t)(g.k >> 4) : 0x80000000u;
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
    v2i sa[RSA > 0 ? RSA : 1];
    v2i sb[RSB > 0 ? RSB : 1];
  };

  // ---- global -> registers for chunk kc
  auto load_chunk = [&](Regs& R, int kc) {
    const int sa_off = (MODE == MODE_FP8) ? kc * 128 : (MODE == MODE_NVFP4) ? kc * 64 : kc * 256;
#pragma unroll
    for (int it = 0; it < RA; ++it) R.a[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_a, oa[it], sa_off, 0);
#pragma unroll
    for (int it = 0; it < RB; ++it) R.b[it] = __builtin_amdgcn_raw_buffer_load_b128(rs_b, ob[it], kc * Lds<MODE>::B, 0);
#pragma unroll
    for (int it = 0; it < RSA; ++it) R.sa[it] = __builtin_amdgcn_raw_buffer_load_b64(rs_sa, osa[it], kc * 8, 0);
#pragma unroll
    for (int it = 0; it < RSB; ++it) R.sb[it] = __builtin_amdgcn_raw_buffer_load_b64(rs_sb, osb[it], kc * 256, 0);
  };

  // ---- registers -> LDS stage (block scales expanded once per workgroup)
  auto store_chunk = [&](const Regs& R, uint8_t* st) {
    uint8_t* sa = st;
    uint8_t* sb = st + A_BYTES;
    uint8_t* ssa = st + A_BYTES + B_BYTES;
    uint8_t* ssb = ssa + AS_BYTES;
#pragma unroll
    for (int it = 0; it < RA; ++it) *reinterpret_cast<v4i*>(sa + la[it]) = R.a[it];
#pragma unroll
    for (int it = 0; it < RB; ++it) reinterpret_cast<v4i*>(sb)[it * NT + tid] = R.b[it];
#pragma unroll
    for (int it = 0; it < RSA; ++it) {
      const int q = it * NT + tid;
      if (q < NSA) reinterpret_cast<uint4*>(ssa)[q] = e4m3x8_to_f16(make_uint2(R.sa[it].x, R.sa[it].y));  // row q: 16 B
    }
#pragma unroll
    for (int it = 0; it < RSB; ++it) {
      const int q = it * NT + tid;
      if (q < NSB) {
        if (MODE == MODE_NVFP4) {
          reinterpret_cast<uint4*>(ssb)[q] = e4m3x8_to_f16(make_uint2(R.sb[it].x, R.sb[it].y));
        } else {
          const uint32_t w[2] = {(uint32_t)R.sb[it].x, (uint32_t)R.sb[it].y};
          float f[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) f[j] = dec_e4m3((w[j >> 2] >> (8 * (j & 3))) & 0xFFu);
          reinterpret_cast<float4*>(ssb)[2 * q] = make_float4(f[0], f[1], f[2], f[3]);
          reinterpret_cast<float4*>(ssb)[2 * q + 1] = make_float4(f[4], f[5], f[6], f[7]);
        }
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
    const uint8_t* ssa = st + A_BYTES + B_BYTES;
    const uint8_t* ssb = ssa + AS_BYTES;
    const int r = lane & 31, gq = lane >> 5;
    if (MODE == MODE_FP8) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        v8i fa[TM];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const uint8_t* p = sa + (wm * TM + i) * 4096 + s * 2048;
          const v4i lo = *reinterpret_cast<const v4i*>(p + ((lane ^ (2 * s + 4 * gq)) * 16));
          const v4i hi = *reinterpret_cast<const v4i*>(p + 1024 + ((lane ^ (2 * s + 1 + 4 * gq)) * 16));
          fa[i] = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const uint8_t* p = sb + (wn * TN + j) * 4096 + s * 2048 + lane * 16;
          const v4i lo = *reinterpret_cast<const v4i*>(p), hi = *reinterpret_cast<const v4i*>(p + 1024);
          const v8i fb = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
#pragma unroll
          for (int i = 0; i < TM; ++i)
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fb, fa[i], acc[i][j], 0, 0, 0, 0, 0, 0);
        }
      }
    } else if (MODE == MODE_NVFP4) {
      uint2 sca[TM], scb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) sca[i] = *reinterpret_cast<const uint2*>(ssa + (wm * TM + i) * 512 + r * 16 + 8 * gq);
#pragma unroll
      for (int j = 0; j < TN; ++j) scb[j] = *reinterpret_cast<const uint2*>(ssb + (wn * TN + j) * 512 + r * 16 + 8 * gq);
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {  // 16-byte half of each lane's codes: 4 MFMA steps
        uint4 ca[TM], cb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          ca[i] = *reinterpret_cast<const uint4*>(sa + (wm * TM + i) * 2048 + hh * 1024 + ((lane ^ (hh + 2 * gq)) * 16));
#pragma unroll
        for (int j = 0; j < TN; ++j) cb[j] = *reinterpret_cast<const uint4*>(sb + (wn * TN + j) * 2048 + hh * 1024 + lane * 16);
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
          const int s = 4 * hh + s4;  // blocks: scale index s / 2 of the lane's four
          v8h fa[TM];
#pragma unroll
          for (int i = 0; i < TM; ++i) {
            const uint32_t w = (s4 == 0) ? ca[i].x : (s4 == 1) ? ca[i].y : (s4 == 2) ? ca[i].z : ca[i].w;
            const uint32_t sw = hh ? sca[i].y : sca[i].x;
            fa[i] = dequant8_f16(w, __builtin_bit_cast(_Float16, (uint16_t)((s4 & 2) ? (sw >> 16) : (sw & 0xFFFFu))));
          }
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const uint32_t w = (s4 == 0) ? cb[j].x : (s4 == 1) ? cb[j].y : (s4 == 2) ? cb[j].z : cb[j].w;
            const uint32_t sw = hh ? scb[j].y : scb[j].x;
            const v8h fb = dequant8_f16(w, __builtin_bit_cast(_Float16, (uint16_t)((s4 & 2) ? (sw >> 16) : (sw & 0xFFFFu))));
#pragma unroll
            for (int i = 0; i < TM; ++i)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fb, fa[i], acc[i][j], 0, 0, 0);
          }
        }
      }
    } else {  // W4A16
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
  if (MODE != MODE_W4A16) c = c * *g.a_tscale;
  const bool vec = ((reinterpret_cast<uintptr_t>(g.y) & 15) == 0) && ((g.ldy & 3) == 0);
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
        const float v0 = acc[i][j][4 * qd] * c, v1 = acc[i][j][4 * qd + 1] * c;
        const float v2 = acc[i][j][4 * qd + 2] * c, v3 = acc[i][j][4 * qd + 3] * c;
        if (g.f32out) {
          float* o = reinterpret_cast<float*>(g.y) + (int64_t)m * g.ldy + n;
          if (vec) *reinterpret_cast<float4*>(o) = make_float4(v0, v1, v2, v3);
          else { o[0] = v0; o[1] = v1; o[2] = v2; o[3] = v3; }
        } else {
          uint16_t* o = reinterpret_cast<uint16_t*>(g.y) + (int64_t)m * g.ldy + n;
          const uint32_t w0 = f32_to_bf16(v0) | (f32_to_bf16(v1) << 16);
          const uint32_t w1 = f32_to_bf16(v2) | (f32_to_bf16(v3) << 16);
          if (vec) *reinterpret_cast<uint2*>(o) = make_uint2(w0, w1);
          else { o[0] = (uint16_t)w0; o[1] = (uint16_t)(w0 >> 16); o[2] = (uint16_t)w1; o[3] = (uint16_t)(w1 >> 16); }
        }
      }
    }
  }
}

// ---------------------------------------------------------------- W4A16, few tokens
// bf16 activations with at most 32 * MT rows against NVFP4 weights: the
// weight stream is the whole cost, so one workgroup owns one 32-row weight
// panel (32 output columns) and its NW wavefronts split the reduction
// dimension chunk by chunk, reading the packed weight straight from HBM in
// operand order (32 B of codes + 4 B of scales per lane per chunk, no LDS
// staging). Partial accumulators are summed through LDS at the end.
template <int MT, int NW>
__global__ void __launch_bounds__(64 * NW) k_w4a16_skinny(GemmArgs g) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int panel = blockIdx.x;
  const int kcn = g.k >> 7;
  const int r = lane & 31, gq = lane >> 5;
  const uint16_t* x = reinterpret_cast<const uint16_t*>(g.a);
  v16f acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[i][v] = 0.0f;
  for (int kc = wave; kc < kcn; kc += NW) {
    const int64_t chunk = (int64_t)panel * kcn + kc;
    const uint4 c0 = reinterpret_cast<const uint4*>(g.w_codes + chunk * 2048)[lane];
    const uint4 c1 = reinterpret_cast<const uint4*>(g.w_codes + chunk * 2048 + 1024)[lane];
    const uint32_t sc = *reinterpret_cast<const uint32_t*>(g.w_scales + chunk * 256 + r * 8 + 4 * gq);
    const uint32_t cw[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const v8bf wb = __builtin_bit_cast(v8bf, dequant8_bf16(cw[s], dec_e4m3((sc >> (8 * (s >> 1))) & 0xFFu)));
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const int m = 32 * i + r;
        v4i xv = {0, 0, 0, 0};
        if (m < g.m) xv = *reinterpret_cast<const v4i*>(x + (int64_t)m * g.lda + kc * 128 + 64 * gq + 8 * s);
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wb, __builtin_bit_cast(v8bf, xv), acc[i], 0, 0, 0);
      }
    }
  }
  __shared__ v16f red[NW][MT][64];
#pragma unroll
  for (int i = 0; i < MT; ++i) red[wave][i][lane] = acc[i];
  __syncthreads();
  if (wave != 0) return;
  const float c = *g.w_tscale;
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    v16f t = red[0][i][lane];
#pragma unroll
    for (int w = 1; w < NW; ++w) t += red[w][i][lane];
    const int m = 32 * i + r;
    if (m >= g.m) continue;
#pragma unroll
    for (int qd = 0; qd < 4; ++qd) {
      const int n = panel * 32 + 8 * qd + 4 * gq;
      if (n >= g.n) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float v = t[4 * qd + e] * c;
        if (g.f32out) reinterpret_cast<float*>(g.y)[(int64_t)m * g.ldy + n + e] = v;
        else reinterpret_cast<uint16_t*>(g.y)[(int64_t)m * g.ldy + n + e] = (uint16_t)f32_to_bf16(v);
      }
    }
  }
}

__global__ void k_zero_rows(void* y, int64_t m, int64_t n, int64_t ldy, int f32out) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= m * n) return;
  const int64_t r = t / n, c = t - r * n;
  if (f32out) reinterpret_cast<float*>(y)[r * ldy + c] = 0.0f;
  else reinterpret_cast<uint16_t*>(y)[r * ldy + c] = 0;
}

template <int MODE, int WM, int WN, int TM, int TN, int DEPTH = 1>
static hipError_t run(GemmArgs g, hipStream_t st) {
  constexpr int BM = 32 * TM * WM, BN = 32 * TN * WN;
  g.tiles_m = (g.m + BM - 1) / BM;
  g.tiles_n = (g.n + BN - 1) / BN;
  hipLaunchKernelGGL((k_gemm<MODE, WM, WN, TM, TN, DEPTH>), dim3(g.tiles_m * g.tiles_n), dim3(64 * WM * WN), 0, st, g);
  return hipGetLastError();
}



hipError_t launch_gemm(int a_fmt, const void* a, const uint8_t* a_bscale, const float* a_tscale,
                       int64_t lda, const uint8_t* w_packed, int64_t m, int64_t n, int64_t k,
                       void* y, int64_t ldy, bool f32out, hipStream_t st) {
  if (m == 0 || n == 0) return hipSuccess;
  if (k == 0) {
    hipLaunchKernelGGL(k_zero_rows, dim3((unsigned)((m * n + 255) / 256)), dim3(256), 0, st, y, m, n, ldy, (int)f32out);
    return hipGetLastError();
  }
  const int w_fmt = (a_fmt == 1) ? 1 : 2;
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
  g.f32out = f32out ? 1 : 0;
  g.tiles_m = g.tiles_n = 0;
  // Large tiles: 256 x 256 per workgroup, 8 wavefronts (two per SIMD, so
  // one wave's MFMAs cover the other's LDS and barrier waits), 128 x 64 each.
  if (a_fmt == 1) {
    if (m <= 128) return run<MODE_FP8, 2, 2, 1, 2>(g, st);
    return run<MODE_FP8, 2, 4, 4, 2>(g, st);
  } else if (a_fmt == 2) {
    if (m <= 128) return run<MODE_NVFP4, 2, 2, 1, 2>(g, st);
    return run<MODE_NVFP4, 2, 4, 4, 2>(g, st);
  } else {
    if (m <= 64) {
      const unsigned grid = (unsigned)((n + 31) / 32);
      if (m <= 32) hipLaunchKernelGGL((k_w4a16_skinny<1, 8>), dim3(grid), dim3(512), 0, st, g);
      else hipLaunchKernelGGL((k_w4a16_skinny<2, 8>), dim3(grid), dim3(512), 0, st, g);
      return hipGetLastError();
    }
    if (m <= 1024) return run<MODE_W4A16, 2, 2, 1, 2>(g, st);
    return run<MODE_W4A16, 2, 2, 2, 4>(g, st);
  }
}

}  // namespace qg
