// gemm.hip -- quantized linear layers on gfx950 matrix cores.
//
// Y[m, n] = s_a * s_w * sum_k deq'(A)[m, k] * deq'(W)[n, k], the low-bit
// linears of the paper's denoising transformer (Sec. 4, quantization
// paragraph; Table 2) and of its small text encoder (weight-only).
//
// One kernel template, three operand modes:
//   W8A8  (FP8 x FP8)   : codes go straight into v_mfma_f32_16x16x128_f8f6f4
//                         (OCP E4M3 operands); per-tensor scales in the epilogue.
//   W4A4  (NVFP4 x NVFP4): the E4M3 block scale changes every 16 reduction
//                         elements and is not a power of two, so it cannot
//                         ride in the hardware's per-32 power-of-two operand
//                         scale. Each E2M1 code times its E4M3 block scale is
//                         exact in fp16 (<= 6 significant bits, magnitudes in
//                         [2^-10, 2688]), so both operands are expanded to
//                         fp16 in registers (v_cvt_scalef32_pk_f16_fp4 then
//                         v_pk_mul_f16) and fed to v_mfma_f32_16x16x32_f16.
//                         The tensor scales are applied in the epilogue.
//   W4A16 (bf16 x NVFP4): the weight is expanded the same way to bf16 (exact)
//                         and the product runs on v_mfma_f32_16x16x32_bf16.
//
// Tiling: a workgroup of WM x WN wavefronts owns a (16*TM*WM) x (16*TN*WN)
// output tile; each wave owns TM x TN MFMA tiles of 16 x 16. The reduction
// runs in chunks of 128. Each chunk of both operands is staged in LDS in
// "lane-major" order -- the 16-row panel's operand exactly as the 64 lanes
// hold it -- so every LDS read is one contiguous 1 KiB wave access. Global
// loads for chunk c+1 are issued before the MFMAs of chunk c and written to
// the other LDS buffer after them (one barrier per chunk).
//
// MFMA orientation: the weight panel is the MFMA A operand and the
// activation panel the B operand, so a lane ends with 4 consecutive output
// columns of one output row (one 8-byte bf16 store per tile).
#include "common.hpp"
#include "kernels.hpp"

namespace qg {

enum { MODE_FP8 = 1, MODE_NVFP4 = 2, MODE_W4A16 = 3 };

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
  int tiles_n;
};

// LDS bytes per 16-row panel per 128-chunk, operand A (activations) and B (weights).
template <int MODE> struct Lds;
template <> struct Lds<MODE_FP8> { static constexpr int A = 2048, B = 2048, AS = 0, BS = 0; };
template <> struct Lds<MODE_NVFP4> { static constexpr int A = 1024, B = 1024, AS = 256, BS = 256; };
template <> struct Lds<MODE_W4A16> { static constexpr int A = 4096, B = 1024, AS = 0, BS = 512; };

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
    float2 f;
    switch (b) {
      case 0: { auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 0); f = make_float2(t[0], t[1]); break; }
      case 1: { auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 1); f = make_float2(t[0], t[1]); break; }
      case 2: { auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 2); f = make_float2(t[0], t[1]); break; }
      default: { auto t = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, 3); f = make_float2(t[0], t[1]); break; }
    }
    const uint32_t lo = f2u(f.x * sc), hi = f2u(f.y * sc);
    o[b] = (int)((lo >> 16) | (hi & 0xFFFF0000u));
  }
  return o;
}

template <int MODE, int WM, int WN, int TM, int TN>
__global__ void __launch_bounds__(64 * WM * WN) k_gemm(GemmArgs g) {
  constexpr int NT = 64 * WM * WN;
  constexpr int PA = TM * WM, PB = TN * WN;  // 16-row panels per tile
  constexpr int BM = 16 * PA, BN = 16 * PB;
  constexpr int A_BYTES = PA * Lds<MODE>::A, B_BYTES = PB * Lds<MODE>::B;
  constexpr int AS_BYTES = PA * Lds<MODE>::AS, BS_BYTES = PB * Lds<MODE>::BS;
  constexpr int STAGE = A_BYTES + B_BYTES + AS_BYTES + BS_BYTES;
  // 16-byte pieces per stage of each operand's codes, and 8-byte scale runs
  constexpr int NPA = A_BYTES / 16, NPB = B_BYTES / 16;
  constexpr int RA = (NPA + NT - 1) / NT, RB = (NPB + NT - 1) / NT;
  constexpr int NSA = (MODE == MODE_NVFP4) ? BM : 0;   // A scale runs (one per row)
  constexpr int NSB = (MODE == MODE_FP8) ? 0 : BN;     // B scale runs
  constexpr int RSA = (NSA + NT - 1) / NT, RSB = (NSB + NT - 1) / NT;

  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int tile = blockIdx.x;
  const int bm = tile / g.tiles_n, bn = tile - bm * g.tiles_n;
  const int m0 = bm * BM, n0 = bn * BN;
  const int kcn = g.k >> 7;
  const int npanels_w = g.n >> 4;

  uint4 ra[RA > 0 ? RA : 1], rb[RB > 0 ? RB : 1];
  uint2 rsa[RSA > 0 ? RSA : 1], rsb[RSB > 0 ? RSB : 1];

  // ---- global -> registers for chunk kc
  auto load_chunk = [&](int kc) {
#pragma unroll
    for (int it = 0; it < RA; ++it) {
      const int q = it * NT + tid;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (q < NPA) {
        if (MODE == MODE_FP8) {
          const int p = q >> 7, s = q & 127, h = s >> 6, l = s & 63;
          const int row = m0 + 16 * p + (l & 15);
          if (row < g.m)
            v = *reinterpret_cast<const uint4*>(g.a + (int64_t)row * g.lda + kc * 128 + 32 * (l >> 4) + 16 * h);
        } else if (MODE == MODE_NVFP4) {
          const int p = q >> 6, l = q & 63;
          const int row = m0 + 16 * p + (l & 15);
          if (row < g.m)
            v = *reinterpret_cast<const uint4*>(g.a + (int64_t)row * (g.k >> 1) + kc * 64 + 16 * (l >> 4));
        } else {
          const int p = q >> 8, s = q & 255, h = s >> 6, l = s & 63;
          const int row = m0 + 16 * p + (l & 15);
          if (row < g.m)
            v = *reinterpret_cast<const uint4*>(g.a + 2 * ((int64_t)row * g.lda + kc * 128 + 32 * (l >> 4) + 8 * h));
        }
      }
      ra[it] = v;
    }
#pragma unroll
    for (int it = 0; it < RB; ++it) {
      const int q = it * NT + tid;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (q < NPB) {
        constexpr int PIECES = Lds<MODE>::B / 16;  // per panel chunk
        const int p = q / PIECES, s = q - p * PIECES;
        const int panel = (n0 >> 4) + p;
        if (panel < npanels_w)
          v = reinterpret_cast<const uint4*>(g.w_codes + ((int64_t)panel * kcn + kc) * Lds<MODE>::B)[s];
      }
      rb[it] = v;
    }
#pragma unroll
    for (int it = 0; it < RSA; ++it) {
      const int q = it * NT + tid;
      uint2 v = make_uint2(0u, 0u);
      if (q < NSA) {
        const int row = m0 + q;
        if (row < g.m) v = *reinterpret_cast<const uint2*>(g.a_bscale + (int64_t)row * (g.k >> 4) + kc * 8);
      }
      rsa[it] = v;
    }
#pragma unroll
    for (int it = 0; it < RSB; ++it) {
      const int q = it * NT + tid;
      uint2 v = make_uint2(0u, 0u);
      if (q < NSB) {
        const int p = q >> 4, r = q & 15;
        const int panel = (n0 >> 4) + p;
        if (panel < npanels_w)
          v = reinterpret_cast<const uint2*>(g.w_scales + ((int64_t)panel * kcn + kc) * 128)[r];
      }
      rsb[it] = v;
    }
  };

  // ---- registers -> LDS stage (block scales expanded to fp16 / fp32 here, once per workgroup)
  auto store_chunk = [&](uint8_t* st) {
    uint8_t* sa = st;
    uint8_t* sb = st + A_BYTES;
    uint8_t* ssa = st + A_BYTES + B_BYTES;
    uint8_t* ssb = ssa + AS_BYTES;
#pragma unroll
    for (int it = 0; it < RA; ++it) {
      const int q = it * NT + tid;
      if (q < NPA) reinterpret_cast<uint4*>(sa)[q] = ra[it];
    }
#pragma unroll
    for (int it = 0; it < RB; ++it) {
      const int q = it * NT + tid;
      if (q < NPB) reinterpret_cast<uint4*>(sb)[q] = rb[it];
    }
#pragma unroll
    for (int it = 0; it < RSA; ++it) {
      const int q = it * NT + tid;
      if (q < NSA) {
        const uint32_t w[2] = {rsa[it].x, rsa[it].y};
        uint32_t h[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t c0 = (w[j >> 1] >> (16 * (j & 1))) & 0xFFu;
          const uint32_t c1 = (w[j >> 1] >> (16 * (j & 1) + 8)) & 0xFFu;
          h[j] = (uint32_t)__builtin_bit_cast(uint16_t, e4m3_to_f16(c0)) |
                 ((uint32_t)__builtin_bit_cast(uint16_t, e4m3_to_f16(c1)) << 16);
        }
        // panel q/16, row q%16: 16 bytes at panel*256 + row*16
        reinterpret_cast<uint4*>(ssa)[q] = make_uint4(h[0], h[1], h[2], h[3]);
      }
    }
#pragma unroll
    for (int it = 0; it < RSB; ++it) {
      const int q = it * NT + tid;
      if (q < NSB) {
        const uint32_t w[2] = {rsb[it].x, rsb[it].y};
        if (MODE == MODE_NVFP4) {
          uint32_t h[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const uint32_t c0 = (w[j >> 1] >> (16 * (j & 1))) & 0xFFu;
            const uint32_t c1 = (w[j >> 1] >> (16 * (j & 1) + 8)) & 0xFFu;
            h[j] = (uint32_t)__builtin_bit_cast(uint16_t, e4m3_to_f16(c0)) |
                   ((uint32_t)__builtin_bit_cast(uint16_t, e4m3_to_f16(c1)) << 16);
          }
          reinterpret_cast<uint4*>(ssb)[q] = make_uint4(h[0], h[1], h[2], h[3]);
        } else {
          float f[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) f[j] = dec_e4m3((w[j >> 2] >> (8 * (j & 3))) & 0xFFu);
          reinterpret_cast<float4*>(ssb)[2 * q] = make_float4(f[0], f[1], f[2], f[3]);
          reinterpret_cast<float4*>(ssb)[2 * q + 1] = make_float4(f[4], f[5], f[6], f[7]);
        }
      }
    }
  };

  v4f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  // ---- MFMAs over one staged chunk
  auto compute_chunk = [&](const uint8_t* st) {
    const uint8_t* sa = st;
    const uint8_t* sb = st + A_BYTES;
    const uint8_t* ssa = st + A_BYTES + B_BYTES;
    const uint8_t* ssb = ssa + AS_BYTES;
    if (MODE == MODE_FP8) {
      v8i fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const uint8_t* p = sa + (wm * TM + i) * 2048 + lane * 16;
        const v4i lo = *reinterpret_cast<const v4i*>(p), hi = *reinterpret_cast<const v4i*>(p + 1024);
        fa[i] = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const uint8_t* p = sb + (wn * TN + j) * 2048 + lane * 16;
        const v4i lo = *reinterpret_cast<const v4i*>(p), hi = *reinterpret_cast<const v4i*>(p + 1024);
        fb[j] = (v8i){lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(fb[j], fa[i], acc[i][j], 0, 0, 0, 0, 0, 0);
    } else if (MODE == MODE_NVFP4) {
      uint4 ca[TM], cb[TN];
      v2h sca[TM], scb[TN];
      const int r = lane & 15, gq = lane >> 4;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int p = wm * TM + i;
        ca[i] = *reinterpret_cast<const uint4*>(sa + p * 1024 + lane * 16);
        sca[i] = *reinterpret_cast<const v2h*>(ssa + p * 256 + r * 16 + 4 * gq);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int p = wn * TN + j;
        cb[j] = *reinterpret_cast<const uint4*>(sb + p * 1024 + lane * 16);
        scb[j] = *reinterpret_cast<const v2h*>(ssb + p * 256 + r * 16 + 4 * gq);
      }
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        v8h fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const uint32_t w = (s == 0) ? ca[i].x : (s == 1) ? ca[i].y : (s == 2) ? ca[i].z : ca[i].w;
          fa[i] = dequant8_f16(w, (s < 2) ? sca[i].x : sca[i].y);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const uint32_t w = (s == 0) ? cb[j].x : (s == 1) ? cb[j].y : (s == 2) ? cb[j].z : cb[j].w;
          fb[j] = dequant8_f16(w, (s < 2) ? scb[j].x : scb[j].y);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fb[j], fa[i], acc[i][j], 0, 0, 0);
      }
    } else {  // W4A16
      uint4 cb[TN];
      float2 scb[TN];
      const int r = lane & 15, gq = lane >> 4;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int p = wn * TN + j;
        cb[j] = *reinterpret_cast<const uint4*>(sb + p * 1024 + lane * 16);
        scb[j] = *reinterpret_cast<const float2*>(ssb + p * 512 + r * 32 + 8 * gq);
      }
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        v8bf fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          fa[i] = __builtin_bit_cast(v8bf, *reinterpret_cast<const v4i*>(sa + (wm * TM + i) * 4096 + s * 1024 + lane * 16));
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const uint32_t w = (s == 0) ? cb[j].x : (s == 1) ? cb[j].y : (s == 2) ? cb[j].z : cb[j].w;
          fb[j] = __builtin_bit_cast(v8bf, dequant8_bf16(w, (s < 2) ? scb[j].x : scb[j].y));
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
      }
    }
  };

  // ---- main loop: prefetch chunk kc+1 into registers while chunk kc is multiplied
  if (kcn > 0) {
    load_chunk(0);
    store_chunk(smem);
    __syncthreads();
    for (int kc = 0; kc < kcn; ++kc) {
      uint8_t* cur = smem + (kc & 1) * STAGE;
      uint8_t* nxt = smem + ((kc + 1) & 1) * STAGE;
      const bool more = (kc + 1 < kcn);
      if (more) load_chunk(kc + 1);
      compute_chunk(cur);
      if (more) store_chunk(nxt);
      __syncthreads();
    }
  }

  // ---- epilogue: scale, round, store. Lane holds Y[m][n .. n+3].
  float c = *g.w_tscale;
  if (MODE != MODE_W4A16) c = c * *g.a_tscale;
  const bool vec = ((reinterpret_cast<uintptr_t>(g.y) & 15) == 0) && ((g.ldy & 3) == 0);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + (wm * TM + i) * 16 + (lane & 15);
    if (m >= g.m) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + (wn * TN + j) * 16 + 4 * (lane >> 4);
      if (n >= g.n) continue;
      const float v0 = acc[i][j].x * c, v1 = acc[i][j].y * c, v2 = acc[i][j].z * c, v3 = acc[i][j].w * c;
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

__global__ void k_zero_rows(void* y, int64_t m, int64_t n, int64_t ldy, int f32out) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= m * n) return;
  const int64_t r = t / n, c = t - r * n;
  if (f32out) reinterpret_cast<float*>(y)[r * ldy + c] = 0.0f;
  else reinterpret_cast<uint16_t*>(y)[r * ldy + c] = 0;
}

template <int MODE, int WM, int WN, int TM, int TN>
static hipError_t run(GemmArgs g, hipStream_t st) {
  constexpr int BM = 16 * TM * WM, BN = 16 * TN * WN;
  const int tiles_m = (g.m + BM - 1) / BM;
  g.tiles_n = (g.n + BN - 1) / BN;
  hipLaunchKernelGGL((k_gemm<MODE, WM, WN, TM, TN>), dim3(tiles_m * g.tiles_n), dim3(64 * WM * WN), 0, st, g);
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
  g.tiles_n = 0;
  if (a_fmt == 1) {
    if (m <= 64) return run<MODE_FP8, 1, 4, 1, 2>(g, st);
    return run<MODE_FP8, 2, 2, 8, 8>(g, st);
  } else if (a_fmt == 2) {
    if (m <= 64) return run<MODE_NVFP4, 1, 4, 1, 2>(g, st);
    return run<MODE_NVFP4, 2, 2, 8, 8>(g, st);
  } else {
    if (m <= 64) return run<MODE_W4A16, 1, 4, 1, 2>(g, st);
    return run<MODE_W4A16, 2, 2, 4, 8>(g, st);
  }
}

}  // namespace qg
