// mpfa_device.h -- gfx950 device helpers for the QK4PV8 kernels: number-format
// codecs written from the format definitions, exact NVFP4 dequantization into
// FP16 MFMA operands, and thin wrappers over the CDNA4 matrix instructions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpfa {

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;        // head dimension
constexpr int kPage = 64;      // tokens per cache page
constexpr int kTile = 128;     // keys per KV tile
constexpr float kLog2_448 = 8.807354922057604f;   // log2(448): P carries the fixed FP8 scale

// ---------------------------------------------------------------------------
// Number formats (Sec. 2.1 Eq. 1; Sec. 4.1)
// ---------------------------------------------------------------------------

// FP32 -> OCP E4M3 (bias 7, max 448), round to nearest even, saturating at 448,
// sign kept.  Subnormal range (< 2^-6) is a fixed grid of 2^-9; above it the
// 23-bit mantissa is rounded to 3 bits by the add-and-truncate rule with the
// carry flowing into the exponent.
__device__ __forceinline__ uint32_t e4m3_rne_sat(float x) {
  uint32_t u = __float_as_uint(x);
  uint32_t sign = (u >> 24) & 0x80u;
  float a = __builtin_fabsf(x);
  uint32_t code;
  if (!(a < 448.0f)) {
    code = 0x7Eu;
  } else if (a < 0.015625f) {
    code = (uint32_t)__builtin_rintf(a * 512.0f);
  } else {
    uint32_t ua = __float_as_uint(a);
    uint32_t r = ua + 0x7FFFFu + ((ua >> 20) & 1u);
    code = (r >> 20) - (120u << 3);
  }
  return sign | code;
}

// FP32 -> E2M1 (magnitudes 0, .5, 1, 1.5, 2, 3, 4, 6), round to nearest with
// ties to the even code, saturating at 6, sign kept in bit 3.  The code is the
// number of decision thresholds the magnitude passes; a tie sits on a
// threshold and goes to the even side ('>' vs '>=').
__device__ __forceinline__ uint32_t e2m1_rne_sat(float y) {
  float a = __builtin_fabsf(y);
  uint32_t c = (uint32_t)(a > 0.25f) + (uint32_t)(a >= 0.75f) + (uint32_t)(a > 1.25f) +
               (uint32_t)(a >= 1.75f) + (uint32_t)(a > 2.5f) + (uint32_t)(a >= 3.5f) +
               (uint32_t)(a > 5.0f);
  return c | ((__float_as_uint(y) >> 28) & 8u);
}

// E4M3 code -> value (exact in FP32).
__device__ __forceinline__ float e4m3_value(uint32_t c) {
  uint32_t e = (c >> 3) & 15u, m = c & 7u;
  float v = e ? __builtin_ldexpf(1.0f + (float)m * 0.125f, (int)e - 7) : (float)m * (1.0f / 512.0f);
  return (c & 0x80u) ? -v : v;
}

// FP32 -> BF16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint16_t bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// floor(log2 |x|) for finite nonzero x (v_frexp_exp returns it plus one).
__device__ __forceinline__ int ilog2f(float x) { return __builtin_amdgcn_frexp_expf(x) - 1; }

// Second-level NVFP4 scale: smallest 2^k, k in [-63, 63], with 2688 * 2^k >= amax
// (so the largest group scale amax / (6 t) is at most 448); 1 when amax == 0.
// The range keeps tQ * tK and its inverse normal FP32 numbers (2^-126 .. 2^126),
// which the attention kernels fold into lambda and the compensation scale.
__device__ __forceinline__ float tensor_scale(float amax) {
  if (!(amax > 0.0f)) return 1.0f;
  int e = ilog2f(amax);                    // amax in [2^e, 2^(e+1))
  int k = e - 12;
  while (k < 63 && __builtin_ldexpf(2688.0f, k) < amax) ++k;
  while (k > -63 && __builtin_ldexpf(2688.0f, k - 1) >= amax) --k;
  if (k < -63) k = -63;
  if (k > 63) k = 63;
  return __builtin_ldexpf(1.0f, k);
}

// Element conversions through the gfx950 converters.  Over every finite FP32
// input these give the same bytes as e2m1_rne_sat / e4m3_rne_sat (checked
// exhaustively on the device): v_cvt_scalef32_pk_fp4_f32 rounds to nearest
// even and saturates at 6 after dividing by the power of two in its scale
// operand; v_cvt_pk_fp8_f32 rounds to nearest even, and clamping to +-448
// first makes it saturate as the E4M3 encoder does.
__device__ __forceinline__ uint32_t fp4_pair(uint32_t w, float a, float b, float pow2, int sel) {
  switch (sel) {   // the byte selector must be an immediate
    case 0: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, a, b, pow2, 0);
    case 1: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, a, b, pow2, 1);
    case 2: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, a, b, pow2, 2);
    default: return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, a, b, pow2, 3);
  }
}
__device__ __forceinline__ uint32_t fp8_sat_pair(uint32_t w, float a, float b, bool hi) {
  a = fminf(fmaxf(a, -448.0f), 448.0f);
  b = fminf(fmaxf(b, -448.0f), 448.0f);
  return hi ? (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)w, true)
            : (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)w, false);
}

// RN(x / s) from r = RN(1 / s): one product and one residual correction.  For
// divisors s = 2^k * (E4M3 value) this equals the correctly rounded quotient
// for every FP32 x whose quotient is at least 2^-100 in magnitude (checked
// exhaustively on the device over all x and all 126 positive E4M3 values);
// smaller quotients round to the zero E2M1 code either way.  The sign is
// restored for x = -0 (the correction would return +0).
__device__ __forceinline__ float div_by_scale(float x, float s, float r) {
  const float q0 = x * r;
  const float e = __builtin_fmaf(-s, q0, x);
  return __builtin_copysignf(__builtin_fmaf(e, r, q0), x);
}

constexpr float kRcp6 = 0x1.555556p-3f;   // RN(1/6)

// ---------------------------------------------------------------------------
// Exact NVFP4 -> FP16 dequantization.
// An E4M3 scale s = 2^E * M splits into a power of two (E in [-6, 8]) and a
// mantissa M = 1 + m/8 (normal) or m/8 (subnormal).  v_cvt_scalef32_pk_f16_fp4
// applies only the exponent of its scale operand, giving q * 2^E exactly; one
// packed FP16 multiply by M then yields s * q exactly (at most 6 significant
// bits, magnitude in [2^-10, 2688]: always an FP16 normal number).
// ---------------------------------------------------------------------------
struct ScaleSplit {
  float pow2;     // 2^E
  f16x2 mant;     // (M, M)
};

__device__ __forceinline__ ScaleSplit split_e4m3(uint32_t code) {
  const uint32_t e = (code >> 3) & 15u, m = code & 7u;
  ScaleSplit s;
  // subnormal codes (e == 0) share the exponent of e == 1 without the implicit 1
  s.pow2 = __uint_as_float((uint32_t)(max(e, 1u) + 120u) << 23);   // 2^(max(e,1) - 7)
  const _Float16 mm = (_Float16)((float)((e ? 8u : 0u) + m) * 0.125f);
  s.mant = (f16x2){mm, mm};
  return s;
}

// Eight E2M1 codes (one dword, channel order low nibble first) -> eight FP16.
__device__ __forceinline__ f16x8 dequant8(uint32_t codes, ScaleSplit s) {
  f16x2 a = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, s.pow2, 0) * s.mant;
  f16x2 b = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, s.pow2, 1) * s.mant;
  f16x2 c = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, s.pow2, 2) * s.mant;
  f16x2 d = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, s.pow2, 3) * s.mant;
  return (f16x8){a[0], a[1], b[0], b[1], c[0], c[1], d[0], d[1]};
}

// ---------------------------------------------------------------------------
// Matrix instructions (16x16 output tiles, 64-lane wavefront).
// Operand layout (verified on gfx950): lane l supplies row (A) / column (B)
// l % 16 and a contiguous slice of the reduction dimension selected by l / 16;
// the accumulator lane l holds rows 4*(l/16) .. 4*(l/16)+3 of column l % 16.
// ---------------------------------------------------------------------------
__device__ __forceinline__ f32x4 mfma_f16(f16x8 a, f16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_bf16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// FP8 E4M3 x FP8 E4M3, K = 128, unit block scales (E8M0 127 = 2^0).
__device__ __forceinline__ f32x4 mfma_fp8(i32x8 a, i32x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, 0, 0, 0, 0x7F7F7F7F, 0, 0x7F7F7F7F);
}

// Scaled FP4 MFMA (MXFP4): A and B hold 32 E2M1 values per lane (16 bytes in
// the low four registers, element 2j in the low nibble of byte j), each lane
// with its own E8M0 scale byte for its 32-element block.
__device__ __forceinline__ f32x4 mfma_fp4(u32x4 a, u32x4 b, f32x4 c, int scale_a, int scale_b) {
  const i32x8 av = {(int)a[0], (int)a[1], (int)a[2], (int)a[3], 0, 0, 0, 0};
  const i32x8 bv = {(int)b[0], (int)b[1], (int)b[2], (int)b[3], 0, 0, 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(av, bv, c, 4, 4, 0, scale_a, 0, scale_b);
}

// Four FP32 values in [0, 448] -> four E4M3 bytes (hardware RNE).
__device__ __forceinline__ uint32_t pack_fp8x4(float a, float b, float c, float d) {
  // both halves of the word are written, so its previous contents do not
  // matter: passing a's bits lets the result take a's register
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, __float_as_int(a), false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return (uint32_t)w;
}

// Maximum over the four lanes l, l^16, l^32, l^48 (the four 16-lane rows).
// v_permlane16_swap exchanges the odd rows of its first operand with the even
// rows of its second; with both operands x the two results hold, in every
// lane, the values of rows {2r, 2r+1}.  v_permlane32_swap does the same for
// the two halves of the wave.  Both are plain vector instructions (no LDS
// round trip as a shuffle through ds_bpermute would take).
__device__ __forceinline__ float wave_max16(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ float wave_sum16(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

}  // namespace mpfa
