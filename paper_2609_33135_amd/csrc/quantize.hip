// quantize.hip -- Algorithm 1 stage one on gfx950: sequence statistics (Eq. 7),
// centering, NVFP4 quantization of Q and K (Sec. 2.1 Eq. 1), FP8 V, and the
// Delta_S compensation vector (Eq. 9) written into the paged side cache
// (Sec. 6).  Memory-bound; every rounding follows the ABI contract exactly so
// that codes are bit-reproducible.
#include "mpfa_device.h"
#include "mpfa_internal.h"

#pragma clang fp contract(off)

namespace mpfa {

// One workgroup per (sequence, head), 16 waves.  Each wave sums one 128-token
// block at a time (lane l owns channels 2l, 2l+1; loads issued 16 tokens
// ahead), FP32 in token order; wave 0 then adds the block partials in block
// order, divides in FP32 and rounds to BF16.  A second pass takes the amax of
// the centered values for the power-of-two tensor scale.
__global__ __launch_bounds__(1024) void stats_kernel(QuantParams p) {
  constexpr int kW = 16;                     // waves per workgroup
  __shared__ float part[kW][kD];
  __shared__ float meanf[kD];
  __shared__ float red[kW];
  const int Htot = p.stats_k ? p.h_q + p.h_kv : p.h_q;
  const int b = blockIdx.x / Htot;
  const int hh = blockIdx.x % Htot;
  const bool is_k = hh >= p.h_q;
  const int h = is_k ? hh - p.h_q : hh;
  const int H = is_k ? p.h_kv : p.h_q;
  const uint32_t* x = reinterpret_cast<const uint32_t*>(is_k ? p.k : p.q);   // BF16 pairs
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int c0 = 2 * lane;
  const int64_t t0 = p.cu_seqlens[b];
  const int n = p.cu_seqlens[b + 1] - p.cu_seqlens[b];
  uint16_t* mean_out = (is_k ? p.k_mean : p.q_mean) + ((int64_t)b * H + h) * kD;
  // BF16 pair of token t (relative to the sequence) for this lane's channels
  auto row = [&](int t) { return x[((t0 + t) * H + h) * (kD / 2) + lane]; };

  if (p.compute_stats) {
    float tot0 = 0.0f, tot1 = 0.0f;
    if (p.smooth && n > 0) {
      const int nblk = (n + 127) / 128;
      for (int blk0 = 0; blk0 < nblk; blk0 += kW) {
        const int blk = blk0 + wv;
        float s0 = 0.0f, s1 = 0.0f;
        if (blk < nblk) {
          const int tb = blk * 128, te = min(n, tb + 128);
          for (int t = tb; t < te; t += 16) {
            uint32_t v[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) v[u] = (t + u < te) ? row(t + u) : 0u;
#pragma unroll
            for (int u = 0; u < 16; ++u) {
              if (t + u < te) {
                s0 += __uint_as_float(v[u] << 16);
                s1 += __uint_as_float(v[u] & 0xFFFF0000u);
              }
            }
          }
        }
        part[wv][c0] = s0;
        part[wv][c0 + 1] = s1;
        __syncthreads();
        if (wv == 0) {
          for (int j = 0; j < kW && blk0 + j < nblk; ++j) {
            tot0 += part[j][c0];
            tot1 += part[j][c0 + 1];
          }
        }
        __syncthreads();
      }
    }
    if (wv == 0) {
      uint16_t m0 = 0, m1 = 0;
      if (p.smooth && n > 0) {
        m0 = bf16_rne(__fdiv_rn(tot0, (float)n));
        m1 = bf16_rne(__fdiv_rn(tot1, (float)n));
      }
      mean_out[c0] = m0;
      mean_out[c0 + 1] = m1;
      meanf[c0] = bf16_to_f32(m0);
      meanf[c0 + 1] = bf16_to_f32(m1);
    }
  } else if (wv == 0) {
    meanf[c0] = p.smooth ? bf16_to_f32(mean_out[c0]) : 0.0f;
    meanf[c0 + 1] = p.smooth ? bf16_to_f32(mean_out[c0 + 1]) : 0.0f;
  }
  __syncthreads();

  // amax of the centered values (any order)
  float amax = 0.0f;
  const float m0 = meanf[c0], m1 = meanf[c0 + 1];
  int t = wv;
  for (; t + 3 * kW < n; t += 4 * kW) {
    uint32_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = row(t + u * kW);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      amax = fmaxf(amax, __builtin_fabsf(__uint_as_float(v[u] << 16) - m0));
      amax = fmaxf(amax, __builtin_fabsf(__uint_as_float(v[u] & 0xFFFF0000u) - m1));
    }
  }
  for (; t < n; t += kW) {
    const uint32_t v = row(t);
    amax = fmaxf(amax, __builtin_fabsf(__uint_as_float(v << 16) - m0));
    amax = fmaxf(amax, __builtin_fabsf(__uint_as_float(v & 0xFFFF0000u) - m1));
  }
  for (int off = 32; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  if (lane == 0) red[wv] = amax;
  __syncthreads();
  if (threadIdx.x == 0) {
    float a = 0.0f;
    for (int i = 0; i < kW; ++i) a = fmaxf(a, red[i]);
    const float ts = (p.tscale_unit || p.mx) ? 1.0f : tensor_scale(a);
    if (is_k) p.k_tscale[b * p.h_kv + h] = ts;
    else p.q_tscale[b * p.h_q + h] = ts;
  }
}

// NVFP4 quantization of one 16-channel group held as 16 centered FP32 values:
// returns 8 code bytes (as a 64-bit word, low nibble first) and the scale byte.
__device__ __forceinline__ uint64_t nvfp4_group(const float* xc, float t, uint32_t* scale_code) {
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) a = fmaxf(a, __builtin_fabsf(xc[i]));
  const uint32_t s = e4m3_rne_sat(__fdiv_rn(a, 6.0f * t));
  *scale_code = s;
  const float sd = e4m3_value(s);
  uint64_t w = 0;
  if (sd == 0.0f) {
#pragma unroll
    for (int i = 0; i < 16; ++i) w |= (uint64_t)((__float_as_uint(xc[i]) >> 28) & 8u) << (4 * i);
  } else {
    const float scale = t * sd;   // exact: t is a power of two
#pragma unroll
    for (int i = 0; i < 16; ++i) w |= (uint64_t)e2m1_rne_sat(__fdiv_rn(xc[i], scale)) << (4 * i);
  }
  return w;
}

// One workgroup (256 threads) per token: NVFP4 Q rows, NVFP4 K rows and FP8 V
// into the token's cache slot, then Delta_S for every query head.
// MXFP4 quantization of one 32-channel block held as 32 centered FP32 values:
// X = 2^e, e = floor(log2 amax) - 2 clamped to [-127, 127] (-127 for an
// all-zero block); codes E2M1_RNE_sat(x / X) (exact scaling by a power of two).
// Returns 16 code bytes (element 2j in the low nibble of byte j).
__device__ __forceinline__ u32x4 mxfp4_group(const float* xc, uint32_t* scale_code) {
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < 32; ++i) a = fmaxf(a, __builtin_fabsf(xc[i]));
  int e = -127;
  if (a > 0.0f) e = max(-127, min(127, ilog2f(a) - 2));
  *scale_code = (uint32_t)(e + 127);
  u32x4 w = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int i = 0; i < 32; ++i)
    w[i >> 3] |= e2m1_rne_sat(__builtin_ldexpf(xc[i], -e)) << (4 * (i & 7));
  return w;
}

__global__ __launch_bounds__(256) void quantize_kernel(QuantParams p) {
  __shared__ float kc[kMaxKvHeadsQuant][kD];
  const int64_t tok = blockIdx.x;
  // sequence of this token: binary search over cu_seqlens
  int lo = 0, hi = p.batch - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (p.cu_seqlens[mid] <= tok) lo = mid; else hi = mid - 1;
  }
  const int b = lo;
  const int64_t slot = p.slot_mapping[tok];
  const int64_t page = slot / kPage, off = slot % kPage;
  const int tid = threadIdx.x;
  const int grp_q = p.h_q / p.h_kv;

  // K groups (h_kv * 8 NVFP4 groups or h_kv * 4 MXFP4 blocks) and V
  if (p.mx) {
    for (int i = tid; i < p.h_kv * 4; i += blockDim.x) {
      const int h = i >> 2, g = i & 3;
      const uint16_t* src = p.k + (tok * p.h_kv + h) * kD + g * 32;
      const uint16_t* mean = p.k_mean + ((int64_t)b * p.h_kv + h) * kD + g * 32;
      float xc[32];
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        xc[e] = bf16_to_f32(src[e]) - (p.smooth ? bf16_to_f32(mean[e]) : 0.0f);
        kc[h][g * 32 + e] = xc[e];
      }
      uint32_t sc;
      const u32x4 w = mxfp4_group(xc, &sc);
      const int64_t row = (page * p.h_kv + h) * kPage + off;
      *reinterpret_cast<u32x4*>(p.k_codes + row * 64 + g * 16) = w;
      p.k_scales[row * 8 + g] = (uint8_t)sc;
      p.k_scales[row * 8 + 4 + g] = 0;
    }
  } else {
    for (int i = tid; i < p.h_kv * 8; i += blockDim.x) {
      const int h = i >> 3, g = i & 7;
      const uint16_t* src = p.k + (tok * p.h_kv + h) * kD + g * 16;
      const uint16_t* mean = p.k_mean + ((int64_t)b * p.h_kv + h) * kD + g * 16;
      float xc[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        xc[e] = bf16_to_f32(src[e]) - (p.smooth ? bf16_to_f32(mean[e]) : 0.0f);
        kc[h][g * 16 + e] = xc[e];
      }
      uint32_t sc;
      const uint64_t w = nvfp4_group(xc, p.k_tscale[b * p.h_kv + h], &sc);
      const int64_t row = (page * p.h_kv + h) * kPage + off;
      *reinterpret_cast<uint64_t*>(p.k_codes + row * 64 + g * 8) = w;
      p.k_scales[row * 8 + g] = (uint8_t)sc;
    }
  }
  for (int i = tid; i < p.h_kv * kD; i += blockDim.x) {
    const int h = i >> 7, c = i & 127;
    const float v = bf16_to_f32(p.v[(tok * p.h_kv + h) * kD + c]);
    p.v_codes[((page * p.h_kv + h) * kD + c) * kPage + off] = (uint8_t)e4m3_rne_sat(v);
  }
  // Q groups
  if (p.mx) {
    for (int i = tid; i < p.h_q * 4; i += blockDim.x) {
      const int h = i >> 2, g = i & 3;
      const uint16_t* src = p.q + (tok * p.h_q + h) * kD + g * 32;
      const uint16_t* mean = p.q_mean + ((int64_t)b * p.h_q + h) * kD + g * 32;
      float xc[32];
#pragma unroll
      for (int e = 0; e < 32; ++e) xc[e] = bf16_to_f32(src[e]) - (p.smooth ? bf16_to_f32(mean[e]) : 0.0f);
      uint32_t sc;
      const u32x4 w = mxfp4_group(xc, &sc);
      *reinterpret_cast<u32x4*>(p.q_codes + (tok * p.h_q + h) * 64 + g * 16) = w;
      p.q_scales[(tok * p.h_q + h) * 8 + g] = (uint8_t)sc;
      p.q_scales[(tok * p.h_q + h) * 8 + 4 + g] = 0;
    }
  } else {
    for (int i = tid; i < p.h_q * 8; i += blockDim.x) {
      const int h = i >> 3, g = i & 7;
      const uint16_t* src = p.q + (tok * p.h_q + h) * kD + g * 16;
      const uint16_t* mean = p.q_mean + ((int64_t)b * p.h_q + h) * kD + g * 16;
      float xc[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) xc[e] = bf16_to_f32(src[e]) - (p.smooth ? bf16_to_f32(mean[e]) : 0.0f);
      uint32_t sc;
      const uint64_t w = nvfp4_group(xc, p.q_tscale[b * p.h_q + h], &sc);
      *reinterpret_cast<uint64_t*>(p.q_codes + (tok * p.h_q + h) * 64 + g * 8) = w;
      p.q_scales[(tok * p.h_q + h) * 8 + g] = (uint8_t)sc;
    }
  }
  if (!p.smooth) return;
  __syncthreads();
  // Delta_S[h_q] = BF16(fma chain over channels of Qbar[h_q] * K_c[h_kv])
  for (int h = tid; h < p.h_q; h += blockDim.x) {
    const uint16_t* qm = p.q_mean + ((int64_t)b * p.h_q + h) * kD;
    const float* k = kc[h / grp_q];
    float d = 0.0f;
    for (int c = 0; c < kD; ++c) d = __builtin_fmaf(bf16_to_f32(qm[c]), k[c], d);
    p.ds[(page * p.h_q + h) * kPage + off] = bf16_rne(d);
  }
}

__global__ void convert_kernel(int fmt, const float* x, int64_t n, uint8_t* out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  out[i] = (uint8_t)(fmt == 0 ? e4m3_rne_sat(x[i]) : e2m1_rne_sat(x[i]));
}

hipError_t launch_quantize(const QuantParams& p, hipStream_t stream) {
  const int Htot = p.stats_k ? p.h_q + p.h_kv : p.h_q;
  stats_kernel<<<dim3(p.batch * Htot), dim3(1024), 0, stream>>>(p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.total_tokens > 0) {
    quantize_kernel<<<dim3(p.total_tokens), dim3(256), 0, stream>>>(p);
    e = hipGetLastError();
  }
  return e;
}

hipError_t launch_convert(int fmt, const float* x, int64_t n, uint8_t* out, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  convert_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(fmt, x, n, out);
  return hipGetLastError();
}

}  // namespace mpfa
