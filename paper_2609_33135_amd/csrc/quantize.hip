// quantize.hip -- Algorithm 1 stage one on gfx950: sequence statistics (Eq. 7),
// centering, NVFP4 quantization of Q and K (Sec. 2.1 Eq. 1), FP8 V, and the
// Delta_S compensation vector (Eq. 9) written into the paged side cache
// (Sec. 6).  Memory-bound; every rounding follows the ABI contract exactly so
// that codes are bit-reproducible.
#include "mpfa_device.h"
#include "mpfa_internal.h"

#pragma clang fp contract(off)

namespace mpfa {

// One workgroup per (sequence, head).  1024 threads = 8 token blocks in flight
// x 128 channels.  Means: FP32 sum inside each 128-token block in token order,
// then the block partials in block order (thread group 0 adds them), FP32
// division, BF16 rounding.  Then the amax of the centered values gives the
// power-of-two tensor scale.
__global__ __launch_bounds__(1024) void stats_kernel(QuantParams p) {
  __shared__ float part[8][kD];
  __shared__ float meanf[kD];
  __shared__ float red[32];
  const int Htot = p.stats_k ? p.h_q + p.h_kv : p.h_q;
  const int b = blockIdx.x / Htot;
  const int hh = blockIdx.x % Htot;
  const bool is_k = hh >= p.h_q;
  const int h = is_k ? hh - p.h_q : hh;
  const int H = is_k ? p.h_kv : p.h_q;
  const uint16_t* x = is_k ? p.k : p.q;
  const int c = threadIdx.x & 127, slot = threadIdx.x >> 7;
  const int64_t t0 = p.cu_seqlens[b];
  const int n = p.cu_seqlens[b + 1] - p.cu_seqlens[b];
  uint16_t* mean_out = (is_k ? p.k_mean : p.q_mean) + ((int64_t)b * H + h) * kD;

  if (p.compute_stats) {
    float total = 0.0f;
    if (p.smooth && n > 0) {
      const int nblk = (n + 127) / 128;
      for (int blk0 = 0; blk0 < nblk; blk0 += 8) {
        const int blk = blk0 + slot;
        float s = 0.0f;
        if (blk < nblk) {
          const int e = min(n, blk * 128 + 128);
          for (int t = blk * 128; t < e; ++t)
            s += bf16_to_f32(x[((t0 + t) * H + h) * kD + c]);
        }
        part[slot][c] = s;
        __syncthreads();
        if (slot == 0)
          for (int j = 0; j < 8 && blk0 + j < nblk; ++j) total += part[j][c];
        __syncthreads();
      }
    }
    if (slot == 0) {
      uint16_t mb = 0;
      if (p.smooth && n > 0) mb = bf16_rne(__fdiv_rn(total, (float)n));
      mean_out[c] = mb;
      meanf[c] = bf16_to_f32(mb);
    }
  } else if (slot == 0) {
    meanf[c] = p.smooth ? bf16_to_f32(mean_out[c]) : 0.0f;
  }
  __syncthreads();

  // amax of the centered values
  float amax = 0.0f;
  const float mc = meanf[c];
  for (int t = slot; t < n; t += 8) {
    float xc = bf16_to_f32(x[((t0 + t) * H + h) * kD + c]) - mc;
    amax = fmaxf(amax, __builtin_fabsf(xc));
  }
  for (int off = 32; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
  __syncthreads();
  if (threadIdx.x == 0) {
    float a = 0.0f;
    for (int i = 0; i < 16; ++i) a = fmaxf(a, red[i]);
    float t = p.tscale_unit ? 1.0f : tensor_scale(a);
    if (is_k) p.k_tscale[b * p.h_kv + h] = t;
    else p.q_tscale[b * p.h_q + h] = t;
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

  // K groups (h_kv * 8 of them) and V
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
  for (int i = tid; i < p.h_kv * kD; i += blockDim.x) {
    const int h = i >> 7, c = i & 127;
    const float v = bf16_to_f32(p.v[(tok * p.h_kv + h) * kD + c]);
    p.v_codes[((page * p.h_kv + h) * kD + c) * kPage + off] = (uint8_t)e4m3_rne_sat(v);
  }
  // Q groups
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
