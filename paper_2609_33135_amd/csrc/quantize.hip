// quantize.hip -- Algorithm 1 stage one on gfx950: sequence statistics (Eq. 7),
// centering, NVFP4 quantization of Q and K (Sec. 2.1 Eq. 1), FP8 V, and the
// Delta_S compensation vector (Eq. 9) written into the paged side cache
// (Sec. 6).  Memory-bound; every rounding follows the ABI contract exactly so
// that codes are bit-reproducible.
#include "mpfa_device.h"
#include "mpfa_internal.h"

#pragma clang fp contract(off)

namespace mpfa {

// ---------------------------------------------------------------------------
// Sequence statistics (Eq. 7) and tensor scales.
//
// stats_partial_kernel: one workgroup per (sequence, 128-token block).  Lane
// groups of 16 own one head row (8 channels per lane, 16-byte loads); each lane
// sums its channels over the block's tokens in token order (FP32) and keeps
// their max and min.  The amax of the centered values needs no second read:
// x -> fl(x - mean) is monotone, so max_t |fl(x_t - mean)| is reached at the
// channel's max or min.  A one-block sequence is finished in place; otherwise
// the block partials (sum, max, min) are parked in the q_codes rows of the
// sequence, which quantize_kernel overwrites later on the same stream.
// stats_final_kernel adds the block partials in block order and finishes.
// ---------------------------------------------------------------------------
constexpr int kStatUnits = 4;   // (head, 8-channel) units per thread and pass

struct StatsShape {
  int hs;                 // heads with statistics: h_q, plus h_kv with stats_k
  bool want_sum, want_amax;
};

__device__ __forceinline__ StatsShape stats_shape(const QuantParams& p) {
  StatsShape s;
  s.hs = p.h_q + (p.stats_k ? p.h_kv : 0);
  s.want_sum = p.compute_stats && p.smooth;
  s.want_amax = !(p.tscale_unit || p.mx);
  return s;
}

// block partials of block blk: float [3][hs][128] (sum, max, min).  Block i <
// nblk-1 uses the q_codes rows of its own 128 tokens; the last block uses the
// rows of block nblk-2 after that block's partials (2 * 1536 * hs bytes fit in
// the 8192 * h_q bytes of 128 token rows since hs <= 2 h_q).
__device__ __forceinline__ float* partial_ptr(const QuantParams& p, int64_t t0, int nblk, int blk, int hs) {
  const bool last = blk == nblk - 1;
  const int64_t r = last ? nblk - 2 : blk;
  uint8_t* base = p.q_codes + (t0 + r * 128) * (int64_t)p.h_q * 64;
  if (last) base += (int64_t)3 * hs * kD * 4;
  return reinterpret_cast<float*>(base);
}

// the per-head arrival counters (uint32 [hs]) and slice amaxes (float [hs][4])
__device__ __forceinline__ uint8_t* fin_scratch(const QuantParams& p, int64_t t0, int hs) {
  return p.q_codes + t0 * (int64_t)p.h_q * 64 + (int64_t)6 * hs * kD * 4;
}

// mean of head hh (0..h_q-1: Q, then K) and its BF16 output row
__device__ __forceinline__ uint16_t* mean_row(const QuantParams& p, int b, int hh) {
  return hh < p.h_q ? p.q_mean + ((int64_t)b * p.h_q + hh) * kD
                    : p.k_mean + ((int64_t)b * p.h_kv + (hh - p.h_q)) * kD;
}

__device__ __forceinline__ void write_tscale(const QuantParams& p, int b, int hh, float amax) {
  const float ts = (p.tscale_unit || p.mx) ? 1.0f : tensor_scale(amax);
  if (hh < p.h_q) p.q_tscale[b * p.h_q + hh] = ts;
  else p.k_tscale[b * p.h_kv + (hh - p.h_q)] = ts;
}

__global__ __launch_bounds__(256) void stats_partial_kernel(QuantParams p) {
  const int b = blockIdx.y, blk = blockIdx.x;
  const int64_t t0 = p.cu_seqlens[b];
  const int n = p.cu_seqlens[b + 1] - (int)t0;
  const int nblk = (n + 127) >> 7;
  if (blk >= nblk) return;
  const StatsShape ss = stats_shape(p);
  const int tb = blk * 128, te = min(n, tb + 128);
  const int nunits = ss.hs * 16;
  if (nblk >= 2 && blk == 0)   // arrival counters of stats_final_kernel
    for (int i = threadIdx.x; i < ss.hs; i += blockDim.x) reinterpret_cast<uint32_t*>(fin_scratch(p, t0, ss.hs))[i] = 0u;
  for (int u0 = 0; u0 < nunits; u0 += 256 * kStatUnits) {
    const uint4* src[kStatUnits];
    int64_t stride[kStatUnits];   // in 16-byte words per token
    bool act[kStatUnits];
    float sm[kStatUnits][8], mx[kStatUnits][8], mn[kStatUnits][8];
#pragma unroll
    for (int k = 0; k < kStatUnits; ++k) {
      const int u = u0 + k * 256 + threadIdx.x;
      act[k] = u < nunits;
      const int hh = act[k] ? u >> 4 : 0, oct = u & 15;
      const bool isq = hh < p.h_q;
      const int H = isq ? p.h_q : p.h_kv;
      const int h = isq ? hh : hh - p.h_q;
      const uint16_t* base = isq ? p.q : p.k;
      src[k] = reinterpret_cast<const uint4*>(base + ((t0 + tb) * H + h) * kD + oct * 8);
      stride[k] = (int64_t)H * (kD / 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        sm[k][e] = 0.0f;
        mx[k][e] = -INFINITY;
        mn[k][e] = INFINITY;
      }
    }
    for (int t = tb; t < te; t += 4) {
      uint4 w[4][kStatUnits];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int k = 0; k < kStatUnits; ++k)
          w[j][k] = (act[k] && t + j < te) ? src[k][(int64_t)(t - tb + j) * stride[k]] : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (t + j < te) {
#pragma unroll
          for (int k = 0; k < kStatUnits; ++k) {
            const uint32_t wd[4] = {w[j][k].x, w[j][k].y, w[j][k].z, w[j][k].w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float x = __uint_as_float((e & 1) ? (wd[e >> 1] & 0xFFFF0000u) : (wd[e >> 1] << 16));
              sm[k][e] += x;
              mx[k][e] = fmaxf(mx[k][e], x);
              mn[k][e] = fminf(mn[k][e], x);
            }
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kStatUnits; ++k) {
      const int u = u0 + k * 256 + threadIdx.x;
      const int hh = u >> 4, oct = u & 15;
      if (nblk == 1) {
        // one block: its partial sum is the total (0 + partial, exact)
        float amax = 0.0f;
        if (act[k]) {
          uint16_t* mrow = mean_row(p, b, hh) + oct * 8;
          float mu[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            uint16_t m = 0;
            if (ss.want_sum) m = bf16_rne(__fdiv_rn(sm[k][e], (float)n));
            else if (!p.compute_stats && p.smooth) m = mrow[e];
            if (p.compute_stats) mrow[e] = m;
            mu[e] = bf16_to_f32(m);
          }
#pragma unroll
          for (int e = 0; e < 8; ++e)
            amax = fmaxf(amax, fmaxf(__builtin_fabsf(mx[k][e] - mu[e]), __builtin_fabsf(mn[k][e] - mu[e])));
        }
        // 16 lanes of one head row (units of one head are 16 consecutive lanes)
        for (int off = 1; off < 16; off <<= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
        if (act[k] && oct == 0) write_tscale(p, b, hh, amax);
      } else if (act[k]) {
        float* part = partial_ptr(p, t0, nblk, blk, ss.hs) + hh * kD + oct * 8;
#pragma unroll
        for (int e = 0; e < 8; e += 4) {
          *reinterpret_cast<float4*>(part + e) = make_float4(sm[k][e], sm[k][e + 1], sm[k][e + 2], sm[k][e + 3]);
          *reinterpret_cast<float4*>(part + ss.hs * kD + e) =
              make_float4(mx[k][e], mx[k][e + 1], mx[k][e + 2], mx[k][e + 3]);
          *reinterpret_cast<float4*>(part + 2 * ss.hs * kD + e) =
              make_float4(mn[k][e], mn[k][e + 1], mn[k][e + 2], mn[k][e + 3]);
        }
      }
    }
  }
}

// stats_final_kernel: one workgroup of 256 threads per (head, 32-channel
// slice, sequence), so that the partials of one head are read by four compute
// units.  The slice's partials arrive in LDS 256 blocks at a time (coalesced
// 128-byte rows, the next chunk in flight while the current one is added);
// threads 0..31 own one channel each and add its partials strictly in block
// order, then FP32 divide and BF16 rounding.  The tensor scale needs the amax
// of the whole head: each slice stores its own and counts itself in the
// head's arrival counter; the fourth arrival takes the maximum and writes the
// scale.  Counters and slice amaxes live in the spare bytes of the first
// block's q_codes rows (zeroed by stats_partial_kernel), which the quantizer
// overwrites later.  Sequences whose statistics need no partials (frozen
// statistics, empty or one-block sequences) are handled by slice 0 alone.
constexpr int kFinThreads = 256;
constexpr int kFinSlice = 32;                                        // channels per workgroup
constexpr int kFinChunk = 256;                                       // blocks per chunk
constexpr int kFinLoads = 3 * kFinChunk * (kFinSlice / 4) / kFinThreads;   // float4 loads per thread and chunk

__device__ __forceinline__ void fin_load(const QuantParams& p, int64_t t0, int nblk, int hs, int hh, int c0,
                                         int blk0, float4 (&r)[kFinLoads]) {
#pragma unroll
  for (int i = 0; i < kFinLoads; ++i) {
    const int idx = i * kFinThreads + (int)threadIdx.x;
    const int arr = idx / (kFinChunk * (kFinSlice / 4)), rem = idx % (kFinChunk * (kFinSlice / 4));
    const int blk = blk0 + rem / (kFinSlice / 4), q4 = rem % (kFinSlice / 4);
    r[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (blk < nblk)
      r[i] = *reinterpret_cast<const float4*>(partial_ptr(p, t0, nblk, blk, hs) + (int64_t)arr * hs * kD + hh * kD +
                                              c0 + 4 * q4);
  }
}

__global__ __launch_bounds__(kFinThreads) void stats_final_kernel(QuantParams p) {
  __shared__ float4 chunk[3 * kFinChunk * (kFinSlice / 4)];   // [sum, max, min][block][channel / 4]: 96 KB
  const int hh = blockIdx.x >> 2, slice = blockIdx.x & 3, b = blockIdx.y, t = threadIdx.x;
  const int64_t t0 = p.cu_seqlens[b];
  const int n = p.cu_seqlens[b + 1] - (int)t0;
  const int nblk = (n + 127) >> 7;
  if (p.need_partials && nblk == 1) return;   // finished by stats_partial_kernel
  const StatsShape ss = stats_shape(p);
  const bool have = p.need_partials && nblk >= 2;
  if (!have) {
    // no partials: the (frozen or zero) means and a zero amax, by slice 0
    if (slice != 0) return;
    if (t < kD) {
      uint16_t* mrow = mean_row(p, b, hh);
      uint16_t m = 0;
      if (!p.compute_stats && p.smooth) m = mrow[t];
      if (p.compute_stats) mrow[t] = m;
    }
    if (t == 0) write_tscale(p, b, hh, 0.0f);
    return;
  }
  const int c0 = slice * kFinSlice, c = c0 + t;
  float tot = 0.0f, mx = -INFINITY, mn = INFINITY;
  {
    float4 r[kFinLoads];
    fin_load(p, t0, nblk, ss.hs, hh, c0, 0, r);
    for (int blk0 = 0; blk0 < nblk; blk0 += kFinChunk) {
#pragma unroll
      for (int i = 0; i < kFinLoads; ++i) chunk[i * kFinThreads + t] = r[i];
      __syncthreads();
      if (blk0 + kFinChunk < nblk) fin_load(p, t0, nblk, ss.hs, hh, c0, blk0 + kFinChunk, r);
      if (t < kFinSlice) {
        const float* cs = reinterpret_cast<const float*>(chunk);
        const int nb = min(kFinChunk, nblk - blk0);
        // unrolled so that the LDS reads run ahead of the dependent additions
#pragma unroll 16
        for (int j = 0; j < nb; ++j) {
          tot += cs[j * kFinSlice + t];
          mx = fmaxf(mx, cs[(kFinChunk + j) * kFinSlice + t]);
          mn = fminf(mn, cs[(2 * kFinChunk + j) * kFinSlice + t]);
        }
      }
      __syncthreads();
    }
  }
  if (t < 64) {   // one wave: the slice's 32 channels
    float amax = 0.0f;
    if (t < kFinSlice) {
      uint16_t* mrow = mean_row(p, b, hh);
      uint16_t m = 0;
      if (ss.want_sum) m = bf16_rne(__fdiv_rn(tot, (float)n));
      else if (!p.compute_stats && p.smooth) m = mrow[c];
      if (p.compute_stats) mrow[c] = m;
      const float mu = bf16_to_f32(m);
      amax = fmaxf(__builtin_fabsf(mx - mu), __builtin_fabsf(mn - mu));
    }
    for (int off = 16; off >= 1; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
    if (t == 0) {
      uint8_t* scr = fin_scratch(p, t0, ss.hs);
      uint32_t* cnt = reinterpret_cast<uint32_t*>(scr) + hh;
      float* samax = reinterpret_cast<float*>(scr + ss.hs * 4) + hh * 4;
      samax[slice] = amax;
      // release: the slice amax is visible before the arrival is counted
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      if (atomicAdd(cnt, 1u) == 3u) {   // the head's last slice
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        const float a = fmaxf(fmaxf(samax[0], samax[1]), fmaxf(samax[2], samax[3]));
        write_tscale(p, b, hh, a);
      }
    }
  }
}

// NVFP4 quantization (Sec. 2.1 Eq. 1) of a 16-channel group of centered FP32
// values, in two steps so that the group may be spread over lanes: the scale
// from the group amax, then the codes of 8 channels at a time.
// rcp_sd[c] = RN(1 / e4m3_value(c)) for the positive E4M3 codes; with a
// power-of-two t, RN(1 / (t * sd)) = rcp_sd / t and RN(1 / (6 t)) = RN(1/6) / t.
struct Nv4Scale {
  uint32_t code;   // E4M3 scale byte
  float scale;     // t * sd (exact)
  float r;         // RN(1 / scale)
  int mode;        // 0: all codes are signed zeros; 1: product quotients; 2: IEEE division
};

__device__ __forceinline__ Nv4Scale nvfp4_scale(float a, float t, const float* rcp_sd) {
  const int kt = ilog2f(t);
  float q = div_by_scale(a, 6.0f * t, __builtin_ldexpf(kRcp6, -kt));   // RN(amax / (6 t))
  if (!(q < 0x1p100f)) q = 0x1p100f;   // an overflowing quotient saturates like +inf would
  Nv4Scale s;
  s.code = fp8_sat_pair(0u, q, 0.0f, false) & 0xFFu;                   // E4M3_RNE_sat
  const float sd = e4m3_value(s.code);
  s.scale = t * sd;   // exact: t is a power of two
  s.r = __builtin_ldexpf(rcp_sd[s.code], -kt);
  // quotients near the FP32 range (a frozen K tensor scale far below a later
  // token) take the IEEE division and the saturating encoder
  s.mode = sd == 0.0f ? 0 : (a * s.r < 0x1p100f ? 1 : 2);
  return s;
}

// Codes of 8 channels (element i in nibble i) under the group scale s.
__device__ __forceinline__ uint32_t nvfp4_encode8(const float* x, const Nv4Scale& s) {
  uint32_t w = 0;
  if (s.mode == 0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) w |= ((__float_as_uint(x[i]) >> 28) & 8u) << (4 * i);
  } else if (s.mode == 1) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      w = fp4_pair(w, div_by_scale(x[2 * j], s.scale, s.r), div_by_scale(x[2 * j + 1], s.scale, s.r), 1.0f, j);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) w |= e2m1_rne_sat(__fdiv_rn(x[i], s.scale)) << (4 * i);
  }
  return w;
}

// One whole group: 8 code bytes (as a 64-bit word, low nibble first) and the
// scale byte.
__device__ __forceinline__ uint64_t nvfp4_group(const float* xc, float t, const float* rcp_sd,
                                                uint32_t* scale_code) {
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) a = fmaxf(a, __builtin_fabsf(xc[i]));
  const Nv4Scale s = nvfp4_scale(a, t, rcp_sd);
  *scale_code = s.code;
  return (uint64_t)nvfp4_encode8(xc, s) | ((uint64_t)nvfp4_encode8(xc + 8, s) << 32);
}

// MXFP4 quantization of one 32-channel block held as 32 centered FP32 values:
// X = 2^e, e = floor(log2 amax) - 2 clamped to [-127, 127] (-127 for an
// all-zero block); codes E2M1_RNE_sat(x / X).  Returns 16 code bytes (element
// 2j in the low nibble of byte j).
__device__ __forceinline__ u32x4 mxfp4_group(const float* xc, uint32_t* scale_code) {
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < 32; ++i) a = fmaxf(a, __builtin_fabsf(xc[i]));
  int e = -127;
  if (a > 0.0f) e = max(-127, min(127, ilog2f(a) - 2));
  *scale_code = (uint32_t)(e + 127);
  // e = -127 only for an all-zero block, whose codes keep just the signs under
  // any scale; 2^-126 keeps the scale operand a normal number
  const float pw = __builtin_ldexpf(1.0f, max(e, -126));
  u32x4 w = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int j = 0; j < 4; ++j) w[q] = fp4_pair(w[q], xc[8 * q + 2 * j], xc[8 * q + 2 * j + 1], pw, j);
  return w;
}

// ---------------------------------------------------------------------------
// Quantization and cache write.  One workgroup (256 threads) per (sequence,
// 64-token chunk).
//   Q: group u of the chunk's rows is at u * group_elems in the packed input,
//   so consecutive lanes read and write consecutive groups; each lane has the
//   loads of several groups in flight before it quantizes them.
//   K and Delta_S: one lane per (token, KV head) row, the lanes of a wave on
//   consecutive tokens of one head.  The lane reads its row once; each group's
//   centered values feed both the quantizer and the Delta_S chains, so K is
//   read from HBM once.  Codes, scale rows and Delta_S entries of consecutive
//   tokens are consecutive in the cache pages: the stores are contiguous.
//   V: when the chunk's 64 tokens fill one cache page in order (the common
//   prefill case), each lane converts two channels of all 64 tokens and writes
//   their two channel-major 64-byte page rows whole; otherwise one byte per
//   (token, channel).
// ---------------------------------------------------------------------------
constexpr int kChunk = 64;
constexpr int kMeanStride = kD * 2 + 16;   // bytes per BF16 mean row in LDS (padded: rows on distinct banks)

// 8 centered values (x - mean, FP32) of the BF16 words v and m.
__device__ __forceinline__ void center8(const uint4 v, const uint4 m, float* xc) {
  const uint32_t vv[4] = {v.x, v.y, v.z, v.w}, mm[4] = {m.x, m.y, m.z, m.w};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const bool lo = (e & 1) == 0;
    const float xv = __uint_as_float(lo ? (vv[e >> 1] << 16) : (vv[e >> 1] & 0xFFFF0000u));
    const float mv = __uint_as_float(lo ? (mm[e >> 1] << 16) : (mm[e >> 1] & 0xFFFF0000u));
    xc[e] = xv - mv;
  }
}

// Max over the lanes of one quantization group (lane pairs, or quads for
// MXFP4): DPP swaps inside each quad of lanes.
template <bool MX>
__device__ __forceinline__ float group_max(float a) {
  a = fmaxf(a, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(a), 0xB1, 0xF, 0xF, false)));  // lane ^ 1
  if (MX) a = fmaxf(a, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(a), 0x4E, 0xF, 0xF, false)));  // lane ^ 2
  return a;
}

// Q rows: one lane per 8 channels (16 bytes) of a row, so a wave reads and
// writes 4 whole rows; the lanes of a group (2 for NVFP4, 4 for MXFP4) share
// its amax.  Each lane has U units in flight before it quantizes them.
template <bool MX>
__device__ __forceinline__ void quant_q_rows(const QuantParams& p, const uint8_t* mean_base, const float* tscale,
                                             int64_t tok0, int cnt, const float* rcp_sd) {
  constexpr int L = MX ? 4 : 2;          // lanes per group
  constexpr int U = 8;                   // units per lane in flight
  const int H = p.h_q;
  const int nun = cnt * H * 16;          // a multiple of 16: the lanes of a group act together
  const uint4* src = reinterpret_cast<const uint4*>(p.q + (tok0 * H) * kD);
  for (int u0 = threadIdx.x; u0 < nun; u0 += 256 * U) {
    uint4 v[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      v[k] = src[min(u0 + 256 * k, nun - 1)];   // past the end: not stored
      // the loads issue in unit order, all before the first unit is used
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int u = u0 + 256 * k;
      if (u < nun) {
        const int r = u >> 4, c8 = u & 15, h = r % H, g = c8 / L;
        float xc[8];
        center8(v[k], *reinterpret_cast<const uint4*>(mean_base + h * kMeanStride + c8 * 16), xc);
        float a = 0.0f;
#pragma unroll
        for (int i = 0; i < 8; ++i) a = fmaxf(a, __builtin_fabsf(xc[i]));
        a = group_max<MX>(a);
        const int64_t row = tok0 * H + r;
        uint32_t w, sc;
        if (MX) {
          int e = -127;
          if (a > 0.0f) e = max(-127, min(127, ilog2f(a) - 2));
          sc = (uint32_t)(e + 127);
          const float pw = __builtin_ldexpf(1.0f, max(e, -126));
          w = 0u;
#pragma unroll
          for (int j = 0; j < 4; ++j) w = fp4_pair(w, xc[2 * j], xc[2 * j + 1], pw, j);
        } else {
          const Nv4Scale s = nvfp4_scale(a, tscale[h], rcp_sd);
          sc = s.code;
          w = nvfp4_encode8(xc, s);
        }
        *reinterpret_cast<uint32_t*>(p.q_codes + row * 64 + c8 * 4) = w;
        if (c8 % L == 0) {
          p.q_scales[row * 8 + g] = (uint8_t)sc;
          if (MX) p.q_scales[row * 8 + 4 + g] = 0;
        }
      }
    }
  }
}

// codes[q] = w for a runtime q (selects, no indexed register access)
__device__ __forceinline__ void codes_put(u32x4 (&codes)[4], int q, u32x4 w) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (i == q) codes[i] = w;
}

// One K row: NVFP4 / MXFP4 codes and scale row into the cache, and
// Delta_S[h] = BF16(sum_c Qbar[h][c] * K_c[c]) as an FMA chain over c from +0
// (Eq. 9) for the query heads of the KV head's group, eight at a time.  The
// row is read a quarter (32 channels) at a time, the next quarter's loads in
// flight while the current one is used.
template <bool MX>
__device__ __forceinline__ void quant_k_rows(const QuantParams& p, const uint8_t* kmean_s, const uint8_t* qmean_s,
                                             const float* tscale, int64_t tok0, int cnt, const float* rcp_sd) {
  const int H = p.h_kv, grp = p.h_q / p.h_kv;
  for (int r = threadIdx.x; r < kChunk * H; r += 256) {
    const int i = r % kChunk, hk = r / kChunk;
    if (i >= cnt) continue;
    const uint4* kr = reinterpret_cast<const uint4*>(p.k + ((tok0 + i) * H + hk) * kD);
    const uint4* km = reinterpret_cast<const uint4*>(kmean_s + hk * kMeanStride);
    const int64_t slot = p.slot_mapping[tok0 + i];
    const int64_t crow = ((slot / kPage) * H + hk) * kPage + slot % kPage;
    const float t = tscale[hk];
    uint32_t scw[2] = {0u, 0u};
    u32x4 codes[4];   // the row's 64 code bytes, stored whole (partial-line stores cost write-backs)
    // the first pass over the row also quantizes it
    for (int j0 = 0; j0 == 0 || (p.smooth && j0 < grp); j0 += 8) {
      const int nj = p.smooth ? min(8, grp - j0) : 0;
      const uint8_t* qm = qmean_s + (hk * grp + j0) * kMeanStride;
      float d[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) d[j] = 0.0f;
      uint4 nxt[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) nxt[w] = kr[w];
#pragma unroll 1
      for (int qt = 0; qt < 4; ++qt) {   // channels 32 qt .. 32 qt + 31
        uint4 v[4];
#pragma unroll
        for (int w = 0; w < 4; ++w) v[w] = nxt[w];
        if (qt < 3) {
#pragma unroll
          for (int w = 0; w < 4; ++w) nxt[w] = kr[4 * (qt + 1) + w];
        }
        float xc[32];
#pragma unroll
        for (int w = 0; w < 4; ++w) center8(v[w], km[4 * qt + w], xc + 8 * w);
        if (j0 == 0) {
          uint32_t sc;
          if (MX) {
            const u32x4 cw = mxfp4_group(xc, &sc);
            codes_put(codes, qt, cw);
            scw[0] |= sc << (8 * qt);
          } else {
            uint32_t sc1;
            const uint64_t c0 = nvfp4_group(xc, t, rcp_sd, &sc);
            const uint64_t c1 = nvfp4_group(xc + 16, t, rcp_sd, &sc1);
            codes_put(codes, qt, (u32x4){(uint32_t)c0, (uint32_t)(c0 >> 32), (uint32_t)c1, (uint32_t)(c1 >> 32)});
            scw[qt >> 1] |= (sc | (sc1 << 8)) << (16 * (qt & 1));
          }
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          if (j < nj) {
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const uint4 qv = *reinterpret_cast<const uint4*>(qm + j * kMeanStride + (4 * qt + w) * 16);
              const uint32_t q4[4] = {qv.x, qv.y, qv.z, qv.w};
#pragma unroll
              for (int e = 0; e < 8; ++e) {
                const float qx = __uint_as_float((e & 1) == 0 ? (q4[e >> 1] << 16) : (q4[e >> 1] & 0xFFFF0000u));
                d[j] = __builtin_fmaf(qx, xc[8 * w + e], d[j]);
              }
            }
          }
        }
      }
      if (j0 == 0) {
        u32x4* co = reinterpret_cast<u32x4*>(p.k_codes + crow * 64);
#pragma unroll
        for (int q = 0; q < 4; ++q) co[q] = codes[q];
        *reinterpret_cast<uint2*>(p.k_scales + crow * 8) = make_uint2(scw[0], scw[1]);
      }
      uint16_t* dsrow = p.ds + ((slot / kPage) * p.h_q + hk * grp + j0) * kPage + slot % kPage;
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (j < nj) dsrow[(int64_t)j * kPage] = bf16_rne(d[j]);
    }
  }
}

template <bool MX>
__global__ __launch_bounds__(256) void quantize_kernel(QuantParams p) {
  __shared__ int page_start;   // 1: the chunk's tokens are slots 0, 1, ... of one page, in order
  __shared__ float rcp_sd[128];
  // [h_q + h_kv][kMeanStride] BF16 mean rows, then [h_q + h_kv] tensor scales
  extern __shared__ __attribute__((aligned(16))) uint8_t sm_mean[];
  const int b = blockIdx.y;
  const int64_t t0 = p.cu_seqlens[b];
  const int n = p.cu_seqlens[b + 1] - (int)t0;
  const int i0 = blockIdx.x * kChunk;
  if (i0 >= n) return;
  const int cnt = min(kChunk, n - i0);
  const int64_t tok0 = t0 + i0;
  const int tid = threadIdx.x;

  if (tid < 64) {
    const int64_t s0 = p.slot_mapping[tok0];
    const bool ok = (s0 % kPage == 0) && (tid >= cnt || p.slot_mapping[tok0 + tid] == s0 + tid);
    const bool all = __builtin_amdgcn_ballot_w64(!ok) == 0;
    if (tid == 0) page_start = all ? 1 : 0;
  }
  if (!MX && tid < 128) rcp_sd[tid] = (tid & 0x7F) && tid < 0x7F ? __fdiv_rn(1.0f, e4m3_value(tid)) : 0.0f;
  // the sequence's Q and K means (zero rows without smoothing)
  for (int u = tid; u < (p.h_q + p.h_kv) * (kD / 8); u += blockDim.x) {
    const int hh = u / (kD / 8), w = u % (kD / 8);
    uint4 m = make_uint4(0, 0, 0, 0);
    if (p.smooth) {
      const uint16_t* row = hh < p.h_q ? p.q_mean + ((int64_t)b * p.h_q + hh) * kD
                                       : p.k_mean + ((int64_t)b * p.h_kv + (hh - p.h_q)) * kD;
      m = reinterpret_cast<const uint4*>(row)[w];
    }
    *reinterpret_cast<uint4*>(sm_mean + hh * kMeanStride + w * 16) = m;
  }
  float* ts_s = reinterpret_cast<float*>(sm_mean + (p.h_q + p.h_kv) * kMeanStride);
  for (int hh = tid; hh < p.h_q + p.h_kv; hh += blockDim.x)
    ts_s[hh] = hh < p.h_q ? p.q_tscale[b * p.h_q + hh] : p.k_tscale[b * p.h_kv + (hh - p.h_q)];
  __syncthreads();
  const uint8_t* qmean_s = sm_mean;
  const uint8_t* kmean_s = sm_mean + p.h_q * kMeanStride;

  // Q rows (packed output); K rows (cache) with Delta_S
  quant_q_rows<MX>(p, qmean_s, ts_s, tok0, cnt, rcp_sd);
  quant_k_rows<MX>(p, kmean_s, qmean_s, ts_s + p.h_q, tok0, cnt, rcp_sd);
  __syncthreads();

  // V -> E4M3, channel-major page rows (plus the characterization copies in
  // v_aux: BF16 rows, or NVFP4 16-key groups along each channel row)
  const bool page_run = page_start && cnt == kChunk;   // whole page rows can be written
  if (page_run || (p.pv == 2 && page_start)) {
    const int64_t page = p.slot_mapping[tok0] / kPage;
    const int64_t aux_scales = p.num_pages * p.h_kv * kD * 32;   // NVFP4 scale plane offset
    for (int u = tid; u < p.h_kv * (kD / 2); u += blockDim.x) {
      const int h = u / (kD / 2), cp = u % (kD / 2);
      const uint32_t* src = reinterpret_cast<const uint32_t*>(p.v + (tok0 * p.h_kv + h) * kD) + cp;
      const int64_t tstride = (int64_t)p.h_kv * (kD / 2);
      const int64_t crow = (page * p.h_kv + h) * kD + 2 * cp;   // channel row 2cp; 2cp+1 follows
      uint8_t* dst = p.v_codes + crow * kPage;
      // the two 64-byte channel rows (one 128-byte line) are stored whole after
      // all 64 tokens are converted: stores of line pieces far apart in time
      // cost partial-line write-backs
      u32x4 r0s[kPage / 16], r1s[kPage / 16];
      // 16 tokens at a time: 16 bytes of each of the two channel rows
#pragma unroll
      for (int qq = 0; qq < kPage; qq += 16) {
        uint32_t w[16];
#pragma unroll
        for (int j = 0; j < 16; ++j) w[j] = qq + j < cnt ? src[(int64_t)(qq + j) * tstride] : 0u;
        if (page_run) {
          u32x4 r0, r1;   // bytes of channels 2cp and 2cp+1
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t* wq = w + 4 * q;
            uint32_t a = fp8_sat_pair(0u, __uint_as_float(wq[0] << 16), __uint_as_float(wq[1] << 16), false);
            a = fp8_sat_pair(a, __uint_as_float(wq[2] << 16), __uint_as_float(wq[3] << 16), true);
            uint32_t c = fp8_sat_pair(0u, __uint_as_float(wq[0] & 0xFFFF0000u), __uint_as_float(wq[1] & 0xFFFF0000u), false);
            c = fp8_sat_pair(c, __uint_as_float(wq[2] & 0xFFFF0000u), __uint_as_float(wq[3] & 0xFFFF0000u), true);
            r0[q] = a;
            r1[q] = c;
          }
          r0s[qq / 16] = r0;
          r1s[qq / 16] = r1;
          if (p.pv == 1) {   // BF16 rows: 16 keys of each channel, 32 bytes
            uint32_t b0[8], b1[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
              b0[j] = (w[2 * j] & 0xFFFFu) | (w[2 * j + 1] << 16);
              b1[j] = (w[2 * j] >> 16) | (w[2 * j + 1] & 0xFFFF0000u);
            }
            uint16_t* a16 = reinterpret_cast<uint16_t*>(p.v_aux) + crow * kPage + qq;
            *reinterpret_cast<u32x4*>(a16) = (u32x4){b0[0], b0[1], b0[2], b0[3]};
            *reinterpret_cast<u32x4*>(a16 + 8) = (u32x4){b0[4], b0[5], b0[6], b0[7]};
            *reinterpret_cast<u32x4*>(a16 + kPage) = (u32x4){b1[0], b1[1], b1[2], b1[3]};
            *reinterpret_cast<u32x4*>(a16 + kPage + 8) = (u32x4){b1[4], b1[5], b1[6], b1[7]};
          }
        }
        if (p.pv == 2) {   // one NVFP4 group per channel: these 16 keys (absent ones zero)
          float x0[16], x1[16];
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            x0[j] = __uint_as_float(w[j] << 16);
            x1[j] = __uint_as_float(w[j] & 0xFFFF0000u);
          }
          uint32_t sc0, sc1;
          const uint64_t c0 = nvfp4_group(x0, 1.0f, rcp_sd, &sc0);
          const uint64_t c1 = nvfp4_group(x1, 1.0f, rcp_sd, &sc1);
          *reinterpret_cast<uint64_t*>(p.v_aux + crow * 32 + qq / 2) = c0;
          *reinterpret_cast<uint64_t*>(p.v_aux + (crow + 1) * 32 + qq / 2) = c1;
          p.v_aux[aux_scales + crow * 4 + qq / 16] = (uint8_t)sc0;
          p.v_aux[aux_scales + (crow + 1) * 4 + qq / 16] = (uint8_t)sc1;
        }
      }
      if (page_run) {
#pragma unroll
        for (int q = 0; q < kPage / 16; ++q) {
          *reinterpret_cast<u32x4*>(dst + 16 * q) = r0s[q];
          *reinterpret_cast<u32x4*>(dst + kPage + 16 * q) = r1s[q];
        }
      }
    }
  }
  if (!page_run) {
    for (int u = tid; u < cnt * p.h_kv * kD; u += blockDim.x) {
      const int c = u % kD, ih = u / kD;
      const int h = ih % p.h_kv, i = ih / p.h_kv;
      const int64_t slot = p.slot_mapping[tok0 + i];
      const uint16_t vb = p.v[(tok0 + i) * p.h_kv * kD + (int64_t)h * kD + c];
      const int64_t at = (((slot / kPage) * p.h_kv + h) * kD + c) * kPage + slot % kPage;
      p.v_codes[at] = (uint8_t)e4m3_rne_sat(bf16_to_f32(vb));
      if (p.pv == 1) reinterpret_cast<uint16_t*>(p.v_aux)[at] = vb;
    }
  }
}

__global__ void convert_kernel(int fmt, const float* x, int64_t n, uint8_t* out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  uint32_t c;
  if (fmt >= 0x400) {   // reference for 0x200 + b: exact scaling, then the software encoder
    c = e2m1_rne_sat(__builtin_ldexpf(x[i], 127 - (fmt & 0xFF)));
  } else if (fmt >= 0x300) {   // reference for 0x100 + c: IEEE division, then the software encoder
    c = e2m1_rne_sat(__fdiv_rn(x[i], e4m3_value(fmt & 0xFF)));
  } else if (fmt >= 0x200) {   // MXFP4 element: x / 2^e, e = (fmt & 0xFF) - 127 >= -126
    c = fp4_pair(0u, x[i], 0.0f, __builtin_ldexpf(1.0f, (fmt & 0xFF) - 127), 0) & 0xFu;
  } else if (fmt >= 0x100) {   // NVFP4 element: x / e4m3_value(fmt & 0xFF), the quantizer's division
    const float s = e4m3_value(fmt & 0xFF), r = __fdiv_rn(1.0f, s);
    if (__builtin_fabsf(x[i]) * r < 0x1p100f) c = fp4_pair(0u, div_by_scale(x[i], s, r), 0.0f, 1.0f, 0) & 0xFu;
    else c = e2m1_rne_sat(__fdiv_rn(x[i], s));   // the quantizer's fallback near the FP32 range
  } else {
    switch (fmt) {
      case 0: c = e4m3_rne_sat(x[i]); break;
      case 1: c = e2m1_rne_sat(x[i]); break;
      case 2: c = fp8_sat_pair(0u, x[i], 0.0f, false) & 0xFFu; break;
      default: c = fp4_pair(0u, x[i], 0.0f, 1.0f, 0) & 0xFu; break;
    }
  }
  out[i] = (uint8_t)c;
}

hipError_t launch_quantize(const QuantParams& p, hipStream_t stream) {
  const int hs = p.h_q + (p.stats_k ? p.h_kv : 0);
  if (p.need_partials && p.max_seqlen > 0) {
    stats_partial_kernel<<<dim3((p.max_seqlen + 127) / 128, p.batch), dim3(256), 0, stream>>>(p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  stats_final_kernel<<<dim3(hs * 4, p.batch), dim3(kFinThreads), 0, stream>>>(p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.total_tokens > 0 && p.max_seqlen > 0) {
    const dim3 grid((p.max_seqlen + kChunk - 1) / kChunk, p.batch);
    const size_t lds = (size_t)(p.h_q + p.h_kv) * (kMeanStride + sizeof(float));
    if (p.mx) quantize_kernel<true><<<grid, dim3(256), lds, stream>>>(p);
    else quantize_kernel<false><<<grid, dim3(256), lds, stream>>>(p);
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
