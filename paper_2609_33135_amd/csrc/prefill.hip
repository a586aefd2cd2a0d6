// prefill.hip -- causal QK4PV8 prefill for gfx950 (Algorithm 1 main loop).
//
// One workgroup = 8 waves = 256 query rows of one query head; each wave owns
// 32 rows (two 16-row MFMA column blocks).  Per 128-key tile (visited from the
// block's last tile down to tile 0, Sec. 4.1):
//   * the workgroup stages the tile in LDS: NVFP4 K dequantized once to exact
//     FP16 (group scale applied, tensor scale factored out), FP8 V in its
//     channel-major page layout, and the compensation vector Delta_S;
//   * each wave computes S^T = K Q^T on FP16 MFMA (16x16x32), seeded by one
//     BF16 rank-one MFMA per 16x16 block that writes Delta_S into the
//     accumulator first (Sec. 4.3 Eq. 11, Sec. 5.2);
//   * mask, row max, P = 2^(lambda (S - m) + log2 448), row sum of the FP32 P,
//     FP8 conversion in registers; the S^T accumulator layout is already the
//     B-operand layout of the FP8 PV MFMA (O^T = V^T P^T), so P never leaves
//     registers;
//   * O^T rescale (skipped when no row maximum moved) and FP8 MFMA
//     (16x16x128) accumulation.
// The key order inside a 16-row MFMA block is permuted so that the 32 keys a
// lane holds after the QK product are contiguous: MFMA row r of key block mb
// is key 32*(r/4) + 4*mb + r%4.
#include "mpfa_device.h"
#include "mpfa_internal.h"

namespace mpfa {

namespace {

constexpr int kWaves = 8;
constexpr int kNB = 2;                       // 16-row query blocks per wave
constexpr int kQRows = kWaves * kNB * 16;    // 256 query rows per workgroup
constexpr int kThreads = kWaves * 64;

struct PrefillSmem {
  uint8_t k[kTile * 256];   // FP16 [key][128], 16-byte chunks XOR-swizzled per key
  uint8_t v[kD * kTile];    // FP8 [channel][key], 16-byte chunks XOR-swizzled per channel
  uint16_t ds[kTile];       // BF16 seed values in accumulator units
};

// chunk swizzles: conflict-free 16-byte reads for the MFMA operand patterns
__device__ __forceinline__ int k_swz(int key) { return (((key >> 5) << 2) | (key & 3)) & 15; }
__device__ __forceinline__ int v_swz(int d) { return (d >> 1) & 7; }

__device__ __forceinline__ u32x4 zero_tail(u32x4 w, int nvalid) {
  // keep bytes [0, nvalid) of the 16-byte word
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int keep = nvalid - 4 * i;
    uint32_t mask = keep >= 4 ? 0xFFFFFFFFu : (keep <= 0 ? 0u : ((1u << (8 * keep)) - 1u));
    w[i] &= mask;
  }
  return w;
}

__device__ __forceinline__ void load_tile(PrefillSmem& sm, const PrefillParams& p, int b, int hk,
                                          int h, int j, int kvl, float seed_scale) {
  const int t = threadIdx.x;
  const int32_t* pt = p.page_table + (int64_t)b * p.max_pages;
  {  // K: 4 threads per key, 32 channels each
    const int key = t >> 2, qt = t & 3;
    const int kabs = j * kTile + key;
    u32x4 codes = {0u, 0u, 0u, 0u};
    uint32_t sc = 0;
    if (kabs < kvl) {
      const int64_t page = pt[kabs >> 6];
      const int64_t row = (page * p.h_kv + hk) * kPage + (kabs & 63);
      codes = *reinterpret_cast<const u32x4*>(p.k_codes + row * 64 + qt * 16);
      sc = *reinterpret_cast<const uint16_t*>(p.k_scales + row * 8 + qt * 2);
    }
    const ScaleSplit s0 = split_e4m3(sc & 0xFFu), s1 = split_e4m3((sc >> 8) & 0xFFu);
    uint8_t* rowp = sm.k + key * 256;
    const int sw = k_swz(key);
    *reinterpret_cast<f16x8*>(rowp + (((4 * qt + 0) ^ sw) << 4)) = dequant8(codes[0], s0);
    *reinterpret_cast<f16x8*>(rowp + (((4 * qt + 1) ^ sw) << 4)) = dequant8(codes[1], s0);
    *reinterpret_cast<f16x8*>(rowp + (((4 * qt + 2) ^ sw) << 4)) = dequant8(codes[2], s1);
    *reinterpret_cast<f16x8*>(rowp + (((4 * qt + 3) ^ sw) << 4)) = dequant8(codes[3], s1);
  }
  {  // V: 4 threads per channel, 32 keys each
    const int d = t >> 2, part = t & 3;
    const int kbase = j * kTile + part * 32;
    u32x4 v0 = {0u, 0u, 0u, 0u}, v1 = {0u, 0u, 0u, 0u};
    if (kbase < kvl) {
      const int64_t page = pt[kbase >> 6];
      const uint8_t* src = p.v_codes + ((page * p.h_kv + hk) * kD + d) * kPage + (kbase & 63);
      v0 = *reinterpret_cast<const u32x4*>(src);
      v1 = *reinterpret_cast<const u32x4*>(src + 16);
      if (kbase + 32 > kvl) {
        v0 = zero_tail(v0, kvl - kbase);
        v1 = zero_tail(v1, kvl - kbase - 16);
      }
    }
    uint8_t* rowp = sm.v + d * kTile;
    const int sw = v_swz(d);
    *reinterpret_cast<u32x4*>(rowp + (((2 * part) ^ sw) << 4)) = v0;
    *reinterpret_cast<u32x4*>(rowp + (((2 * part + 1) ^ sw) << 4)) = v1;
  }
  if (t < kTile) {
    const int kabs = j * kTile + t;
    uint16_t v = 0;
    if (p.smooth && kabs < kvl) {
      const int64_t page = pt[kabs >> 6];
      const float x = bf16_to_f32(p.ds[(page * p.h_q + h) * kPage + (kabs & 63)]) * seed_scale;
      v = bf16_rne(x);   // exact: a BF16 value times a power of two
    }
    sm.ds[t] = v;
  }
}

template <bool SMOOTH>
__global__ __launch_bounds__(kThreads, 1) void prefill_kernel(PrefillParams p) {
  __shared__ __attribute__((aligned(16))) PrefillSmem sm;

  // ---- work item: largest query tiles first (longest-processing-time order)
  int b, h, rank;
  {
    const int bid = blockIdx.x;
    if (p.xcd_remap) {
      // block ids are dealt round-robin to the 8 XCDs; give each XCD the query
      // heads of a fixed subset of KV heads so their K/V tiles share its L2.
      const int xcd = bid & 7, slot = bid >> 3;
      const int kvpx = p.h_kv / 8, grp = p.h_q / p.h_kv;
      const int ipr = kvpx * grp * p.batch;
      rank = slot / ipr;
      int r = slot % ipr;
      const int hk = xcd * kvpx + r % kvpx;
      r /= kvpx;
      h = hk * grp + r % grp;
      b = r / grp;
    } else {
      const int per = p.h_q * p.batch;
      rank = bid / per;
      const int rem = bid % per;
      h = rem % p.h_q;
      b = rem / p.h_q;
    }
  }
  const int qtile = p.n_qtiles - 1 - rank;
  const int q0 = p.cu_seqlens_q[b];
  const int nq = p.cu_seqlens_q[b + 1] - q0;
  const int r0 = qtile * kQRows;
  if (r0 >= nq) return;

  const int qs = p.q_start[b], kvl = p.kv_len[b];
  const int grp = p.h_q / p.h_kv, hk = h / grp;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 4, lr = lane & 15;
  const int last_row = min(r0 + kQRows, nq) - 1;
  const int j_hi = (qs + last_row) >> 7;

  const float tq = p.q_tscale[b * p.h_q + h], tk = p.k_tscale[b * p.h_kv + hk];
  const int eqk = ilog2f(tq) + ilog2f(tk);
  const float lam2 = __builtin_ldexpf(p.lam, eqk);        // lambda * tQ * tK
  const float seed_scale = __builtin_ldexpf(1.0f, -eqk);  // Delta_S in accumulator units

  const int wrow0 = r0 + wave * (kNB * 16);
  const bool wave_active = wrow0 < nq;
  const int wpos_min = qs + wrow0;
  const int wpos_max = qs + min(wrow0 + kNB * 16, nq) - 1;

  // ---- Q operands (B of S^T = K Q^T): exact FP16, tensor scale factored out
  f16x8 qop[kNB][4];
  int pos[kNB];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const int row = wrow0 + nb * 16 + lr;
    pos[nb] = qs + row;
    const bool valid = row < nq;
    const int64_t tok = q0 + (valid ? row : 0);
    const uint8_t* qc = p.q_codes + (tok * p.h_q + h) * 64;
    const uint8_t* qsc = p.q_scales + (tok * p.h_q + h) * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint32_t cw = valid ? *reinterpret_cast<const uint32_t*>(qc + 16 * ks + 4 * g) : 0u;
      const uint32_t sc = valid ? qsc[2 * ks + (g >> 1)] : 0u;
      qop[nb][ks] = dequant8(cw, split_e4m3(sc));
    }
  }

  bf16x8 bseed = {};
  if (lane < 16) bseed[0] = (__bf16)1.0f;

  float m[kNB], l[kNB];
  f32x4 o[8][kNB];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    m[nb] = -INFINITY;
    l[nb] = 0.0f;
#pragma unroll
    for (int db = 0; db < 8; ++db) o[db][nb] = (f32x4){0.f, 0.f, 0.f, 0.f};
  }

  for (int j = j_hi; j >= 0; --j) {
    __syncthreads();
    load_tile(sm, p, b, hk, h, j, kvl, seed_scale);
    __syncthreads();
    if (!wave_active) continue;
    const int key0 = j * kTile;
    if (key0 > wpos_max) continue;   // tile entirely after every row of this wave
    const bool need_mask = key0 + kTile - 1 > wpos_min;

    // ---- S^T = seed + K Q^T
    f32x4 s[8][kNB];
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const int krow = 32 * (lr >> 2) + 4 * mb + (lr & 3);
      if (SMOOTH) {
        bf16x8 aseed = {};
        if (lane < 16) aseed[0] = __builtin_bit_cast(__bf16, sm.ds[krow]);
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) s[mb][nb] = mfma_bf16(aseed, bseed, (f32x4){0.f, 0.f, 0.f, 0.f});
      } else {
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) s[mb][nb] = (f32x4){0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const f16x8 kop = *reinterpret_cast<const f16x8*>(sm.k + krow * 256 + (((4 * ks + g) ^ lr) << 4));
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) s[mb][nb] = mfma_f16(kop, qop[nb][ks], s[mb][nb]);
      }
    }
    if (need_mask) {
#pragma unroll
      for (int mb = 0; mb < 8; ++mb)
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (key0 + 32 * g + 4 * mb + i > pos[nb]) s[mb][nb][i] = -INFINITY;
    }

    // ---- online softmax; P (x448) to FP8 in the PV operand layout
    i32x8 pb[kNB];
    float alpha[kNB];
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) {
      float mx = -INFINITY;
#pragma unroll
      for (int mb = 0; mb < 8; ++mb)
        mx = fmaxf(fmaxf(mx, fmaxf(s[mb][nb][0], s[mb][nb][1])), fmaxf(s[mb][nb][2], s[mb][nb][3]));
      mx = wave_max16(mx);
      const float mnew = fmaxf(m[nb], mx);
      const float muse = (mnew == -INFINITY) ? 0.0f : mnew;
      alpha[nb] = (m[nb] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f((m[nb] - muse) * lam2);
      m[nb] = mnew;
      float ps = 0.0f;
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
        float e[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) e[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[mb][nb][i] - muse, lam2, kLog2_448));
        ps += (e[0] + e[1]) + (e[2] + e[3]);
        pb[nb][mb] = (int)pack_fp8x4(e[0], e[1], e[2], e[3]);
      }
      l[nb] = alpha[nb] * l[nb] + ps;
    }
    bool moved = false;
#pragma unroll
    for (int nb = 0; nb < kNB; ++nb) moved |= alpha[nb] != 1.0f;
    if (__builtin_amdgcn_ballot_w64(moved) != 0) {
#pragma unroll
      for (int db = 0; db < 8; ++db)
#pragma unroll
        for (int nb = 0; nb < kNB; ++nb) o[db][nb] *= alpha[nb];
    }

    // ---- O^T += V^T P^T (FP8)
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      const int d = 16 * db + lr;
      const uint8_t* vr = sm.v + d * kTile;
      const int sw = v_swz(d);
      const u32x4 va = *reinterpret_cast<const u32x4*>(vr + (((2 * g) ^ sw) << 4));
      const u32x4 vb = *reinterpret_cast<const u32x4*>(vr + (((2 * g + 1) ^ sw) << 4));
      const i32x8 vop = {(int)va[0], (int)va[1], (int)va[2], (int)va[3],
                         (int)vb[0], (int)vb[1], (int)vb[2], (int)vb[3]};
#pragma unroll
      for (int nb = 0; nb < kNB; ++nb) o[db][nb] = mfma_fp8(vop, pb[nb], o[db][nb]);
    }
  }

  if (!wave_active) return;
  // ---- epilogue: out = O / (448 l), BF16
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    const float lt = wave_sum16(l[nb]);
    const int row = wrow0 + nb * 16 + lr;
    if (row < nq) {
      uint16_t* dst = p.out + ((int64_t)(q0 + row) * p.h_q + h) * kD;
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const uint32_t lo = (uint32_t)bf16_rne(__fdiv_rn(o[db][nb][0], lt)) |
                            ((uint32_t)bf16_rne(__fdiv_rn(o[db][nb][1], lt)) << 16);
        const uint32_t hi = (uint32_t)bf16_rne(__fdiv_rn(o[db][nb][2], lt)) |
                            ((uint32_t)bf16_rne(__fdiv_rn(o[db][nb][3], lt)) << 16);
        *reinterpret_cast<uint2*>(dst + 16 * db + 4 * g) = make_uint2(lo, hi);
      }
    }
  }
}

}  // namespace

hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream) {
  const unsigned blocks = (unsigned)(p.n_qtiles * p.h_q * p.batch);
  if (blocks == 0) return hipSuccess;
  if (p.smooth)
    prefill_kernel<true><<<dim3(blocks), dim3(kThreads), 0, stream>>>(p);
  else
    prefill_kernel<false><<<dim3(blocks), dim3(kThreads), 0, stream>>>(p);
  return hipGetLastError();
}

int prefill_query_rows_per_block() { return kQRows; }

}  // namespace mpfa
