// prefill_body.h -- the causal prefill work item (Algorithm 1 main loop) as a
// device function, shared by the prefill kernel and the fused mixed-step kernel.
#pragma once
#include "mpfa_device.h"
#include "mpfa_internal.h"

namespace mpfa {

namespace {

constexpr int kQRows = 256;                  // query rows per workgroup
constexpr int kNB = 2;                       // 16-row query blocks per wave (two waves per SIMD)
// threads of a workgroup whose waves own NB 16-row query blocks each
constexpr int threads_for(int nb) { return kQRows / (nb * 16) * 64; }
constexpr int kThreads = threads_for(kNB);

// Precision of the PV product: the method's FP8 (P * 448 and V in E4M3), or
// the two other assignments compared in Sec. 3.1 / Fig. 3a, BF16 P and V, and
// NVFP4 P (2688 P quantized per 16 keys with dynamic E4M3 scales) with NVFP4 V
// (16-key groups per channel, tensor scale 1), both on FP16 / BF16 MFMA after
// exact dequantization.
enum PvMode { kPvFp8 = 0, kPvBf16 = 1, kPvNvfp4 = 2 };

template <int PV>
struct PrefillSmemT {
  // NVFP4: FP16 [key][128], 16-byte chunks XOR-swizzled per key.  MXFP4: raw
  // codes [key][64] (chunks swizzled by mx_swz) in the first 8 KB, then the
  // E8M0 scales transposed to [MFMA row][32-channel block][16-key block].
  uint8_t k[kTile * 256];
  // FP8: [channel][key] bytes, 16-byte chunks XOR-swizzled per channel (v_swz).
  // BF16 / NVFP4: [channel][key] BF16 or exact FP16, 256-byte rows of 16
  // chunks, chunk c of channel d stored at position c ^ (d & 15).
  uint8_t v[kD * kTile * (PV == kPvFp8 ? 1 : 2)];
  float ds[kTile];          // seed values (BF16 values in accumulator units) as FP32, key order
  // the same values ordered for the rank-one seed MFMA: the 8 values lane lr
  // contributes (row lr of key blocks 0..7) are contiguous, one 16-byte read
  uint16_t dss[kTile];
};

// position in PrefillSmemT::dss of key `key`: MFMA row 4*(key/32) + key%4 of
// 16-key block (key/4)%8 (the key permutation of the score blocks)
__device__ __forceinline__ int seed_slot(int key) {
  return (4 * (key >> 5) + (key & 3)) * 8 + ((key >> 2) & 7);
}

// chunk swizzles: conflict-free 16-byte reads for the MFMA operand patterns
__device__ __forceinline__ int k_swz(int key) { return (((key >> 5) << 2) | (key & 3)) & 15; }
__device__ __forceinline__ int v_swz(int d) { return (d >> 1) & 7; }
__device__ __forceinline__ int mx_swz(int key) { return ((key >> 1) & 1) | (((key >> 5) & 1) << 1); }
constexpr int kMxScaleOff = kTile * 64;   // byte offset of the MXFP4 scales in PrefillSmem::k

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

// Raw bytes of one KV tile held in registers between the global load and the
// LDS store (software pipelining: the next tile is fetched while the current
// one is computed).
template <int PV>
struct TileRegs {
  u32x4 kc;        // 16 NVFP4 code bytes: key t/4, channels 32*(t%4) .. +31
  uint32_t ksc;    // their two E4M3 group scales
  // channel t/4, keys 32*(t%4) .. +31 of the tile: 32 FP8 bytes, 32 BF16
  // values, or 32 E2M1 codes (16 bytes)
  static constexpr int kVWords = PV == kPvFp8 ? 2 : (PV == kPvBf16 ? 4 : 1);
  u32x4 v[kVWords];
  uint32_t vsc;    // NVFP4 V: the two E4M3 scales of those keys
  uint32_t ds;     // BF16 Delta_S of key t (threads 0..127)
};

// t: the unit of the tile (0..511) this call loads
template <bool MX, int PV>
__device__ __forceinline__ void fetch_tile(TileRegs<PV>& r, const PrefillParams& p, const int32_t* pt,
                                           int hk, int h, int j, int kvl, int t) {
  // the two pages of tile j: uniform across the workgroup (scalar loads)
  const int npg = (kvl + 63) >> 6;
  const int64_t pg0 = pt[min(2 * j, npg - 1)];
  const int64_t pg1 = pt[min(2 * j + 1, npg - 1)];
  {
    const int key = t >> 2, qt = t & 3;
    const int kabs = j * kTile + key;
    const int64_t row = ((key < 64 ? pg0 : pg1) * p.h_kv + hk) * kPage + (kabs & 63);
    r.kc = (u32x4){0u, 0u, 0u, 0u};
    r.ksc = 0;
    if (kabs < kvl) {
      r.kc = *reinterpret_cast<const u32x4*>(p.k_codes + row * 64 + qt * 16);
      r.ksc = MX ? (uint32_t)p.k_scales[row * 8 + qt]
                 : (uint32_t)*reinterpret_cast<const uint16_t*>(p.k_scales + row * 8 + qt * 2);
    }
  }
  {
    const int d = t >> 2, part = t & 3;
    const int kbase = j * kTile + part * 32;
    const int64_t crow = ((part < 2 ? pg0 : pg1) * p.h_kv + hk) * kD + d;   // channel row of the page
#pragma unroll
    for (int i = 0; i < TileRegs<PV>::kVWords; ++i) r.v[i] = (u32x4){0u, 0u, 0u, 0u};
    r.vsc = 0;
    if (kbase < kvl) {
      if (PV == kPvFp8) {
        const uint8_t* src = p.v_codes + crow * kPage + (kbase & 63);
        r.v[0] = *reinterpret_cast<const u32x4*>(src);
        r.v[1 % TileRegs<PV>::kVWords] = *reinterpret_cast<const u32x4*>(src + 16);
        if (kbase + 32 > kvl) {
          r.v[0] = zero_tail(r.v[0], kvl - kbase);
          r.v[1 % TileRegs<PV>::kVWords] = zero_tail(r.v[1 % TileRegs<PV>::kVWords], kvl - kbase - 16);
        }
      } else if (PV == kPvBf16) {
        const uint8_t* src = p.v_aux + (crow * kPage + (kbase & 63)) * 2;
#pragma unroll
        for (int i = 0; i < TileRegs<PV>::kVWords; ++i) {
          r.v[i] = *reinterpret_cast<const u32x4*>(src + 16 * i);
          // keys past kv_len: zero (slots not written may hold any bits)
          if (kbase + 32 > kvl) r.v[i] = zero_tail(r.v[i], 2 * (kvl - kbase) - 16 * i);
        }
      } else {
        // NVFP4 dequantizes to finite values whatever the bytes, and P is 0 on
        // keys past kv_len: nothing to clear
        r.v[0] = *reinterpret_cast<const u32x4*>(p.v_aux + crow * 32 + (kbase & 63) / 2);
        r.vsc = *reinterpret_cast<const uint16_t*>(p.v_aux + p.num_pages * p.h_kv * kD * 32 + crow * 4 +
                                                   (kbase & 63) / 16);
      }
    }
  }
  r.ds = 0;
  if (t < kTile) {
    const int kabs = j * kTile + t;
    if (p.smooth && kabs < kvl)
      r.ds = p.ds[((t < 64 ? pg0 : pg1) * p.h_q + h) * kPage + (kabs & 63)];
  }
}

template <bool MX, int PV>
__device__ __forceinline__ void store_tile(PrefillSmemT<PV>& sm, const TileRegs<PV>& r, float seed_scale, int t) {
  if (MX) {
    const int key = t >> 2, qt = t & 3;
    *reinterpret_cast<u32x4*>(sm.k + key * 64 + ((qt ^ mx_swz(key)) << 4)) = r.kc;
    // key -> MFMA row 4*(key/32) + key%4 of 16-key block (key/4)%8
    const int mrow = 4 * (key >> 5) + (key & 3), mblk = (key >> 2) & 7;
    sm.k[kMxScaleOff + (mrow * 4 + qt) * 8 + mblk] = (uint8_t)r.ksc;
  } else {
    const int key = t >> 2, qt = t & 3;
    const ScaleSplit s0 = split_e4m3(r.ksc & 0xFFu), s1 = split_e4m3((r.ksc >> 8) & 0xFFu);
    uint8_t* rowp = sm.k + key * 256;
    const int sw = k_swz(key);
    *reinterpret_cast<f16x8*>(rowp + (((4 * qt + 0) ^ sw) << 4)) = dequant8(r.kc[0], s0);
    *reinterpret_cast<f16x8*>(rowp + (((4 * qt + 1) ^ sw) << 4)) = dequant8(r.kc[1], s0);
    *reinterpret_cast<f16x8*>(rowp + (((4 * qt + 2) ^ sw) << 4)) = dequant8(r.kc[2], s1);
    *reinterpret_cast<f16x8*>(rowp + (((4 * qt + 3) ^ sw) << 4)) = dequant8(r.kc[3], s1);
  }
  {
    const int d = t >> 2, part = t & 3;
    if (PV == kPvFp8) {
      uint8_t* rowp = sm.v + d * kTile;
      const int sw = v_swz(d);
      *reinterpret_cast<u32x4*>(rowp + (((2 * part) ^ sw) << 4)) = r.v[0];
      *reinterpret_cast<u32x4*>(rowp + (((2 * part + 1) ^ sw) << 4)) = r.v[1 % TileRegs<PV>::kVWords];
    } else {
      uint8_t* rowp = sm.v + d * (kTile * 2);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        u32x4 w;
        if (PV == kPvBf16) {
          w = r.v[i % TileRegs<PV>::kVWords];
        } else {   // 8 codes of keys 32 part + 8i .. +7, the scale of their 16-key group
          const f16x8 hv = dequant8(r.v[0][i], split_e4m3((r.vsc >> (8 * (i >> 1))) & 0xFFu));
          w = __builtin_bit_cast(u32x4, hv);
        }
        *reinterpret_cast<u32x4*>(rowp + (((4 * part + i) ^ (d & 15)) << 4)) = w;
      }
    }
  }
  // exact: a BF16 value times a power of two stays a BF16 value
  if (t < kTile) {
    const uint16_t v = bf16_rne(bf16_to_f32((uint16_t)r.ds) * seed_scale);
    sm.ds[t] = bf16_to_f32(v);
    sm.dss[seed_slot(t)] = v;
  }
}

// How the compensation 1 Delta_S^T (Sec. 4.3 Eq. 11) enters the score
// accumulator before the QK product:
//  kSeedMfma  one BF16 rank-one MFMA per 16-key block (A = the block's Delta_S
//             in reduction slot 0, B = ones in slot 0); it depends on the keys
//             only, so its result seeds every query block of the wave;
//  kSeedInit  the same rank-one matrix loaded directly as the accumulator input
//             of the first FP16 MFMA (bit-identical: both start the accumulator
//             at the FP32 value of the BF16 Delta_S);
//  kSeedNone  no compensation (the unsmoothed "direct" variant);
//  kSeedElem  the placement the rank-one seed replaces (Sec. 3.2, Fig. 10):
//             the accumulator starts at zero and Delta_S is added to every
//             score in FP32 after the QK product, on the softmax path.  Same
//             values up to the FP32 rounding order.
enum SeedMode { kSeedNone = 0, kSeedMfma = 1, kSeedInit = 2, kSeedElem = 3 };

// Per-item state of one wave: the work item, the query operands, the softmax
// scale and the row positions.
template <int NB = kNB>
struct ItemState {
  int b, h, hk, q0, nq, qs, kvl, j_hi;
  int lane, wave, g, lr;
  int wrow0, wpos_min, wpos_max;
  bool wave_active;
  float lam2, seed_scale;
  int pos[NB];
  f16x8 qop[NB][4];   // NVFP4: exact FP16 query operands, tensor scale factored out
  u32x4 qraw[NB];     // MXFP4: raw codes of channels 32g .. 32g+31
  int qscale[NB];     // MXFP4: their E8M0 scale
  bf16x8 bseed;        // B operand of the rank-one seed MFMA: 1 in slot 0 of lanes 0..15
};

// Decode work item `bid` (largest query tiles first, longest-processing-time
// order) and load the wave's query operands.  Returns false when the item has
// no rows.
template <bool MX, int NB = kNB>
__device__ __forceinline__ bool item_setup(const PrefillParams& p, int bid, ItemState<NB>& st) {
  int b, h, rank;
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
  const int qtile = p.n_qtiles - 1 - rank;
  const int q0 = p.cu_seqlens_q[b];
  const int nq = p.cu_seqlens_q[b + 1] - q0;
  const int r0 = qtile * kQRows;
  if (r0 >= nq) return false;

  st.b = b;
  st.h = h;
  st.q0 = q0;
  st.nq = nq;
  st.qs = p.q_start[b];
  st.kvl = p.kv_len[b];
  st.hk = h / (p.h_q / p.h_kv);
  st.lane = threadIdx.x & 63;
  st.wave = threadIdx.x >> 6;
  st.g = st.lane >> 4;
  st.lr = st.lane & 15;
  const int last_row = min(r0 + kQRows, nq) - 1;
  st.j_hi = (st.qs + last_row) >> 7;

  const float tq = p.q_tscale[b * p.h_q + h], tk = p.k_tscale[b * p.h_kv + st.hk];
  const int eqk = ilog2f(tq) + ilog2f(tk);
  st.lam2 = __builtin_ldexpf(p.lam, eqk);        // lambda * tQ * tK
  st.seed_scale = __builtin_ldexpf(1.0f, -eqk);  // Delta_S in accumulator units

  st.wrow0 = r0 + st.wave * (NB * 16);
  st.wave_active = st.wrow0 < nq;
  st.wpos_min = st.qs + st.wrow0;
  st.wpos_max = st.qs + min(st.wrow0 + NB * 16, nq) - 1;

  // ---- Q operands (B of S^T = K Q^T).  NVFP4: exact FP16, tensor scale
  // factored out.  MXFP4: the raw codes of channels 32g .. 32g+31 and their
  // E8M0 scale (the lane's 32-element block of the scaled FP4 MFMA).
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int row = st.wrow0 + nb * 16 + st.lr;
    st.pos[nb] = st.qs + row;
    const bool valid = row < nq;
    const int64_t tok = q0 + (valid ? row : 0);
    const uint8_t* qc = p.q_codes + (tok * p.h_q + h) * 64;
    const uint8_t* qsc = p.q_scales + (tok * p.h_q + h) * 8;
    if (MX) {
      st.qraw[nb] = valid ? *reinterpret_cast<const u32x4*>(qc + 16 * st.g) : (u32x4){0u, 0u, 0u, 0u};
      st.qscale[nb] = valid ? qsc[st.g] : 127;
    } else {
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const uint32_t cw = valid ? *reinterpret_cast<const uint32_t*>(qc + 16 * ks + 4 * st.g) : 0u;
        const uint32_t sc = valid ? qsc[2 * ks + (st.g >> 1)] : 0u;
        st.qop[nb][ks] = dequant8(cw, split_e4m3(sc));
      }
    }
  }
  st.bseed = (bf16x8){};
  if (st.lane < 16) st.bseed[0] = (__bf16)1.0f;
  return true;
}

// S^T = seed + K Q^T of the tile in sm (Algorithm 1, scores of one tile).
template <int SEED, bool MX, int PV, int NB = kNB>
__device__ __forceinline__ void qk_tile(f32x4 (&s)[8][NB], const PrefillSmemT<PV>& sm, const ItemState<NB>& st) {
  const int g = st.g, lr = st.lr;
  // rank-one seed operands: every lane reads the 8 values of its row lr;
  // only reduction slot 0 of lanes 0..15 meets a nonzero B element, so the
  // other (finite) values contribute exact zeros
  const u32x4 dsv = SEED == kSeedMfma ? *reinterpret_cast<const u32x4*>(&sm.dss[8 * lr])
                                      : (u32x4){0u, 0u, 0u, 0u};
#pragma unroll
  for (int mb = 0; mb < 8; ++mb) {
    f32x4 seed = (f32x4){0.f, 0.f, 0.f, 0.f};
    if (SEED == kSeedMfma) {
      const uint32_t w = dsv[mb >> 1];
      const u32x4 a = {(mb & 1) ? (w >> 16) : w, 0u, 0u, 0u};
      seed = mfma_bf16(__builtin_bit_cast(bf16x8, a), st.bseed, seed);
    } else if (SEED == kSeedInit) {
      // keys 32g + 4mb .. +3 of the lane's accumulator rows
      seed = *reinterpret_cast<const f32x4*>(&sm.ds[32 * g + 4 * mb]);
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) s[mb][nb] = seed;
  }
  if (MX) {
    // one scaled FP4 MFMA per 16x16 block covers all 128 channels
    const uint64_t ks8 = *reinterpret_cast<const uint64_t*>(sm.k + kMxScaleOff + (lr * 4 + g) * 8);
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const int krow = 32 * (lr >> 2) + 4 * mb + (lr & 3);
      const u32x4 kop = *reinterpret_cast<const u32x4*>(sm.k + krow * 64 + ((g ^ mx_swz(krow)) << 4));
      const int sk = (int)((ks8 >> (8 * mb)) & 0xFFu);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) s[mb][nb] = mfma_fp4(kop, st.qraw[nb], s[mb][nb], sk, st.qscale[nb]);
    }
  } else {
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
        for (int mb = 4 * half; mb < 4 * half + 4; ++mb) {
          const int krow = 32 * (lr >> 2) + 4 * mb + (lr & 3);
          const f16x8 kop = *reinterpret_cast<const f16x8*>(sm.k + krow * 256 + (((4 * ks + g) ^ lr) << 4));
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) s[mb][nb] = mfma_f16(kop, st.qop[nb][ks], s[mb][nb]);
        }
      }
  }
  if (SEED == kSeedElem) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) s[mb][nb] += *reinterpret_cast<const f32x4*>(&sm.ds[32 * g + 4 * mb]);
  }
}

// P operands of the PV product of one tile: FP8 words (kPvFp8) or eight
// BF16 / exact FP16 values per MFMA (kPvBf16, kPvNvfp4).
template <int NB = kNB>
struct PTile {
  i32x8 pb[NB];
  f16x8 ph[NB][4];   // keys 32g + 8kk .. +7
};

// Causal mask, online softmax and P quantization of one tile (Algorithm 1,
// softmax steps), with the rescale of O when a row maximum moved.
// ABL > 0 only in the characterization library (built with
// MPFA_ABLATION_BUILD), whose outputs are meaningless by design: the cost of
// a softmax stage is the time difference to the build without it (Sec. 3.2,
// Fig. 3c).  ABL 1: P = its exponent argument (no exp2); ABL 2: also no row
// maximum, row sum or O rescale.
template <int PV, int ABL = 0, int NB = kNB>
__device__ __forceinline__ void softmax_tile(f32x4 (&s)[8][NB], int key0, bool need_mask, const ItemState<NB>& st,
                                             float (&m)[NB], float (&l)[NB], f32x4 (&o)[8][NB], PTile<NB>& pt) {
  const int g = st.g;
  const float lam2 = st.lam2;
  if (need_mask) {
    // key 32g + 4mb + i of the tile lies after query position pos
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int lim = st.pos[nb] - key0 - 32 * g;
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * mb + i > lim) s[mb][nb][i] = -INFINITY;
        // keep each compare next to its select: scheduled as one batch, the
        // 64 compare masks exhaust the scalar registers
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  // log2 of the fixed factor the P quantizer applies: 448 (FP8), 1 (BF16),
  // 2688 = 6 * 448 (NVFP4: the largest P, 1, maps to the top E2M1 code
  // under the largest E4M3 scale)
  constexpr float kLog2PScale = PV == kPvFp8 ? kLog2_448 : (PV == kPvBf16 ? 0.0f : 11.392317422778760f);
  float alpha[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    // two independent chains of v_max3 (two new scores per instruction)
    float mxa = -INFINITY, mxb = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 8; mb += 2) {
      mxa = fmaxf(fmaxf(mxa, s[mb][nb][0]), s[mb][nb][1]);
      mxa = fmaxf(fmaxf(mxa, s[mb][nb][2]), s[mb][nb][3]);
      mxb = fmaxf(fmaxf(mxb, s[mb + 1][nb][0]), s[mb + 1][nb][1]);
      mxb = fmaxf(fmaxf(mxb, s[mb + 1][nb][2]), s[mb + 1][nb][3]);
    }
    const float mx = ABL >= 2 ? 0.0f : wave_max16(fmaxf(mxa, mxb));
    const float mnew = fmaxf(m[nb], mx);
    const float muse = (mnew == -INFINITY) ? 0.0f : mnew;
    alpha[nb] = (m[nb] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f((m[nb] - muse) * lam2);
    m[nb] = mnew;
    const float bias = ABL >= 2 ? kLog2PScale : __builtin_fmaf(-muse, lam2, kLog2PScale);
    float ps;
    float ev[8][4];
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      float e[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float arg = __builtin_fmaf(s[mb][nb][i], lam2, bias);
        e[i] = ABL >= 1 ? arg : __builtin_amdgcn_exp2f(arg);
      }
      if (ABL < 2) {
        const float q4 = (e[0] + e[1]) + (e[2] + e[3]);
        ps = mb == 0 ? q4 : ps + q4;
      }
      if (PV == kPvFp8) {
        pt.pb[nb][mb] = (int)pack_fp8x4(e[0], e[1], e[2], e[3]);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) ev[mb][i] = e[i];
      }
    }
    if (ABL < 2) l[nb] = alpha[nb] * l[nb] + ps;
    if (PV == kPvBf16) {
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        bf16x8 b;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          b[i] = (__bf16)ev[2 * kk][i];
          b[4 + i] = (__bf16)ev[2 * kk + 1][i];
        }
        pt.ph[nb][kk] = __builtin_bit_cast(f16x8, b);
      }
    } else if (PV == kPvNvfp4) {
      // the lane's 32 keys are two 16-key groups: keys 32g .. +15 (mb 0..3)
      // and 32g + 16 .. +31 (mb 4..7); scale E4M3(amax / 6), codes E2M1(P'/scale)
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        float amax = 0.0f;
#pragma unroll
        for (int mb = 4 * half; mb < 4 * half + 4; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) amax = fmaxf(amax, ev[mb][i]);
        const uint32_t sc = fp8_sat_pair(0u, div_by_scale(amax, 6.0f, kRcp6), 0.0f, false) & 0xFFu;
        const float sd = e4m3_value(sc);
        uint32_t cw[2] = {0u, 0u};
        if (sd > 0.0f) {
          const float r = __fdiv_rn(1.0f, sd);
#pragma unroll
          for (int w = 0; w < 2; ++w)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int mb = 4 * half + 2 * w + (j >> 1), i0 = 2 * (j & 1);
              cw[w] = fp4_pair(cw[w], div_by_scale(ev[mb][i0], sd, r), div_by_scale(ev[mb][i0 + 1], sd, r),
                               1.0f, j);
            }
        }
        const ScaleSplit sp = split_e4m3(sc);
        pt.ph[nb][2 * half] = dequant8(cw[0], sp);
        pt.ph[nb][2 * half + 1] = dequant8(cw[1], sp);
      }
    }
  }
  // rescale the O rows of a query block only when one of its maxima moved
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (ABL < 2 && __builtin_amdgcn_ballot_w64(alpha[nb] != 1.0f) != 0) {
#pragma unroll
      for (int db = 0; db < 8; ++db) o[db][nb] *= alpha[nb];
    }
  }
}

// O^T += V^T P^T with V of the tile in sm.
template <int PV, int NB = kNB>
__device__ __forceinline__ void pv_tile(const PrefillSmemT<PV>& sm, const PTile<NB>& pt, f32x4 (&o)[8][NB],
                                        const ItemState<NB>& st) {
  const int g = st.g, lr = st.lr;
  if (PV == kPvFp8) {
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
      for (int nb = 0; nb < NB; ++nb) o[db][nb] = mfma_fp8(vop, pt.pb[nb], o[db][nb]);
    }
  } else {
    // four 32-key MFMAs per channel block: MFMA kk reduces keys 32g + 8kk .. +7
    // of every lane group g, so A (V row chunk 4g + kk) and B (the lane's own
    // P values) pair the same keys
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      const uint8_t* vr = sm.v + (16 * db + lr) * (kTile * 2);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const u32x4 va = *reinterpret_cast<const u32x4*>(vr + (((4 * g + kk) ^ lr) << 4));
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          if (PV == kPvBf16)
            o[db][nb] = mfma_bf16(__builtin_bit_cast(bf16x8, va), __builtin_bit_cast(bf16x8, pt.ph[nb][kk]),
                                  o[db][nb]);
          else
            o[db][nb] = mfma_f16(__builtin_bit_cast(f16x8, va), pt.ph[nb][kk], o[db][nb]);
        }
      }
    }
  }
}

// out = O / (448 l) as BF16 (for the other PV precisions the factor is the
// one their P carries).
template <int NB = kNB>
__device__ __forceinline__ void store_output(const PrefillParams& p, const ItemState<NB>& st, const float (&l)[NB],
                                             const f32x4 (&o)[8][NB]) {
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const float lt = wave_sum16(l[nb]);
    const int row = st.wrow0 + nb * 16 + st.lr;
    if (row < st.nq) {
      uint16_t* dst = p.out + ((int64_t)(st.q0 + row) * p.h_q + st.h) * kD;
      const float inv = __frcp_rn(lt);
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const uint32_t lo = (uint32_t)bf16_rne(o[db][nb][0] * inv) |
                            ((uint32_t)bf16_rne(o[db][nb][1] * inv) << 16);
        const uint32_t hi = (uint32_t)bf16_rne(o[db][nb][2] * inv) |
                            ((uint32_t)bf16_rne(o[db][nb][3] * inv) << 16);
        *reinterpret_cast<uint2*>(dst + 16 * db + 4 * st.g) = make_uint2(lo, hi);
      }
    }
  }
}

// One prefill work item (query head, 256-row query tile) executed by a whole
// workgroup of kThreads threads; `bid` is the item's position in the dispatch
// order (largest tiles first) and smem two tile buffers in LDS.  Every wave
// runs QK, softmax and PV of a tile back to back; the next tile is fetched
// into registers meanwhile (two tiles ahead for MXFP4) and stored to the other
// buffer at the end.
template <int SEED, bool MX, int PV, int ABL = 0>
__device__ __forceinline__ void prefill_item(const PrefillParams& p, int bid, PrefillSmemT<PV>* smem) {
  ItemState<> st;
  if (!item_setup<MX>(p, bid, st)) return;

  float m[kNB], l[kNB];
  f32x4 o[8][kNB];
#pragma unroll
  for (int nb = 0; nb < kNB; ++nb) {
    m[nb] = -INFINITY;
    l[nb] = 0.0f;
#pragma unroll
    for (int db = 0; db < 8; ++db) o[db][nb] = (f32x4){0.f, 0.f, 0.f, 0.f};
  }

  const int32_t* pt = p.page_table + (int64_t)st.b * p.max_pages;
  {
    TileRegs<PV> r0r;
    fetch_tile<MX, PV>(r0r, p, pt, st.hk, st.h, st.j_hi, st.kvl, threadIdx.x);
    store_tile<MX, PV>(smem[st.j_hi & 1], r0r, st.seed_scale, threadIdx.x);
  }
  if constexpr (MX && SEED != kSeedElem) {
    // MXFP4 keeps two fetched tiles in registers (its register budget allows
    // it, except with the element-wise compensation): tile j-2 is loaded during step j and stored at the end of step j-1,
    // so its loads have two steps to arrive.  The loop is unrolled twice so the
    // two register sets keep fixed names.
    TileRegs<PV> ra, rb;
    if (st.j_hi >= 1) fetch_tile<MX, PV>(ra, p, pt, st.hk, st.h, st.j_hi - 1, st.kvl, threadIdx.x);
    __syncthreads();
    auto step = [&](int j, const TileRegs<PV>& held, TileRegs<PV>& fresh) {
      if (j >= 2) fetch_tile<MX, PV>(fresh, p, pt, st.hk, st.h, j - 2, st.kvl, threadIdx.x);
      const PrefillSmemT<PV>& sm = smem[j & 1];
      const int key0 = j * kTile;
      if (st.wave_active && key0 <= st.wpos_max) {
        f32x4 s[8][kNB];
        qk_tile<SEED, MX, PV>(s, sm, st);
        PTile<> ptile;
        softmax_tile<PV, ABL>(s, key0, key0 + kTile - 1 > st.wpos_min, st, m, l, o, ptile);
        pv_tile<PV>(sm, ptile, o, st);
      }
      if (j >= 1) store_tile<MX, PV>(smem[(j - 1) & 1], held, st.seed_scale, threadIdx.x);
      __syncthreads();
    };
    int j = st.j_hi;
    for (; j >= 1; j -= 2) {
      step(j, ra, rb);
      step(j - 1, rb, ra);
    }
    if (j == 0) step(0, ra, rb);
    if (!st.wave_active) return;
    store_output(p, st, l, o);
    return;
  }
  __syncthreads();
  for (int j = st.j_hi; j >= 0; --j) {
    TileRegs<PV> nxt;
    if (j > 0) fetch_tile<MX, PV>(nxt, p, pt, st.hk, st.h, j - 1, st.kvl, threadIdx.x);
    const PrefillSmemT<PV>& sm = smem[j & 1];
    const int key0 = j * kTile;
    if (st.wave_active && key0 <= st.wpos_max) {
      f32x4 s[8][kNB];
      qk_tile<SEED, MX, PV>(s, sm, st);
      PTile<> ptile;
      softmax_tile<PV, ABL>(s, key0, key0 + kTile - 1 > st.wpos_min, st, m, l, o, ptile);
      pv_tile<PV>(sm, ptile, o, st);
    }
    if (j > 0) store_tile<MX, PV>(smem[(j - 1) & 1], nxt, st.seed_scale, threadIdx.x);
    __syncthreads();
  }

  if (!st.wave_active) return;
  store_output(p, st, l, o);
}

}  // namespace

}  // namespace mpfa
