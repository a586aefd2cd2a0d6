// decode_body.h -- the split-KV decode work item (Sec. 5.3) and the partition
// merge as device functions, shared by the decode kernels and the fused
// mixed-step kernel.
#pragma once
#include "mpfa_device.h"
#include "mpfa_internal.h"

namespace mpfa {

namespace {

constexpr int kWavesPerBlock = 4;

// Per wave, tile j (last to first): PV of tile j+1 (V and P in registers);
// loads of V tile j; QK of tile j (K codes prefetched in registers); loads of
// tile j-1's K codes, scales and compensation; online softmax of tile j.  The
// V loads land directly in the PV operand registers: lane l holds channel
// 16 db + l%16, keys 32 (l/16) + 16 hf .. +15 in va[db] (hf 0) and vb[db]
// (hf 1).  Every load goes to registers (none to LDS), so the compiler counts
// each wait: PV of tile j+1 waits for V(j+1) with K(j) still in flight, QK of
// tile j for K(j) with V(j) in flight.

// Merge of the partition states of query head h of sequence b by one wave:
// lane l owns channels l and l + 64.  Per channel: the maximum of m over the
// partitions, then L and O accumulated over the partitions in order, O / L
// rounded to BF16.  The loads of 16 partitions are issued together.
__device__ __forceinline__ void merge_head(const DecodeParams& p, int b, int h, int np) {
  constexpr int kBatch = 16;
  const int lane = threadIdx.x & 63;
  const float* st = p.ws + ((int64_t)b * p.h_q + h) * p.max_partitions * (kD + 2);
  float M = -INFINITY;
  for (int q0 = 0; q0 < np; q0 += kBatch) {
    float mv[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) mv[j] = q0 + j < np ? st[(q0 + j) * (kD + 2)] : -INFINITY;
#pragma unroll
    for (int j = 0; j < kBatch; ++j) M = fmaxf(M, mv[j]);
  }
  float L = 0.0f, O0 = 0.0f, O1 = 0.0f;
  for (int q0 = 0; q0 < np; q0 += kBatch) {
    float mv[kBatch], lv[kBatch], o0[kBatch], o1[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const bool in = q0 + j < np;
      const float* sq = st + (q0 + j) * (kD + 2);
      mv[j] = in ? sq[0] : 0.0f;
      lv[j] = in ? sq[1] : 0.0f;
      o0[j] = in ? sq[2 + lane] : 0.0f;
      o1[j] = in ? sq[2 + 64 + lane] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (q0 + j < np) {
        const float f = __builtin_amdgcn_exp2f(mv[j] - M);
        L = __builtin_fmaf(f, lv[j], L);
        O0 = __builtin_fmaf(f, o0[j], O0);
        O1 = __builtin_fmaf(f, o1[j], O1);
      }
    }
  }
  uint16_t* o = p.out + ((int64_t)b * p.h_q + h) * kD;
  o[lane] = bf16_rne(np > 0 ? __fdiv_rn(O0, L) : 0.0f);
  o[64 + lane] = bf16_rne(np > 0 ? __fdiv_rn(O1, L) : 0.0f);
}

// One decode work item (sequence b, KV head hk, partition part) executed by
// one wave; it writes the partition state to the workspace.  With FUSED, the
// wave then counts itself in counters[b * h_kv + hk] (device scope); the wave
// that completes the last partition of (b, hk) merges the group's query heads,
// writes the outputs and resets the counter to zero for the next call.
template <bool SMOOTH, bool MX, bool FUSED>
__device__ __forceinline__ void decode_partition(const DecodeParams& p, int b, int hk, int part,
                                                 uint32_t* counters) {
  // the item indices are wave-uniform: in scalar registers, the tile loop and
  // its branches are scalar too
  b = __builtin_amdgcn_readfirstlane(b);
  hk = __builtin_amdgcn_readfirstlane(hk);
  part = __builtin_amdgcn_readfirstlane(part);
  const int lane = threadIdx.x & 63, g = lane >> 4, lr = lane & 15;
  const int kvl = p.kv_len[b];
  const int np = (kvl + p.partition_tokens - 1) / p.partition_tokens;
  if (part >= np) return;
  const int grp = p.h_q / p.h_kv;
  const int kbeg = part * p.partition_tokens;
  const int kend = min(kbeg + p.partition_tokens, kvl);
  const bool qvalid = lr < grp;
  const int h = hk * grp + (qvalid ? lr : 0);
  const int32_t* pt = p.page_table + (int64_t)b * p.max_pages;
  const int npg = (kvl + 63) >> 6;

  const int ek = ilog2f(p.k_tscale[b * p.h_kv + hk]);
  const int eqk = ilog2f(p.q_tscale[b * p.h_q + h]) + ek;
  const float lam2 = __builtin_ldexpf(p.lam, eqk);           // per query head (column lr)
  const float seed_scale = __builtin_ldexpf(1.0f, -eqk);     // Delta_S in accumulator units

  // Q operand: column lr = query head hk*G + lr; channels 32g .. 32g+31 (NVFP4:
  // dequantized to FP16 in four 8-channel slices; MXFP4: the raw codes)
  f16x8 qop[4];
  u32x4 qraw;
  int qscale = 0;
  {
    const uint8_t* qc = p.q_codes + ((int64_t)b * p.h_q + h) * 64;
    const uint8_t* qsc = p.q_scales + ((int64_t)b * p.h_q + h) * 8;
    const u32x4 cw = qvalid ? *reinterpret_cast<const u32x4*>(qc + 16 * g) : (u32x4){0u, 0u, 0u, 0u};
    if (MX) {
      qraw = cw;
      qscale = qvalid ? qsc[g] : 127;
    } else {
      const uint32_t sc = qvalid ? *reinterpret_cast<const uint16_t*>(qsc + 2 * g) : 0u;
      const ScaleSplit s0 = split_e4m3(sc & 0xFFu), s1 = split_e4m3((sc >> 8) & 0xFFu);
      qop[0] = dequant8(cw[0], s0);
      qop[1] = dequant8(cw[1], s0);
      qop[2] = dequant8(cw[2], s1);
      qop[3] = dequant8(cw[3], s1);
    }
  }

  const int j_lo_ = kbeg / kTile, j_hi_ = (kend - 1) / kTile;
  const int krow_in_tile = 32 * (lr >> 2) + (lr & 3);   // + 4 mb: key of MFMA row lr
  const int64_t page_k_rows = (int64_t)p.h_kv * kPage;   // K rows per page
  const int64_t kv_head = (int64_t)hk * kPage;

  // ---- K-side loads of one tile (registers).  Every address stays inside a
  // mapped page (page index clamped to the sequence's last page), so the loads
  // are unconditional; keys at or past the partition end are masked to -inf
  // after QK, which also discards whatever those cache slots hold.
  u32x4 kc[8];
  uint32_t ksc[8];
  uint2 dsw[8];
  // Page indices: 64 consecutive entries of the page table in one register
  // (lane i holds entry base + i), read per tile with v_readlane into scalar
  // registers.  The tile loop then issues no page-table loads, whose results
  // (needed by the next addresses and retiring after every K and V load issued
  // before them) would drain the loads in flight.  The window is loaded below
  // the current pages, so a partition of up to 4096 tokens needs one load.
  int win = 0, win_base = 0;
  auto load_window = [&](int lo, int hi) {   // pages lo .. hi (even lo)
    win_base = max(lo, hi - 63) & ~1;
    win = pt[min(win_base + lane, npg - 1)];
  };
  // The two pages of tile j: keys 0..63 and 64..127.  A lane's K rows lie in
  // page lr / 8 of the tile (MFMA rows 0..7 hold keys 0..63), its V and
  // Delta_S bytes in page g / 2.
  auto tile_pages = [&](int j, int& q0, int& q1) {
    if (2 * j < win_base) {   // next window (partitions above 4096 tokens)
      load_window(2 * j_lo_, 2 * j + 1);
      __builtin_amdgcn_s_waitcnt(0);   // here, so the common path holds no pending window load
    }
    q0 = __builtin_amdgcn_readlane(win, 2 * j - win_base);
    q1 = __builtin_amdgcn_readlane(win, 2 * j + 1 - win_base);
  };
  // With live false (past the partition's first tile) every lane reads row 0
  // of its page instead: the loads stay unconditional, so they can issue
  // between the QK products that free their registers, and cost one cache line.
  auto load_k = [&](int64_t kpage, int64_t dpage, bool live) {
    const int rmask = live ? 63 : 0;
    // compensation of the lane's accumulator rows: keys 32g + 4mb .. +3, head
    // lr; issued first, as the first QK product starts from it
    if (SMOOTH) {
      const uint16_t* dsp = p.ds + (dpage * p.h_q + h) * kPage + ((32 * g) & rmask);
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) dsw[mb] = *reinterpret_cast<const uint2*>(dsp + 4 * mb);
    } else {
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) dsw[mb] = make_uint2(0u, 0u);
    }
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const int64_t row = kpage * page_k_rows + kv_head + ((krow_in_tile + 4 * mb) & rmask);
      ksc[mb] = MX ? (uint32_t)p.k_scales[row * 8 + g]
                   : (uint32_t)*reinterpret_cast<const uint16_t*>(p.k_scales + row * 8 + 2 * g);
      kc[mb] = *reinterpret_cast<const u32x4*>(p.k_codes + row * 64 + 16 * g);
    }
  };
  // ---- V tile j: 16 loads of 16 bytes per lane, straight into the PV
  // operand registers (channel 16 db + lr, keys 32 g + 16 hf .. +15)
  u32x4 va[8], vb[8];
  auto load_v = [&](int64_t vpage) {
    const uint8_t* vsrc = p.v_codes + ((vpage * p.h_kv + hk) * kD + lr) * kPage + ((32 * g) & 63);
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      va[db] = *reinterpret_cast<const u32x4*>(vsrc + db * 16 * kPage);
      vb[db] = *reinterpret_cast<const u32x4*>(vsrc + db * 16 * kPage + 16);
    }
  };

  float m = -INFINITY, l = 0.0f;
  f32x4 o[8];
#pragma unroll
  for (int db = 0; db < 8; ++db) o[db] = (f32x4){0.f, 0.f, 0.f, 0.f};
  i32x8 pb = {};

  // O^T += V^T P^T for tile t (P in pb, V in the LDS slab).  Keys past the end
  // of the sequence carry P = 0, but their V bytes may be stale cache contents:
  // they are cleared so that 0 * NaN cannot occur.
  auto pv = [&](int t) {
    if (t * kTile + kTile > kend) {   // uniform: the partition's last keys
      const int nv = kend - (t * kTile + 32 * g);
      uint32_t ma[4], mb2[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k1 = nv - 4 * i, k2 = nv - 16 - 4 * i;
        ma[i] = k1 >= 4 ? 0xFFFFFFFFu : (k1 <= 0 ? 0u : ((1u << (8 * k1)) - 1u));
        mb2[i] = k2 >= 4 ? 0xFFFFFFFFu : (k2 <= 0 ? 0u : ((1u << (8 * k2)) - 1u));
      }
#pragma unroll
      for (int db = 0; db < 8; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          va[db][i] &= ma[i];
          vb[db][i] &= mb2[i];
        }
    }
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      const i32x8 vop = {(int)va[db][0], (int)va[db][1], (int)va[db][2], (int)va[db][3],
                         (int)vb[db][0], (int)vb[db][1], (int)vb[db][2], (int)vb[db][3]};
      o[db] = mfma_fp8(vop, pb, o[db]);
    }
  };

  const int j_lo = j_lo_, j_hi = j_hi_;
  int c0, c1, n0, n1;   // pages of tile j, of tile j - 1
  load_window(2 * j_lo, 2 * j_hi + 1);
  tile_pages(j_hi, c0, c1);
  load_k((lr >> 3) ? c1 : c0, (g >> 1) ? c1 : c0, true);
  tile_pages(max(j_hi - 1, j_lo), n0, n1);
  for (int j = j_hi; j >= j_lo; --j) {
    const int key0 = j * kTile;
    if (j < j_hi) pv(j + 1);
    load_v((g >> 1) ? c1 : c0);
    // V(j) is issued before the QK waits for K(j): those waits then leave the
    // V loads in flight
    __builtin_amdgcn_sched_barrier(0);
    // ---- S^T = 1 Delta_S^T + K Q^T (the rank-G term as accumulator input)
    f32x4 s[8];
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      f32x4 c = (f32x4){__uint_as_float(dsw[mb].x << 16), __uint_as_float(dsw[mb].x & 0xFFFF0000u),
                        __uint_as_float(dsw[mb].y << 16), __uint_as_float(dsw[mb].y & 0xFFFF0000u)};
      c *= seed_scale;   // exact: power of two
      if (MX) {
        s[mb] = mfma_fp4(kc[mb], qraw, c, (int)ksc[mb], qscale);
      } else {
        const ScaleSplit s0 = split_e4m3(ksc[mb] & 0xFFu), s1 = split_e4m3((ksc[mb] >> 8) & 0xFFu);
        c = mfma_f16(dequant8(kc[mb][0], s0), qop[0], c);
        c = mfma_f16(dequant8(kc[mb][1], s0), qop[1], c);
        c = mfma_f16(dequant8(kc[mb][2], s1), qop[2], c);
        s[mb] = mfma_f16(dequant8(kc[mb][3], s1), qop[3], c);
      }
    }
    load_k((lr >> 3) ? n1 : n0, (g >> 1) ? n1 : n0, j > j_lo);
    c0 = n0;
    c1 = n1;
    tile_pages(max(j - 2, j_lo), n0, n1);
    if (key0 + kTile > kend) {
#pragma unroll
      for (int mb = 0; mb < 8; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (key0 + 32 * g + 4 * mb + i >= kend) s[mb][i] = -INFINITY;
    }
    // ---- online softmax (rows = query heads), P to FP8 (x448)
    // two independent chains of v_max3 (two new scores per instruction)
    float mxa = -INFINITY, mxb = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 8; mb += 2) {
      mxa = fmaxf(fmaxf(mxa, s[mb][0]), s[mb][1]);
      mxa = fmaxf(fmaxf(mxa, s[mb][2]), s[mb][3]);
      mxb = fmaxf(fmaxf(mxb, s[mb + 1][0]), s[mb + 1][1]);
      mxb = fmaxf(fmaxf(mxb, s[mb + 1][2]), s[mb + 1][3]);
    }
    const float mx = wave_max16(fmaxf(mxa, mxb));
    const float mnew = fmaxf(m, mx);
    const float muse = (mnew == -INFINITY) ? 0.0f : mnew;
    const float alpha = (m == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f((m - muse) * lam2);
    m = mnew;
    const float bias = __builtin_fmaf(-muse, lam2, kLog2_448);
    float ps = 0.0f;
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      float e[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) e[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[mb][i], lam2, bias));
      ps += (e[0] + e[1]) + (e[2] + e[3]);
      pb[mb] = (int)pack_fp8x4(e[0], e[1], e[2], e[3]);
    }
    l = alpha * l + ps;
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f) != 0) {
#pragma unroll
      for (int db = 0; db < 8; ++db) o[db] *= alpha;
    }
  }
  pv(j_lo);
  // The scaled FP8 MFMA may otherwise be sunk into the branch below, where
  // lanes of the invalid query-head columns are switched off; the MFMA then
  // reads their (inactive) operand rows as zero.  An empty asm that consumes
  // the accumulators keeps the products in full-wave control flow.
#pragma unroll
  for (int db = 0; db < 8; ++db) asm volatile("" : "+v"(o[db]));

  // partition state: m in log2 units (m * lambda'), l, O[128]
  const float lt = wave_sum16(l);
  if (qvalid) {
    float* st = p.ws + (((int64_t)b * p.h_q + h) * p.max_partitions + part) * (kD + 2);
    if (g == 0) {
      st[0] = m * lam2;
      st[1] = lt;
    }
#pragma unroll
    for (int db = 0; db < 8; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) st[2 + 16 * db + 4 * g + i] = o[db][i];
  }
  if (FUSED) {
    // release: this partition's state is visible device-wide before it is counted
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    uint32_t prev = 0;
    if (lane == 0) prev = atomicAdd(&counters[b * p.h_kv + hk], 1u);
    prev = __shfl(prev, 0);
    if (prev == (uint32_t)(np - 1)) {   // last partition of (b, hk): merge its query heads
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");   // every state counted before is visible
      for (int j = 0; j < grp; ++j) merge_head(p, b, hk * grp + j, np);
      if (lane == 0) atomicExch(&counters[b * p.h_kv + hk], 0u);
    }
  }
}

}  // namespace

}  // namespace mpfa
