// decode_body.h -- the split-KV decode work item (Sec. 5.3) and the partition
// merge as device functions, shared by the decode kernels and the fused
// mixed-step kernel.
#pragma once
#include "mpfa_device.h"
#include "mpfa_internal.h"

namespace mpfa {

namespace {

constexpr int kWavesPerBlock = 4;
constexpr int kVBytes = kD * kTile;   // one FP8 V tile per wave in LDS (16 KB)

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(1))) void* global_ptr_t;

// Software pipeline per wave, iteration j (tiles last to first):
//   wait for every outstanding load;  PV of tile j+1 (V from LDS, P from
//   registers);  direct global->LDS loads of V tile j;  QK of tile j (K codes
//   prefetched in registers);  prefetch of tile j-1's K codes, scales and
//   compensation;  online softmax of tile j.
// V never occupies registers (it is read from LDS as MFMA operands), which
// keeps the wave under the register budget of two waves per SIMD.
// LDS V layout: for channel block db and half hf, the 1 KB slab at
// (2 db + hf) KB holds, at 16 * lane, the bytes the lane feeds to the MFMA:
// channel 16 db + lane%16, keys 32 (lane/16) + 16 hf .. +15.
// Merge of the partition states of one (sequence, query head) for output
// channel d: log-sum-exp over the partitions in order, then O / L, BF16.
// The loads of 16 partitions are issued together; the accumulation order stays
// partition 0, 1, 2, ...
__device__ __forceinline__ float merge_channel(const DecodeParams& p, int b, int h, int d, int np) {
  constexpr int kBatch = 16;
  const float* st = p.ws + ((int64_t)b * p.h_q + h) * p.max_partitions * (kD + 2);
  float M = -INFINITY;
  for (int q0 = 0; q0 < np; q0 += kBatch) {
    float mv[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) mv[j] = q0 + j < np ? st[(q0 + j) * (kD + 2)] : -INFINITY;
#pragma unroll
    for (int j = 0; j < kBatch; ++j) M = fmaxf(M, mv[j]);
  }
  float L = 0.0f, O = 0.0f;
  for (int q0 = 0; q0 < np; q0 += kBatch) {
    float mv[kBatch], lv[kBatch], ov[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const bool in = q0 + j < np;
      const float* sq = st + (q0 + j) * (kD + 2);
      mv[j] = in ? sq[0] : 0.0f;
      lv[j] = in ? sq[1] : 0.0f;
      ov[j] = in ? sq[2 + d] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (q0 + j < np) {
        const float f = __builtin_amdgcn_exp2f(mv[j] - M);
        L = __builtin_fmaf(f, lv[j], L);
        O = __builtin_fmaf(f, ov[j], O);
      }
    }
  }
  return np > 0 ? __fdiv_rn(O, L) : 0.0f;
}

// One decode work item (sequence b, KV head hk, partition part) executed by
// one wave with the 16 KB LDS slab vbuf.  With FUSED, the wave that completes
// the last partition of (b, hk) also merges the group's query heads: each wave
// publishes its state, then counts itself in counters[b * h_kv + hk] (device
// scope); the last arrival reads all states, writes the outputs and resets the
// counter to zero for the next call.
template <bool SMOOTH, bool MX, bool FUSED>
__device__ __forceinline__ void decode_partition(const DecodeParams& p, int b, int hk, int part, uint8_t* vbuf,
                                                 uint32_t* counters) {
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
  // The pages of tile j that the lane reads: its K rows' page (MFMA rows 0..7
  // hold keys 0..63) and its V / Delta_S page (lane groups 0, 1: keys 0..63).
  // They are loaded one tile ahead of their use, so no address computation
  // waits on a page-table load (a dependent load would drain every load the
  // wave has in flight); as per-lane values they stay in vector registers.
  auto tile_pages = [&](int j, int& kp, int& vp) {
    kp = pt[min(2 * j + (lr >> 3), npg - 1)];
    vp = pt[min(2 * j + (g >> 1), npg - 1)];
  };
  auto load_k = [&](int64_t kpage, int64_t dpage) {
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const int64_t row = kpage * page_k_rows + kv_head + ((krow_in_tile + 4 * mb) & 63);
      kc[mb] = *reinterpret_cast<const u32x4*>(p.k_codes + row * 64 + 16 * g);
      ksc[mb] = MX ? (uint32_t)p.k_scales[row * 8 + g]
                   : (uint32_t)*reinterpret_cast<const uint16_t*>(p.k_scales + row * 8 + 2 * g);
    }
    // compensation of the lane's accumulator rows: keys 32g + 4mb .. +3, head lr
    if (SMOOTH) {
      const uint16_t* dsp = p.ds + (dpage * p.h_q + h) * kPage + ((32 * g) & 63);
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) dsw[mb] = *reinterpret_cast<const uint2*>(dsp + 4 * mb);
    } else {
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) dsw[mb] = make_uint2(0u, 0u);
    }
  };
  // ---- V tile j: 16 direct global->LDS loads of 16 bytes per lane
  auto load_v = [&](int64_t vpage) {
    const uint8_t* vsrc = p.v_codes + ((vpage * p.h_kv + hk) * kD + lr) * kPage + ((32 * g) & 63);
#pragma unroll
    for (int db = 0; db < 8; ++db)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
        __builtin_amdgcn_global_load_lds((global_ptr_t)(vsrc + db * 16 * kPage + 16 * hf),
                                         (lds_ptr_t)(vbuf + (2 * db + hf) * 1024), 16, 0, 0);
  };

  float m = -INFINITY, l = 0.0f;
  f32x4 o[8];
#pragma unroll
  for (int db = 0; db < 8; ++db) o[db] = (f32x4){0.f, 0.f, 0.f, 0.f};
  i32x8 pb = {};
  int pv_tile = -1;      // tile whose P (pb) awaits its PV product

  // O^T += V^T P^T for tile pv_tile.  Keys past the end of the sequence carry
  // P = 0, but their V bytes may be stale cache contents: they are cleared so
  // that 0 * NaN cannot occur.
  auto pv = [&]() {
    u32x4 va[8], vb[8];
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      va[db] = *reinterpret_cast<const u32x4*>(vbuf + (2 * db) * 1024 + 16 * lane);
      vb[db] = *reinterpret_cast<const u32x4*>(vbuf + (2 * db + 1) * 1024 + 16 * lane);
    }
    if (pv_tile * kTile + kTile > kend) {   // uniform: the partition's last keys
      const int nv = kend - (pv_tile * kTile + 32 * g);
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

  const int j_lo = kbeg / kTile, j_hi = (kend - 1) / kTile;
  int cur_k, cur_v, nxt_k = 0, nxt_v = 0;   // the lane's pages of tile j, of tile j - 1
  tile_pages(j_hi, cur_k, cur_v);
  load_k(cur_k, cur_v);
  tile_pages(max(j_hi - 1, j_lo), nxt_k, nxt_v);
  for (int j = j_hi; j >= j_lo; --j) {
    const int key0 = j * kTile;
    __builtin_amdgcn_s_waitcnt(0);   // K(j) in registers, V(j+1) in LDS
    if (pv_tile >= 0) pv();
    // the LDS reads of PV(j+1) must be complete before V(j) overwrites them
    __builtin_amdgcn_s_waitcnt(0);
    load_v(cur_v);
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
    if (j > j_lo) load_k(nxt_k, nxt_v);
    // outside the branch: copying a page index inside it would make the
    // compiler wait for the K loads at the join
    cur_k = nxt_k;
    cur_v = nxt_v;
    tile_pages(max(j - 2, j_lo), nxt_k, nxt_v);
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
    pv_tile = j;
  }
  __builtin_amdgcn_s_waitcnt(0);
  pv();
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
    __threadfence();   // this partition's state is visible device-wide before it is counted
    uint32_t prev = 0;
    if (lane == 0) prev = atomicAdd(&counters[b * p.h_kv + hk], 1u);
    prev = __shfl(prev, 0);
    if (prev == (uint32_t)(np - 1)) {   // last partition of (b, hk): merge its query heads
      __threadfence();
      for (int j = 0; j < grp; ++j) {
        const int hq = hk * grp + j;
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const int d = lane + 64 * c;
          p.out[((int64_t)b * p.h_q + hq) * kD + d] = bf16_rne(merge_channel(p, b, hq, d, np));
        }
      }
      if (lane == 0) atomicExch(&counters[b * p.h_kv + hk], 0u);
    }
  }
}

}  // namespace

}  // namespace mpfa
