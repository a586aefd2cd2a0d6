// decode.hip -- split-KV QK4PV8 decode over the paged cache for gfx950
// (Sec. 5.3), plus the log-sum-exp merge of the partition states.
//
// One wave = one (sequence, KV head, partition).  The G = H_q / H_kv query
// heads of the KV head are packed into the 16-wide MFMA column dimension
// (GQA packing); the compensation becomes a rank-G seed: A holds the G
// Delta_S values of each key, B is a G x G identity.  K and V stream straight
// from HBM into registers (no LDS): each lane loads 16 contiguous bytes of
// NVFP4 codes per key it owns and 32 contiguous FP8 bytes of the channel-major
// V page, dequantizes K exactly to FP16 and runs the same S^T = K Q^T /
// O^T = V^T P^T MFMA chain as prefill.  The reduction (head) dimension is
// permuted (lane group g, step ks, element e -> channel 32g + 8ks + e) so that
// every lane's code bytes are contiguous; Q uses the same permutation.
#include "mpfa_device.h"
#include "mpfa_internal.h"

namespace mpfa {

namespace {

constexpr int kWavesPerBlock = 4;

__global__ __launch_bounds__(kWavesPerBlock * 64) void decode_kernel(DecodeParams p) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, g = lane >> 4, lr = lane & 15;
  const int part = blockIdx.x * kWavesPerBlock + wave;
  const int hk = blockIdx.y, b = blockIdx.z;
  const int kvl = p.kv_len[b];
  const int np = (kvl + p.partition_tokens - 1) / p.partition_tokens;
  if (part >= np) return;
  const int grp = p.h_q / p.h_kv;
  const int kbeg = part * p.partition_tokens;
  const int kend = min(kbeg + p.partition_tokens, kvl);
  const bool qvalid = lr < grp;
  const int h = hk * grp + (qvalid ? lr : 0);
  const int32_t* pt = p.page_table + (int64_t)b * p.max_pages;

  const float tk = p.k_tscale[b * p.h_kv + hk];
  const int ek = ilog2f(tk);
  const float tq = p.q_tscale[b * p.h_q + h];
  const int eqk = ilog2f(tq) + ek;
  const float lam2 = __builtin_ldexpf(p.lam, eqk);   // per query head (column lr)

  // Q operand: column lr = query head hk*G + lr; channels 32g + 8ks + e
  f16x8 qop[4];
  {
    const uint8_t* qc = p.q_codes + ((int64_t)b * p.h_q + h) * 64;
    const uint8_t* qsc = p.q_scales + ((int64_t)b * p.h_q + h) * 8;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const uint32_t cw = qvalid ? *reinterpret_cast<const uint32_t*>(qc + 16 * g + 4 * ks) : 0u;
      const uint32_t sc = qvalid ? qsc[2 * g + (ks >> 1)] : 0u;
      qop[ks] = dequant8(cw, split_e4m3(sc));
    }
  }
  // seed operands: lanes 0..15 carry reduction index e = query head slot
  bf16x8 bseed = {};
  if (lane < 16 && lane < grp) bseed[lane & 7] = (__bf16)1.0f;
  float seed_scale[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    seed_scale[e] = 0.0f;
    if (e < grp) {
      const float tqe = p.q_tscale[b * p.h_q + hk * grp + e];
      seed_scale[e] = __builtin_ldexpf(1.0f, -(ilog2f(tqe) + ek));
    }
  }

  float m = -INFINITY, l = 0.0f;
  f32x4 o[8];
#pragma unroll
  for (int db = 0; db < 8; ++db) o[db] = (f32x4){0.f, 0.f, 0.f, 0.f};

  const int j_lo = kbeg / kTile, j_hi = (kend - 1) / kTile;
  for (int j = j_hi; j >= j_lo; --j) {
    const int key0 = j * kTile;
    f32x4 s[8];
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const int kabs = key0 + 32 * (lr >> 2) + 4 * mb + (lr & 3);
      u32x4 codes = {0u, 0u, 0u, 0u};
      uint32_t sc = 0;
      int64_t page = 0;
      const bool kin = kabs < kend;
      if (kin) {
        page = pt[kabs >> 6];
        const int64_t row = (page * p.h_kv + hk) * kPage + (kabs & 63);
        codes = *reinterpret_cast<const u32x4*>(p.k_codes + row * 64 + 16 * g);
        sc = *reinterpret_cast<const uint16_t*>(p.k_scales + row * 8 + 2 * g);
      }
      if (p.smooth) {
        bf16x8 aseed = {};
        if (lane < 16 && kin) {
          const uint16_t* dsp = p.ds + (page * p.h_q + hk * grp) * kPage + (kabs & 63);
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e < grp)
              aseed[e] = __builtin_bit_cast(__bf16, bf16_rne(bf16_to_f32(dsp[e * kPage]) * seed_scale[e]));
        }
        s[mb] = mfma_bf16(aseed, bseed, (f32x4){0.f, 0.f, 0.f, 0.f});
      } else {
        s[mb] = (f32x4){0.f, 0.f, 0.f, 0.f};
      }
      const ScaleSplit s0 = split_e4m3(sc & 0xFFu), s1 = split_e4m3((sc >> 8) & 0xFFu);
      s[mb] = mfma_f16(dequant8(codes[0], s0), qop[0], s[mb]);
      s[mb] = mfma_f16(dequant8(codes[1], s0), qop[1], s[mb]);
      s[mb] = mfma_f16(dequant8(codes[2], s1), qop[2], s[mb]);
      s[mb] = mfma_f16(dequant8(codes[3], s1), qop[3], s[mb]);
    }
    if (key0 + kTile > kend) {
#pragma unroll
      for (int mb = 0; mb < 8; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (key0 + 32 * g + 4 * mb + i >= kend) s[mb][i] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int mb = 0; mb < 8; ++mb)
      mx = fmaxf(fmaxf(mx, fmaxf(s[mb][0], s[mb][1])), fmaxf(s[mb][2], s[mb][3]));
    mx = wave_max16(mx);
    const float mnew = fmaxf(m, mx);
    const float muse = (mnew == -INFINITY) ? 0.0f : mnew;
    const float alpha = (m == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f((m - muse) * lam2);
    m = mnew;
    i32x8 pb;
    float ps = 0.0f;
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      float e[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) e[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[mb][i] - muse, lam2, kLog2_448));
      ps += (e[0] + e[1]) + (e[2] + e[3]);
      pb[mb] = (int)pack_fp8x4(e[0], e[1], e[2], e[3]);
    }
    l = alpha * l + ps;
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f) != 0) {
#pragma unroll
      for (int db = 0; db < 8; ++db) o[db] *= alpha;
    }
    // V^T operand: channel d = 16 db + lr, keys 32g .. 32g+31 of the tile
    const int kv0 = key0 + 32 * g;
    const bool vin = kv0 < kend;
    int64_t vpage = vin ? pt[kv0 >> 6] : 0;
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      u32x4 va = {0u, 0u, 0u, 0u}, vb = {0u, 0u, 0u, 0u};
      if (vin) {
        const uint8_t* src = p.v_codes + ((vpage * p.h_kv + hk) * kD + 16 * db + lr) * kPage + (kv0 & 63);
        va = *reinterpret_cast<const u32x4*>(src);
        vb = *reinterpret_cast<const u32x4*>(src + 16);
        if (kv0 + 32 > kend) {
          const int nv = kend - kv0;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            int k1 = nv - 4 * i, k2 = nv - 16 - 4 * i;
            va[i] &= k1 >= 4 ? 0xFFFFFFFFu : (k1 <= 0 ? 0u : ((1u << (8 * k1)) - 1u));
            vb[i] &= k2 >= 4 ? 0xFFFFFFFFu : (k2 <= 0 ? 0u : ((1u << (8 * k2)) - 1u));
          }
        }
      }
      const i32x8 vop = {(int)va[0], (int)va[1], (int)va[2], (int)va[3],
                         (int)vb[0], (int)vb[1], (int)vb[2], (int)vb[3]};
      o[db] = mfma_fp8(vop, pb, o[db]);
    }
  }

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
}

// One workgroup (128 threads, one per channel) per (sequence, query head).
__global__ __launch_bounds__(128) void merge_kernel(DecodeParams p) {
  const int h = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
  const int kvl = p.kv_len[b];
  const int np = (kvl + p.partition_tokens - 1) / p.partition_tokens;
  const float* st = p.ws + ((int64_t)b * p.h_q + h) * p.max_partitions * (kD + 2);
  float M = -INFINITY;
  for (int q = 0; q < np; ++q) M = fmaxf(M, st[q * (kD + 2)]);
  float L = 0.0f, O = 0.0f;
  for (int q = 0; q < np; ++q) {
    const float f = __builtin_amdgcn_exp2f(st[q * (kD + 2)] - M);
    L = __builtin_fmaf(f, st[q * (kD + 2) + 1], L);
    O = __builtin_fmaf(f, st[q * (kD + 2) + 2 + d], O);
  }
  const float r = np > 0 ? __fdiv_rn(O, L) : 0.0f;
  p.out[((int64_t)b * p.h_q + h) * kD + d] = bf16_rne(r);
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, hipStream_t stream) {
  if (p.batch == 0) return hipSuccess;
  const dim3 grid((p.max_partitions + kWavesPerBlock - 1) / kWavesPerBlock, p.h_kv, p.batch);
  decode_kernel<<<grid, dim3(kWavesPerBlock * 64), 0, stream>>>(p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  merge_kernel<<<dim3(p.h_q, p.batch), dim3(128), 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace mpfa
