// prefill.hip -- causal QK4PV8 prefill for gfx950 (Algorithm 1 main loop).
//
// One workgroup = 8 waves = 256 query rows of one query head; each wave owns
// 32 rows (two 16-row MFMA column blocks).  Per 128-key tile (visited from the
// block's last tile down to tile 0, Sec. 4.1):
//   * the workgroup stages the tile in LDS: NVFP4 K dequantized once to exact
//     FP16 (group scale applied, tensor scale factored out), FP8 V in its
//     channel-major page layout, and the compensation vector Delta_S;
//   * each wave computes S^T = K Q^T on FP16 MFMA (16x16x32) starting from
//     the rank-one term 1 Delta_S^T (Sec. 4.3 Eq. 11): loaded from LDS as the
//     accumulator input, or (MPFA_SEED_MFMA) formed by one BF16 rank-one MFMA
//     per 16x16 block as in Sec. 5.2;
//   * mask, row max, P = 2^(lambda (S - m) + log2 448), row sum of the FP32 P,
//     FP8 conversion in registers; the S^T accumulator layout is already the
//     B-operand layout of the FP8 PV MFMA (O^T = V^T P^T), so P never leaves
//     registers;
//   * O^T rescale (skipped when no row maximum moved) and FP8 MFMA
//     (16x16x128) accumulation.
// The key order inside a 16-row MFMA block is permuted so that the 32 keys a
// lane holds after the QK product are contiguous: MFMA row r of key block mb
// is key 32*(r/4) + 4*mb + r%4.
#include "prefill_body.h"

namespace mpfa {

namespace {

template <int SEED, bool MX, int PV, int ABL = 0>
__global__ __launch_bounds__(kThreads, 1) void prefill_kernel(PrefillParams p) {
  __shared__ __attribute__((aligned(16))) PrefillSmemT<PV> smem[2];
  prefill_item<SEED, MX, PV, ABL>(p, blockIdx.x, smem);
}

#ifdef MPFA_ABLATION_BUILD
// Characterization library only: softmax ablation level of the method's
// kernels (compensation as accumulator input, FP8 PV), see softmax_tile.
int g_ablation = 0;
#endif

}  // namespace

#ifdef MPFA_ABLATION_BUILD
// declared in include/mpfa_ablate.h
extern "C" int mpfa_ablation_set_level(int level) {
  if (level < 0 || level > 2) return 1;
  g_ablation = level;
  return 0;
}
#endif

hipError_t launch_prefill(const PrefillParams& p, hipStream_t stream) {
  const unsigned blocks = (unsigned)(p.n_qtiles * p.h_q * p.batch);
  if (blocks == 0) return hipSuccess;
  const dim3 grid(blocks), block(kThreads);
#ifdef MPFA_ABLATION_BUILD
  if (g_ablation > 0 && p.pv == kPvFp8 && p.smooth && !p.seed_mfma && !p.seed_elem) {
    if (p.mx) {
      if (g_ablation == 1) prefill_kernel<kSeedInit, true, kPvFp8, 1><<<grid, block, 0, stream>>>(p);
      else prefill_kernel<kSeedInit, true, kPvFp8, 2><<<grid, block, 0, stream>>>(p);
    } else {
      if (g_ablation == 1) prefill_kernel<kSeedInit, false, kPvFp8, 1><<<grid, block, 0, stream>>>(p);
      else prefill_kernel<kSeedInit, false, kPvFp8, 2><<<grid, block, 0, stream>>>(p);
    }
    return hipGetLastError();
  }
#endif
  if (p.pv == kPvBf16) {
    if (!p.smooth) prefill_kernel<kSeedNone, false, kPvBf16><<<grid, block, 0, stream>>>(p);
    else prefill_kernel<kSeedInit, false, kPvBf16><<<grid, block, 0, stream>>>(p);
  } else if (p.pv == kPvNvfp4) {
    if (!p.smooth) prefill_kernel<kSeedNone, false, kPvNvfp4><<<grid, block, 0, stream>>>(p);
    else prefill_kernel<kSeedInit, false, kPvNvfp4><<<grid, block, 0, stream>>>(p);
  } else if (p.mx) {
    if (!p.smooth) prefill_kernel<kSeedNone, true, kPvFp8><<<grid, block, 0, stream>>>(p);
    else if (p.seed_mfma) prefill_kernel<kSeedMfma, true, kPvFp8><<<grid, block, 0, stream>>>(p);
    else if (p.seed_elem) prefill_kernel<kSeedElem, true, kPvFp8><<<grid, block, 0, stream>>>(p);
    else prefill_kernel<kSeedInit, true, kPvFp8><<<grid, block, 0, stream>>>(p);
  } else {
    if (!p.smooth) prefill_kernel<kSeedNone, false, kPvFp8><<<grid, block, 0, stream>>>(p);
    else if (p.seed_mfma) prefill_kernel<kSeedMfma, false, kPvFp8><<<grid, block, 0, stream>>>(p);
    else if (p.seed_elem) prefill_kernel<kSeedElem, false, kPvFp8><<<grid, block, 0, stream>>>(p);
    else prefill_kernel<kSeedInit, false, kPvFp8><<<grid, block, 0, stream>>>(p);
  }
  return hipGetLastError();
}

int prefill_query_rows_per_block() { return kQRows; }

}  // namespace mpfa
