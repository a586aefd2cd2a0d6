// mixed.hip -- one launch for a serving step that mixes a causal prefill chunk
// and split-KV decode (Sec. 7.3: prefill and decode requests served together).
//
// The prefill work items (query head, 256-row query tile; matrix-bound) and
// groups of eight decode work items (sequence, KV head, partition; HBM-bound)
// share one grid.  Each decode partition counts itself in a per-(sequence, KV
// head) counter when its state is written; the last one merges the group's
// query heads (log-sum-exp, the same arithmetic as the separate merge kernel)
// and resets the counter, so the step needs no second launch.  A workgroup is
// 512 threads; a prefill item uses about 98 KB of LDS for its two tile buffers, a
// group of eight decode items none (their K and V go straight to registers).
//
// Placement: a prefill workgroup holds a whole compute unit (its LDS and all
// of its registers), so prefill and decode cannot share a unit at the same
// time; decode rounds spread through the prefill only take unit time from it
// (measured slower than two launches).  The host therefore places the decode
// rounds first: they stream the KV pages at full bandwidth on every unit, then
// the prefill tiles follow in their largest-first order.
#include "decode_body.h"
#include "prefill_body.h"

namespace mpfa {

namespace {

constexpr int kMixedLds = sizeof(PrefillSmemT<kPvFp8>) * 2;

// Blocks are dealt to the 8 XCDs round-robin, so the grid is laid out in rounds
// of 8 consecutive blocks.  Decode rounds (8 groups of 8 decode work items)
// sit at round indices first, first + stride, ...; prefill items fill the
// other rounds in their own order (largest query tiles first).  Whole rounds keep
// every prefill item on the XCD its index selects (index = block - 8 * decode
// rounds before it, the same residue mod 8), so the KV-head-per-XCD placement
// of the prefill items holds as in the separate launch.
template <bool SMOOTH, bool MX>
__global__ __launch_bounds__(512, 1) void mixed_kernel(MixedParams m) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[kMixedLds];
  const int i = blockIdx.x, r = i >> 3;
  // decode round k sits at round first + k * stride (k < n_dec_rounds)
  const int rel = r - m.first;
  const bool is_dec = rel >= 0 && rel % m.stride == 0 && rel / m.stride < m.n_dec_rounds;
  const int dec_before = rel < 0 ? 0 : min(rel / m.stride + 1, m.n_dec_rounds);   // rounds <= r
  if (!is_dec) {
    const int bid = i - 8 * dec_before;
    if (bid >= m.n_pre_blocks) return;
    prefill_item<SMOOTH ? kSeedInit : kSeedNone, MX, kPvFp8>(m.pre, bid,
                                                             reinterpret_cast<PrefillSmemT<kPvFp8>*>(lds));
    return;
  }
  // decode group (round, lane of the round): wave w takes item 8 * group + w =
  // ((b * h_kv + hk) * max_partitions + part)
  const int wave = threadIdx.x >> 6;
  const int item = ((dec_before - 1) * 8 + (i & 7)) * 8 + wave;
  const DecodeParams& p = m.dec;
  const int part = item % p.max_partitions;
  const int hk = (item / p.max_partitions) % p.h_kv;
  const int b = item / (p.max_partitions * p.h_kv);
  if (b >= p.batch) return;
  decode_partition<SMOOTH, MX, true>(p, b, hk, part, m.counters);
}

}  // namespace

hipError_t launch_mixed(const MixedParams& m, hipStream_t stream) {
  const unsigned blocks = (unsigned)m.n_blocks;
  if (blocks == 0) return hipSuccess;
  const dim3 grid(blocks), block(512);
  if (m.pre.mx) {
    if (m.pre.smooth) mixed_kernel<true, true><<<grid, block, 0, stream>>>(m);
    else mixed_kernel<false, true><<<grid, block, 0, stream>>>(m);
  } else {
    if (m.pre.smooth) mixed_kernel<true, false><<<grid, block, 0, stream>>>(m);
    else mixed_kernel<false, false><<<grid, block, 0, stream>>>(m);
  }
  return hipGetLastError();
}

}  // namespace mpfa
