// mixed.hip -- one launch for a serving step that mixes a causal prefill chunk
// and split-KV decode (Sec. 7.3: prefill and decode requests served together).
//
// The prefill work items (query head, 256-row query tile; compute-bound on the
// matrix cores) and groups of eight decode work items (sequence, KV head,
// partition; HBM-bound) share one grid.  Decode groups are spread evenly
// through the dispatch order, so while most compute units run prefill tiles
// the others stream KV pages, and both resources stay busy in the same
// interval instead of one launch after the other.  Each decode partition
// counts itself in a per-(sequence, KV head) counter when its state is
// written; the last one merges the group's query heads (log-sum-exp, the same
// arithmetic as the separate merge kernel) and resets the counter, so the
// step needs no second launch.  A workgroup is 512 threads with 128 KB of
// LDS: two prefill tile buffers, or eight 16 KB decode V slabs.
#include "decode_body.h"
#include "prefill_body.h"

namespace mpfa {

namespace {

constexpr int kMixedLds = 8 * kVBytes;
static_assert(sizeof(PrefillSmemT<kPvFp8>) * 2 <= kMixedLds, "prefill tiles must fit the mixed LDS");

// Block i of the grid: the decode groups sit at positions stride-1, 2*stride-1,
// ... (stride = total / decode groups), the prefill items fill the rest in
// their own order (largest query tiles first).
template <bool SMOOTH, bool MX>
__global__ __launch_bounds__(512, 1) void mixed_kernel(MixedParams m) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[kMixedLds];
  const int i = blockIdx.x;
  const int dec_before = min((i + 1) / m.stride, m.n_dec_blocks);
  const bool is_dec = m.n_dec_blocks > 0 && (i + 1) % m.stride == 0 && (i + 1) / m.stride <= m.n_dec_blocks;
  if (!is_dec) {
    prefill_item<SMOOTH ? kSeedMfma : kSeedNone, MX, kPvFp8>(m.pre, i - dec_before,
                                                             reinterpret_cast<PrefillSmemT<kPvFp8>*>(lds));
    return;
  }
  // decode group k: wave w takes item 8k + w = ((b * h_kv + hk) * max_partitions + part)
  const int wave = threadIdx.x >> 6;
  const int item = (dec_before - 1) * 8 + wave;
  const DecodeParams& p = m.dec;
  const int part = item % p.max_partitions;
  const int hk = (item / p.max_partitions) % p.h_kv;
  const int b = item / (p.max_partitions * p.h_kv);
  if (b >= p.batch) return;
  decode_partition<SMOOTH, MX, true>(p, b, hk, part, lds + wave * kVBytes, m.counters);
}

}  // namespace

hipError_t launch_mixed(const MixedParams& m, hipStream_t stream) {
  const unsigned blocks = (unsigned)(m.n_pre_blocks + m.n_dec_blocks);
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
