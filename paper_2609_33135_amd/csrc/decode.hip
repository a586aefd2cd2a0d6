// decode.hip -- split-KV QK4PV8 decode over the paged cache for gfx950
// (Sec. 5.3), plus the log-sum-exp merge of the partition states.
//
// One wave = one (sequence, KV head, partition).  The G = H_q / H_kv query
// heads of the KV head are packed into the 16-wide MFMA column dimension
// (GQA packing); the compensation becomes a rank-G term (Delta_S differs per
// query head), loaded as the input accumulator of the first QK MFMA: each
// lane's four accumulator rows are four consecutive keys of one query head,
// one 8-byte load per 16-key block.  K and V stream straight
// from HBM into registers (no LDS): each lane loads 16 contiguous bytes of
// NVFP4 codes per key it owns and 32 contiguous FP8 bytes of the channel-major
// V page, dequantizes K exactly to FP16 and runs the same S^T = K Q^T /
// O^T = V^T P^T MFMA chain as prefill.  The reduction (head) dimension is
// permuted (lane group g, step ks, element e -> channel 32g + 8ks + e) so that
// every lane's code bytes are contiguous; Q uses the same permutation.
#include "decode_body.h"

#include <mutex>

namespace mpfa {

// Partition states of mpfa_decode_paged_static: one array per GPU, created
// with the code object and held until the process ends.  Host code never uses
// the name itself (on the host it only stands for the symbol); it uses the
// device address that hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_addr[kMaxDevices] = {};
}  // namespace

hipError_t static_decode_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_addr[dev]) {
    void* a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    scratch_addr[dev] = a;
  }
  *ptr = scratch_addr[dev];
  return hipSuccess;
}

namespace {

// Block -> work map.  Workgroups are dealt to the 8 XCDs round-robin by block
// id.  The (sequence, group of kWavesPerBlock partitions) pairs that hold work
// are numbered k = 0, 1, ... in sequence order, so no workgroup is spent on a
// partition past a short sequence's end.  Pair k takes the 8 blocks of slot k
// (one per XCD), and the KV head run on XCD x is (x - k) mod 8: each pair's
// heads spread over all XCDs and every XCD sees every head, so the XCDs share
// the work evenly whatever the sequence lengths.  KV head counts above 8 take
// ceil(h_kv / 8) consecutive slots per pair.  A block finds its pair by a
// prefix sum of the sequences' group counts across the wave's lanes, 64
// sequences at a time.  That lookup costs every block O(batch), so batches
// above kDecodePackedMaxBatch sequences use the plain grid (partition group, KV
// head, sequence) instead, with an odd group count so that each (KV head,
// sequence) row still spreads over the XCDs.  Either map gives every
// partition to exactly one wave; the results do not depend on it.
__device__ __forceinline__ int partition_groups(int kvl, int partition_tokens) {
  const int np = (kvl + partition_tokens - 1) / partition_tokens;
  return (np + kWavesPerBlock - 1) / kWavesPerBlock;
}

template <bool SMOOTH, bool MX, bool PACKED>
__global__ __launch_bounds__(kWavesPerBlock * 64, 2) void decode_kernel(DecodeParams p) {
  const int wave = threadIdx.x >> 6;
  if (!PACKED) {
    // grid (partition group, KV head, sequence); groups past the sequence's
    // partitions return inside decode_partition
    decode_partition<SMOOTH, MX, false>(p, blockIdx.z, blockIdx.y, blockIdx.x * kWavesPerBlock + wave, nullptr);
    return;
  }
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int hrows = (p.h_kv + 7) >> 3;
  const int k = slot / hrows, hk = (slot % hrows) * 8 + ((xcd - k) & 7);
  if (hk >= p.h_kv) return;
  const int lane = threadIdx.x & 63;
  int b = -1, grp = 0, base = 0;
  for (int b0 = 0; b0 < p.batch && b < 0; b0 += 64) {
    const int bb = b0 + lane;
    const int cnt = bb < p.batch ? partition_groups(p.kv_len[bb], p.partition_tokens) : 0;
    int incl = cnt;   // inclusive prefix sum over the lanes
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int up = __shfl_up(incl, d);
      if (lane >= d) incl += up;
    }
    const int total = __shfl(incl, 63);
    if (k < base + total) {
      const uint64_t past = __ballot(base + incl > k);   // lanes whose sequence ends after pair k
      const int first = __ffsll((unsigned long long)past) - 1;
      b = b0 + first;
      grp = k - (base + __shfl(incl, first) - __shfl(cnt, first));
    }
    base += total;
  }
  if (b < 0) return;   // the grid is sized for batch * ceil(max_partitions / 4) pairs
  decode_partition<SMOOTH, MX, false>(p, b, hk, grp * kWavesPerBlock + wave, nullptr);
}

// One wave per (sequence, query head).  A separate launch: merging in the
// last-arriving decode wave needs the partition states made visible across
// the XCDs' L2 caches (an L2 write-back per wave, or write-through stores and
// an arrival counter), which measured slower than this second launch.
__global__ __launch_bounds__(64) void merge_kernel(DecodeParams p) {
  const int h = blockIdx.x, b = blockIdx.y;
  merge_head(p, b, h, (p.kv_len[b] + p.partition_tokens - 1) / p.partition_tokens);
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, hipStream_t stream) {
  if (p.batch == 0) return hipSuccess;
  const int groups = (p.max_partitions + kWavesPerBlock - 1) / kWavesPerBlock;
  const dim3 block(kWavesPerBlock * 64);
  if (p.batch <= kDecodePackedMaxBatch) {
    const int64_t pairs = (int64_t)p.batch * groups;
    const dim3 grid((unsigned)(pairs * ((p.h_kv + 7) / 8 * 8)));
    if (p.mx) {
      if (p.smooth) decode_kernel<true, true, true><<<grid, block, 0, stream>>>(p);
      else decode_kernel<false, true, true><<<grid, block, 0, stream>>>(p);
    } else {
      if (p.smooth) decode_kernel<true, false, true><<<grid, block, 0, stream>>>(p);
      else decode_kernel<false, false, true><<<grid, block, 0, stream>>>(p);
    }
  } else {
    const dim3 grid(groups | 1, p.h_kv, p.batch);
    if (p.mx) {
      if (p.smooth) decode_kernel<true, true, false><<<grid, block, 0, stream>>>(p);
      else decode_kernel<false, true, false><<<grid, block, 0, stream>>>(p);
    } else {
      if (p.smooth) decode_kernel<true, false, false><<<grid, block, 0, stream>>>(p);
      else decode_kernel<false, false, false><<<grid, block, 0, stream>>>(p);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  merge_kernel<<<dim3(p.h_q, p.batch), dim3(64), 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace mpfa
