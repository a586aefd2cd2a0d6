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

namespace mpfa {

namespace {

template <bool SMOOTH, bool MX>
__global__ __launch_bounds__(kWavesPerBlock * 64, 2) void decode_kernel(DecodeParams p) {
  __shared__ __attribute__((aligned(16))) uint8_t vlds[kWavesPerBlock * kVBytes];
  const int wave = threadIdx.x >> 6;
  decode_partition<SMOOTH, MX, false>(p, blockIdx.z, blockIdx.y, blockIdx.x * kWavesPerBlock + wave,
                                      vlds + wave * kVBytes, nullptr);
}

// One workgroup (128 threads, one per channel) per (sequence, query head).
__global__ __launch_bounds__(128) void merge_kernel(DecodeParams p) {
  const int h = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
  const int np = (p.kv_len[b] + p.partition_tokens - 1) / p.partition_tokens;
  p.out[((int64_t)b * p.h_q + h) * kD + d] = bf16_rne(merge_channel(p, b, h, d, np));
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, hipStream_t stream) {
  if (p.batch == 0) return hipSuccess;
  // Workgroups are dealt to the 8 XCDs round-robin by linear block id.  With
  // an even number of partition groups per (KV head, sequence) row the XCD of
  // a block depends mostly on its partition group, and the late groups exist
  // only for the long sequences, so the XCDs get unequal work (0.95 ms
  // against 0.84 ms for the Llama batch when the count is a multiple of 8).
  // An odd count spreads every row over all XCDs; the extra groups hold no
  // partition of any sequence and return at once.
  const int groups = (p.max_partitions + kWavesPerBlock - 1) / kWavesPerBlock;
  const dim3 grid(groups | 1, p.h_kv, p.batch);
  const dim3 block(kWavesPerBlock * 64);
  if (p.mx) {
    if (p.smooth) decode_kernel<true, true><<<grid, block, 0, stream>>>(p);
    else decode_kernel<false, true><<<grid, block, 0, stream>>>(p);
  } else {
    if (p.smooth) decode_kernel<true, false><<<grid, block, 0, stream>>>(p);
    else decode_kernel<false, false><<<grid, block, 0, stream>>>(p);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  merge_kernel<<<dim3(p.h_q, p.batch), dim3(128), 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace mpfa
