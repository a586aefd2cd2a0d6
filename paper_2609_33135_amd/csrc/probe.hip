// Measurement probes: the matrix-core issue rate of each MFMA form and the HBM
// read rate, measured on the device (declared in mpfa_probe.h).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mpfa_probe.h"

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef int i8v __attribute__((ext_vector_type(8)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(1))) void* global_ptr_t;

constexpr int kThreads = 256;   // 4 waves: one per SIMD
constexpr int kChains = 8;      // independent accumulators per wave (covers the MFMA latency)
constexpr int kUnroll = 8;      // 16-byte words per thread and round of the read probe
constexpr int kMaxBlocks = 1 << 20;

template <int KIND>
__device__ __forceinline__ f4 mfma_step(uint32_t pa, uint32_t pb, f4 c) {
  if constexpr (KIND == MPFA_PROBE_MFMA_F16) {
    const h8 a = __builtin_bit_cast(h8, (u4){pa, pa, pa, pa});
    const h8 b = __builtin_bit_cast(h8, (u4){pb, pb, pb, pb});
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
  } else if constexpr (KIND == MPFA_PROBE_MFMA_FP8) {
    const int a = (int)pa, b = (int)pb;
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4((i8v){a, a, a, a, a, a, a, a},
                                                             (i8v){b, b, b, b, b, b, b, b}, c, 0, 0, 0,
                                                             0x7F7F7F7F, 0, 0x7F7F7F7F);
  } else {
    const int a = (int)pa, b = (int)pb;
    return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4((i8v){a, a, a, a, 0, 0, 0, 0},
                                                             (i8v){b, b, b, b, 0, 0, 0, 0}, c, 4, 4, 0,
                                                             0x7F7F7F7F, 0, 0x7F7F7F7F);
  }
}

template <int KIND>
__global__ __launch_bounds__(kThreads) void mfma_probe_kernel(int iters, uint32_t pa, uint32_t pb, float* sink) {
  f4 acc[kChains];
#pragma unroll
  for (int i = 0; i < kChains; ++i) acc[i] = (f4){0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kChains; ++i) acc[i] = mfma_step<KIND>(pa, pb, acc[i]);
    // keep each accumulator in one register tuple across rounds (no copies in the loop)
#pragma unroll
    for (int i = 0; i < kChains; ++i) __asm__ volatile("" : "+v"(acc[i]));
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kChains; ++i) s += (acc[i][0] + acc[i][1]) + (acc[i][2] + acc[i][3]);
  sink[(int64_t)blockIdx.x * kThreads + threadIdx.x] = s;
}

// Workgroup b streams its own contiguous share of the buffer: in round r thread
// x reads words ((b * rounds + r) * kUnroll + u) * kThreads + x, u < kUnroll, so
// every word is read exactly once.  (Contiguous shares stream at about 6.2
// TB/s; interleaving the workgroups word-block by word-block reaches about 6.0.)
template <bool LDS>
__global__ __launch_bounds__(kThreads) void read_probe_kernel(const u4* __restrict__ src, int64_t rounds,
                                                             uint32_t* sink) {
  __shared__ u4 slab[LDS ? kUnroll * kThreads : 1];
  const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  u4 x = {0u, 0u, 0u, 0u};
  for (int64_t r = 0; r < rounds; ++r) {
    const u4* base = src + ((int64_t)blockIdx.x * rounds + r) * kUnroll * kThreads + threadIdx.x;
    if (LDS) {
      // the LDS address operand is the wave's base: lane l's word lands at base + l
      const int wave_base = threadIdx.x & ~63;
      __builtin_amdgcn_s_waitcnt(0);   // the previous round's reads of the slab are done
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        __builtin_amdgcn_global_load_lds((global_ptr_t)(base + u * kThreads), (lds_ptr_t)(slab + u * kThreads + wave_base),
                                         16, 0, 0);
      __builtin_amdgcn_s_waitcnt(0);   // the direct loads have written the slab
      __asm__ volatile("" ::: "memory");
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) x ^= slab[u * kThreads + threadIdx.x];
    } else {
      u4 w[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) w[u] = base[u * kThreads];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) x ^= w[u];
    }
  }
  sink[t] = x[0] ^ x[1] ^ x[2] ^ x[3];
}

}  // namespace

extern "C" {

mpfa_status mpfa_probe_mfma(int32_t kind, int32_t iters, int32_t blocks, uint32_t pa, uint32_t pb, float* sink,
                            mpfa_stream_t stream) {
  if (kind < MPFA_PROBE_MFMA_F16 || kind > MPFA_PROBE_MFMA_FP4 || iters < 1 || blocks < 1 ||
      blocks > kMaxBlocks || !sink)
    return MPFA_ERR_INVALID;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid(blocks), block(kThreads);
  if (kind == MPFA_PROBE_MFMA_F16) mfma_probe_kernel<MPFA_PROBE_MFMA_F16><<<grid, block, 0, s>>>(iters, pa, pb, sink);
  else if (kind == MPFA_PROBE_MFMA_FP8) mfma_probe_kernel<MPFA_PROBE_MFMA_FP8><<<grid, block, 0, s>>>(iters, pa, pb, sink);
  else mfma_probe_kernel<MPFA_PROBE_MFMA_FP4><<<grid, block, 0, s>>>(iters, pa, pb, sink);
  return hipGetLastError() == hipSuccess ? MPFA_OK : MPFA_ERR_HIP;
}

mpfa_status mpfa_probe_read(int32_t mode, const void* src, int64_t bytes, int32_t blocks, uint32_t* sink,
                            mpfa_stream_t stream) {
  if (mode < MPFA_PROBE_READ_VGPR || mode > MPFA_PROBE_READ_LDS || !src || !sink || blocks < 1 ||
      blocks > kMaxBlocks || (reinterpret_cast<uintptr_t>(src) & 15) != 0)
    return MPFA_ERR_INVALID;
  const int64_t per_round = (int64_t)blocks * kThreads * kUnroll * 16;
  if (bytes <= 0 || bytes % per_round != 0) return MPFA_ERR_INVALID;
  const int64_t rounds = bytes / per_round;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const u4* p = reinterpret_cast<const u4*>(src);
  if (mode == MPFA_PROBE_READ_LDS) read_probe_kernel<true><<<dim3(blocks), dim3(kThreads), 0, s>>>(p, rounds, sink);
  else read_probe_kernel<false><<<dim3(blocks), dim3(kThreads), 0, s>>>(p, rounds, sink);
  return hipGetLastError() == hipSuccess ? MPFA_OK : MPFA_ERR_HIP;
}

}  // extern "C"
