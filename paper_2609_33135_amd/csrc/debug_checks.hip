// debug_checks.hip -- device side of the debug build's data checks: a scan of
// BF16 inputs for non-finite values (exponent field all ones).  Called only by
// the host entry points of the debug library, before any kernel that would
// consume the data.
#include <algorithm>

#include "mpfa_internal.h"

namespace mpfa {

namespace {

__global__ __launch_bounds__(256) void scan_nonfinite_kernel(const uint16_t* x, int64_t n, int* flag) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    bad |= (x[i] & 0x7F80u) == 0x7F80u;
  if (__builtin_amdgcn_ballot_w64(bad) != 0 && (threadIdx.x & 63) == 0) atomicOr(flag, 1);
}

}  // namespace

hipError_t launch_scan_nonfinite(const uint16_t* x, int64_t n, int* flag, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>((n + 255) / 256, 4096);
  scan_nonfinite_kernel<<<dim3((unsigned)blocks), dim3(256), 0, stream>>>(x, n, flag);
  return hipGetLastError();
}

}  // namespace mpfa
