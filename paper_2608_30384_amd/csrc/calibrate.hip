// Read-bandwidth calibration: a plain streaming read of a device buffer, the
// reference against which the scan's achieved HBM bandwidth is compared.
// Not part of the method.
#include "rslm_internal.h"

namespace rslm {

constexpr int kCalThreads = 256;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ uint32_t xor16(const uint4 *p) {
  if (NT) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return v.x ^ v.y ^ v.z ^ v.w;
  }
  const uint4 v = *p;
  return v.x ^ v.y ^ v.z ^ v.w;
}

// Each thread XORs the 16-byte words i = t, t + T, t + 2T, ... (T = all
// threads of the grid), four loads in flight, and the workgroup's XOR goes
// to out[blockIdx.x] so that no load can be dropped.  NT: non-temporal loads.
template <bool NT>
__global__ void __launch_bounds__(kCalThreads) k_calibrate_read(const uint4 *__restrict__ buf,
                                                                int64_t n16,
                                                                uint32_t *__restrict__ out) {
  __shared__ uint32_t red[kCalThreads / 64];
  const int64_t T = int64_t(gridDim.x) * kCalThreads;
  int64_t i = int64_t(blockIdx.x) * kCalThreads + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * T < n16; i += 4 * T) {
    const uint32_t a = xor16<NT>(buf + i), b = xor16<NT>(buf + i + T);
    const uint32_t c = xor16<NT>(buf + i + 2 * T), d = xor16<NT>(buf + i + 3 * T);
    acc ^= a ^ b ^ c ^ d;
  }
  for (; i < n16; i += T) acc ^= xor16<NT>(buf + i);
  for (int off = 32; off >= 1; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t v = 0;
    for (int w = 0; w < kCalThreads / 64; ++w) v ^= red[w];
    out[blockIdx.x] = v;
  }
}

}  // namespace rslm

using namespace rslm;

extern "C" int rslm_calibrate_read(const void *buf, int64_t bytes, uint32_t *out, int32_t grid,
                                   int nontemporal, void *stream) {
  if (bytes < 0 || bytes % 16 || grid < 1 || (bytes && !buf) || !out) return RSLM_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(buf) % 16) return RSLM_ERR_INVALID_ARG;
  if (nontemporal)
    hipLaunchKernelGGL(k_calibrate_read<true>, dim3(unsigned(grid)), dim3(kCalThreads), 0,
                       as_stream(stream), reinterpret_cast<const uint4 *>(buf), bytes / 16, out);
  else
    hipLaunchKernelGGL(k_calibrate_read<false>, dim3(unsigned(grid)), dim3(kCalThreads), 0,
                       as_stream(stream), reinterpret_cast<const uint4 *>(buf), bytes / 16, out);
  return check_launch();
}
