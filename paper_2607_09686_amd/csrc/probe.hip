// Reference launches for the short HBM-bound kernels: an empty kernel and a
// plain streaming read of a buffer, timed with the same runtime-stamped kernel
// events as the FFN kernels, so that a kernel's duration can be set against
// what one launch over the same bytes costs at best on this device.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace moecache {
namespace {

constexpr int kProbeThreads = 256;
typedef uint32_t probe_u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kProbeThreads) void empty_probe_kernel(uint32_t *out) {
  if (out != nullptr && threadIdx.x == kProbeThreads) out[0] = 0u;  // never taken
}

// 16-byte loads, grid-strided, four in flight per lane; one word per block so
// that the loads are not dropped.
__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const probe_u32x4 *__restrict__ src,
                                                                   int64_t n16, uint32_t *out) {
  uint32_t acc = 0u;
  const int64_t stride = (int64_t)gridDim.x * kProbeThreads;
  int64_t i = (int64_t)blockIdx.x * kProbeThreads + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const probe_u32x4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc += a.x ^ b.y ^ c.z ^ d.w;
  }
  for (; i < n16; i += stride) acc += src[i].x;
  __shared__ uint32_t red[kProbeThreads];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int h = kProbeThreads / 2; h >= 1; h >>= 1) {
    if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[blockIdx.x] = red[0];
}

}  // namespace

hipError_t launch_read_probe(const uint8_t *src, int64_t bytes, int grid, uint32_t *out, hipStream_t s,
                             const Timing &t) {
  if (grid < 1 || bytes < 0 || bytes % 16 != 0) return hipErrorInvalidValue;
  if (bytes == 0)
    hipExtLaunchKernelGGL(empty_probe_kernel, dim3(grid), dim3(kProbeThreads), 0, s, t.start, t.stop, 0, out);
  else
    hipExtLaunchKernelGGL(read_probe_kernel, dim3(grid), dim3(kProbeThreads), 0, s, t.start, t.stop, 0,
                          reinterpret_cast<const probe_u32x4 *>(src), bytes / 16, out);
  return hipGetLastError();
}

}  // namespace moecache
