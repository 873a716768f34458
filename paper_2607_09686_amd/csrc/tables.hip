// Moving one layer's device-resident slot table to and from a pinned host
// staging buffer with one kernel each way (instead of one runtime copy per
// array), so that a multi-token call, whose table step runs on the host, pays
// one launch for the pull and one for the push.  The staging layout is
// table_stage_bytes(E, C) bytes: stamp [E] i64 | meta [3] i64 | cnt [4] u64 |
// err i32 | pad i32 | slot_of [E] i32 | expert_in [C] i32.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"

namespace moecache {
namespace {

constexpr int kTableThreads = 256;

__global__ __launch_bounds__(kTableThreads) void table_pack_kernel(LruDev L, int E, int C,
                                                                   const int32_t *err,
                                                                   uint8_t *stage) {
  int64_t *stamp = reinterpret_cast<int64_t *>(stage), *meta = stamp + E;
  uint64_t *cnt = reinterpret_cast<uint64_t *>(meta + 3);
  int32_t *errp = reinterpret_cast<int32_t *>(cnt + 4), *so = errp + 2, *ei = so + E;
  for (int i = threadIdx.x; i < E; i += kTableThreads) {
    stamp[i] = L.stamp[i];
    so[i] = L.slot_of[i];
  }
  for (int i = threadIdx.x; i < C; i += kTableThreads) ei[i] = L.expert_in[i];
  if (threadIdx.x < 3) meta[threadIdx.x] = L.meta[threadIdx.x];
  if (threadIdx.x < 4) cnt[threadIdx.x] = L.cnt[threadIdx.x];
  if (threadIdx.x == 0) errp[0] = *err;
}

__global__ __launch_bounds__(kTableThreads) void table_unpack_kernel(LruDev L, int E, int C,
                                                                     const uint8_t *stage) {
  const int64_t *stamp = reinterpret_cast<const int64_t *>(stage), *meta = stamp + E;
  const uint64_t *cnt = reinterpret_cast<const uint64_t *>(meta + 3);
  const int32_t *so = reinterpret_cast<const int32_t *>(cnt + 4) + 2, *ei = so + E;
  for (int i = threadIdx.x; i < E; i += kTableThreads) {
    L.stamp[i] = stamp[i];
    L.slot_of[i] = so[i];
  }
  for (int i = threadIdx.x; i < C; i += kTableThreads) L.expert_in[i] = ei[i];
  if (threadIdx.x < 3) L.meta[threadIdx.x] = meta[threadIdx.x];
  if (threadIdx.x < 4) L.cnt[threadIdx.x] = cnt[threadIdx.x];
}

}  // namespace

size_t table_stage_bytes(int E, int C) { return 8 * (size_t)E + 64 + 4 * (size_t)E + 4 * (size_t)C; }

hipError_t launch_table_pack(const LruDev &L, int E, int C, const int32_t *err, uint8_t *stage,
                             hipStream_t s) {
  hipLaunchKernelGGL(table_pack_kernel, dim3(1), dim3(kTableThreads), 0, s, L, E, C, err, stage);
  return hipGetLastError();
}

hipError_t launch_table_unpack(const LruDev &L, int E, int C, const uint8_t *stage, hipStream_t s) {
  hipLaunchKernelGGL(table_unpack_kernel, dim3(1), dim3(kTableThreads), 0, s, L, E, C, stage);
  return hipGetLastError();
}

}  // namespace moecache
