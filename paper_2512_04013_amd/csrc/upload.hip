// Upload of a step's plan image (the host planner's work list) from pinned
// host memory to device memory by a copy kernel enqueued on the launch
// stream. A DMA-engine copy queued behind the previous step's kernels only
// starts once they have finished and then takes tens of microseconds to get
// going, which leaves the GPU idle between steps; a kernel on the same
// stream starts as soon as the previous kernel ends and reads the few
// hundred kilobytes over the host link directly.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "aug.h"
#include "status.h"

namespace {

constexpr int kThreads = 256;
constexpr int64_t kMaxGrid = 256;

// 16-byte lane loads from host memory, 16-byte stores to device memory;
// the last bytes % 16 bytes are copied one by one by the first workgroup.
__global__ __launch_bounds__(kThreads) void upload_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                          int64_t n16, int32_t tail) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; i < n16; i += stride)
    dst[i] = src[i];
  if (blockIdx.x == 0 && static_cast<int32_t>(threadIdx.x) < tail) {
    const uint8_t* s = reinterpret_cast<const uint8_t*>(src + n16);
    uint8_t* d = reinterpret_cast<uint8_t*>(dst + n16);
    d[threadIdx.x] = s[threadIdx.x];
  }
}

}  // namespace

extern "C" aug_status aug_plan_upload(const void* host_src, void* dev_dst, size_t bytes, void* stream) {
  const char* who = "aug_plan_upload";
  if (bytes == 0) return AUG_OK;
  if (!host_src || !dev_dst) return aug::fail(AUG_ERR_INVALID, "%s: NULL pointer", who);
  if (((reinterpret_cast<uintptr_t>(host_src) | reinterpret_cast<uintptr_t>(dev_dst)) & 15) != 0)
    return aug::fail(AUG_ERR_INVALID, "%s: pointers must be 16-byte aligned", who);
  if (bytes > (static_cast<size_t>(1) << 40)) return aug::fail(AUG_ERR_INVALID, "%s: %zu bytes", who, bytes);

  // the kernel dereferences host_src: it must be page-locked memory the
  // device can reach, and dev_dst device memory
  hipPointerAttribute_t ha{}, da{};
  if (hipPointerGetAttributes(&ha, host_src) != hipSuccess || ha.type != hipMemoryTypeHost ||
      ha.devicePointer == nullptr || ha.hostPointer == nullptr) {
    (void)hipGetLastError();
    return aug::fail(AUG_ERR_INVALID, "%s: host_src is not pinned host memory known to HIP", who);
  }
  if (hipPointerGetAttributes(&da, dev_dst) != hipSuccess || da.type != hipMemoryTypeDevice) {
    (void)hipGetLastError();
    return aug::fail(AUG_ERR_INVALID, "%s: dev_dst is not device memory", who);
  }
  // the device address of host_src (attributes may describe the allocation's
  // base or the queried address itself; the offset covers both)
  const char* src = static_cast<const char*>(ha.devicePointer) +
                    (static_cast<const char*>(host_src) - static_cast<const char*>(ha.hostPointer));

  const int64_t n16 = static_cast<int64_t>(bytes / 16);
  const int32_t tail = static_cast<int32_t>(bytes % 16);
  int64_t grid = (n16 + kThreads - 1) / kThreads;
  grid = grid < 1 ? 1 : grid > kMaxGrid ? kMaxGrid : grid;
  hipLaunchKernelGGL(upload_kernel, dim3(static_cast<uint32_t>(grid)), dim3(kThreads), 0,
                     static_cast<hipStream_t>(stream), reinterpret_cast<const uint4*>(src),
                     static_cast<uint4*>(dev_dst), n16, tail);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return aug::fail(AUG_ERR_HIP, "%s: launch: %s", who, hipGetErrorString(e));
  return AUG_OK;
}
