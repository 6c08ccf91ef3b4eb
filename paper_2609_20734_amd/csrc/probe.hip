// Measurement aid: a plain streaming read of a device buffer, the ceiling the
// attention kernels' KV reads are compared with.  Every 16-byte group is read
// once with the same nontemporal loads the attention kernels use for KV; the
// words are folded into one XOR per thread so the loads cannot be dropped, and
// the fold is stored only when it equals a fixed constant (so the kernel's
// traffic is reads only).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "oda.h"
#include "oda_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kReadThreads = 256;
constexpr int kReadUnroll = 8;            // 16-byte loads in flight per thread
constexpr int kDefaultReadGroups = 256;   // one workgroup per CU streamed best in a sweep of grids
constexpr uint32_t kNeverWritten = 0x9E3779B9u;

__global__ __launch_bounds__(kReadThreads) void stream_read_kernel(const u32x4* __restrict__ p, int64_t n16,
                                                                   uint32_t* sink) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + (kReadUnroll - 1) * stride < n16; i += kReadUnroll * stride) {
    u32x4 v[kReadUnroll];
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < kReadUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(p + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == kNeverWritten) sink[0] = acc;
}

}  // namespace

extern "C" oda_status oda_stream_read(const void* src, size_t bytes, uint32_t* sink, int32_t groups,
                                      hipStream_t stream) {
  if (src == nullptr || sink == nullptr) return oda::fail(ODA_ERR_NULL, "src and sink are required");
  if (!oda::aligned(src, 16) || bytes % 16 != 0)
    return oda::fail(ODA_ERR_SHAPE, "src must be 16-byte aligned and bytes a multiple of 16 (got %zu)", bytes);
  if (groups < 0 || groups > (1 << 20)) return oda::fail(ODA_ERR_SHAPE, "groups %d: 0 (default) .. 2^20", groups);
  if (bytes == 0) return oda::ok();
  const int g = groups == 0 ? kDefaultReadGroups : groups;
  (void)hipGetLastError();
  hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)g), dim3(kReadThreads), 0, stream,
                     reinterpret_cast<const u32x4*>(src), (int64_t)(bytes / 16), sink);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return oda::fail(ODA_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return oda::ok();
}
