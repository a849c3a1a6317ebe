// Measurement: the HBM rate of plain streaming reads on this device, the
// ceiling a read-bound kernel such as the split attention can reach.  Each lane
// keeps four 16-byte non-temporal loads in flight over a grid-stride walk of
// the buffer; the loaded words are folded into a checksum that is stored only
// if it equals a value the caller passes (so the loads cannot be dropped), and
// nothing else is written.
#include <hip/hip_runtime.h>

#include "../../include/sp_probe.h"
#include "common.h"

#define SP_API extern "C" __attribute__((visibility("default")))

namespace {

using namespace sp;

__global__ __launch_bounds__(256) void stream_read(const u32x4* buf, size_t n16, uint32_t key, uint32_t* sink) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 a = __builtin_nontemporal_load(buf + i);
    const u32x4 b = __builtin_nontemporal_load(buf + i + stride);
    const u32x4 c = __builtin_nontemporal_load(buf + i + 2 * stride);
    const u32x4 d = __builtin_nontemporal_load(buf + i + 3 * stride);
    acc ^= (a.x + b.y) ^ (c.z + d.w) ^ (a.w + b.x) ^ (c.y + d.z) ^ (a.y ^ a.z ^ b.z ^ b.w ^ c.x ^ c.w ^ d.x ^ d.y);
  }
  for (; i < n16; i += stride) {
    const u32x4 a = __builtin_nontemporal_load(buf + i);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  if (acc == key) sink[0] = acc;
}

}  // namespace

SP_API int sp_probe_measure_read(const void* buf, size_t bytes, int32_t reps, void* sink, float* gbps,
                                 void* stream) {
  if (!buf || !sink || !gbps || reps < 1 || bytes < 16 || ((uintptr_t)buf & 15) || ((uintptr_t)sink & 3))
    return SP_ERR_INVALID_ARG;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return SP_ERR_NO_DEVICE;
  hipStream_t s = (hipStream_t)stream;
  const size_t n16 = bytes / 16;
  const dim3 grid((unsigned)(cus * 8)), block(256);
  hipEvent_t a = nullptr, b = nullptr;
  int st = SP_OK;
  if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) st = SP_ERR_HIP;
  if (st == SP_OK) {
    // one launch to warm the code object, then the timed ones
    hipLaunchKernelGGL(stream_read, grid, block, 0, s, (const u32x4*)buf, n16, 0x9E3779B9u, (uint32_t*)sink);
    if (hipEventRecord(a, s) != hipSuccess) st = SP_ERR_HIP;
    for (int r = 0; st == SP_OK && r < reps; ++r)
      hipLaunchKernelGGL(stream_read, grid, block, 0, s, (const u32x4*)buf, n16, 0x9E3779B9u + r,
                         (uint32_t*)sink);
    if (st == SP_OK && (hipGetLastError() != hipSuccess || hipEventRecord(b, s) != hipSuccess ||
                        hipEventSynchronize(b) != hipSuccess))
      st = SP_ERR_HIP;
    float ms = 0.f;
    if (st == SP_OK && hipEventElapsedTime(&ms, a, b) != hipSuccess) st = SP_ERR_HIP;
    if (st == SP_OK) *gbps = (float)((double)n16 * 16.0 * reps / (ms * 1e-3) / 1e9);
  }
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  return st;
}
