// Streaming-read probe: the HBM read rate that a plain kernel reaches on this
// device, the reference next to which the decode kernel's read rate is judged.
// Each thread reads 16-byte words grid-stride (four independent loads per
// iteration) and folds them with xor; one word per thread goes to `sink`, so the
// loads cannot be dropped and the xor of all sink words is the xor of all source
// words.
#include "../../include/oscar.h"
#include "internal.h"

namespace oscar {
namespace {

constexpr int kProbeThreads = 256;

__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const uint4* __restrict__ src,
                                                                  size_t n,
                                                                  uint32_t* __restrict__ sink) {
  const size_t tid = (size_t)blockIdx.x * kProbeThreads + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * kProbeThreads;
  uint32_t acc = 0;
  size_t i = tid;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^
           d.w;
  }
  for (; i < n; i += stride) {
    const uint4 a = src[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  sink[tid] = acc;
}

}  // namespace
}  // namespace oscar

extern "C" int oscar_hbm_read_probe(const void* src, size_t bytes, uint32_t* sink, int32_t blocks,
                                    void* stream) {
  if (!src || !sink || blocks < 1 || bytes == 0 || bytes % 16 != 0 ||
      reinterpret_cast<uintptr_t>(src) % 16 != 0 || reinterpret_cast<uintptr_t>(sink) % 4 != 0)
    return OSCAR_ERR_INVALID_ARG;
  hipLaunchKernelGGL(oscar::read_probe_kernel, dim3((unsigned)blocks), dim3(oscar::kProbeThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint4*>(src), bytes / 16,
                     sink);
  return hipGetLastError() == hipSuccess ? OSCAR_OK : OSCAR_ERR_HIP;
}
