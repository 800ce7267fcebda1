// Streaming-read probes: the HBM read rate that a plain kernel reaches on this
// device, the reference next to which the decode kernel's read rate is judged.
// Each thread reads 16-byte words and folds them with xor; one word per thread
// goes to `sink`, so the loads cannot be dropped and the xor of all sink words
// is the xor of all source words.
//
// Access patterns (one template):
//   grid-stride : word i of thread t is t + i * threads, U independent loads per
//                 iteration (U words of one thread are `threads` words apart);
//   wave chunks : wave w reads U KiB contiguous per iteration (lane l, load u:
//                 word 64 u + l of the chunk), waves stride by all waves' chunks.
// Loads are plain or non-temporal (`nt`: the line is not kept for reuse).
#include "../../include/oscar.h"
#include "internal.h"

namespace oscar {
namespace {

constexpr int kProbeThreads = 256;
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ inline u4v ld(const u4v* p) {
  if (NT) return __builtin_nontemporal_load(p);
  return *p;
}
__device__ inline uint32_t fold(u4v v) { return v.x ^ v.y ^ v.z ^ v.w; }

template <int U, bool NT, bool CHUNK>
__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const u4v* __restrict__ src,
                                                                  size_t n,
                                                                  uint32_t* __restrict__ sink) {
  const size_t tid = (size_t)blockIdx.x * kProbeThreads + threadIdx.x;
  const size_t threads = (size_t)gridDim.x * kProbeThreads;
  uint32_t acc = 0;
  if (CHUNK) {
    const size_t lane = tid & 63, wave = tid >> 6, waves = threads >> 6;
    const size_t step = waves * 64 * U;  // words per iteration over all waves
    size_t i = wave * 64 * U + lane;
    for (; i + 64 * (U - 1) < n; i += step) {
      u4v v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = ld<NT>(src + i + 64 * u);
#pragma unroll
      for (int u = 0; u < U; ++u) acc ^= fold(v[u]);
    }
    // at most one partial chunk per wave remains (the next would start past n)
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (i + 64 * u < n) acc ^= fold(ld<NT>(src + i + 64 * u));
  } else {
    size_t i = tid;
    for (; i + (U - 1) * threads < n; i += U * threads) {
      u4v v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = ld<NT>(src + i + u * threads);
#pragma unroll
      for (int u = 0; u < U; ++u) acc ^= fold(v[u]);
    }
    for (; i < n; i += threads) acc ^= fold(ld<NT>(src + i));
  }
  sink[tid] = acc;
}

template <int U>
void launch_u(bool nt, bool chunk, dim3 grid, hipStream_t st, const u4v* src, size_t n,
              uint32_t* sink) {
  auto k = nt ? (chunk ? read_probe_kernel<U, true, true> : read_probe_kernel<U, true, false>)
              : (chunk ? read_probe_kernel<U, false, true> : read_probe_kernel<U, false, false>);
  hipLaunchKernelGGL(k, grid, dim3(kProbeThreads), 0, st, src, n, sink);
}

}  // namespace
}  // namespace oscar

extern "C" int oscar_hbm_read_probe_ex(const void* src, size_t bytes, uint32_t* sink,
                                       int32_t blocks, int32_t loads_per_thread, int32_t flags,
                                       void* stream) {
  if (!src || !sink || blocks < 1 || bytes == 0 || bytes % 16 != 0 ||
      reinterpret_cast<uintptr_t>(src) % 16 != 0 || reinterpret_cast<uintptr_t>(sink) % 4 != 0)
    return OSCAR_ERR_INVALID_ARG;
  if ((flags & ~(OSCAR_PROBE_NONTEMPORAL | OSCAR_PROBE_WAVE_CHUNKS)) != 0)
    return OSCAR_ERR_INVALID_ARG;
  if (loads_per_thread != 4 && loads_per_thread != 8 && loads_per_thread != 16)
    return OSCAR_ERR_INVALID_ARG;
  const bool nt = (flags & OSCAR_PROBE_NONTEMPORAL) != 0;
  const bool chunk = (flags & OSCAR_PROBE_WAVE_CHUNKS) != 0;
  const auto* s = static_cast<const oscar::u4v*>(src);
  const size_t n = bytes / 16;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const dim3 grid((unsigned)blocks);
  if (loads_per_thread == 4) oscar::launch_u<4>(nt, chunk, grid, st, s, n, sink);
  else if (loads_per_thread == 8) oscar::launch_u<8>(nt, chunk, grid, st, s, n, sink);
  else oscar::launch_u<16>(nt, chunk, grid, st, s, n, sink);
  return hipGetLastError() == hipSuccess ? OSCAR_OK : OSCAR_ERR_HIP;
}

extern "C" int oscar_hbm_read_probe(const void* src, size_t bytes, uint32_t* sink, int32_t blocks,
                                    void* stream) {
  return oscar_hbm_read_probe_ex(src, bytes, sink, blocks, 4, 0, stream);
}
