// A plain streaming-read kernel: the HBM read rate a kernel that does
// nothing but read can reach on this GPU, the practical ceiling the decode
// kernels' achieved bandwidth is set against (next to the published 8 TB/s).
// Measurement tooling, built into its own library (libhbm_probe.so) and
// loaded only by the benchmark; not part of the decode-attention boundary.
//
//   int hbm_read_probe(const void* src, int64_t bytes, void* sink, int64_t sink_bytes,
//                      int workgroups, int nontemporal, hipStream_t stream);
//   int hbm_read_probe_waves(const void* src, int64_t bytes, void* sink, int64_t sink_bytes,
//                            int workgroups, int nontemporal, hipStream_t stream);
//
// Reads `bytes` (a multiple of 16) from device memory `src` with 16-byte
// vector loads by `workgroups` workgroups of 256 threads; with `nontemporal`
// the loads carry the nontemporal hint.  hbm_read_probe walks the buffer in
// grid-stride order, each thread four loads per step (the whole grid reads
// one front).  hbm_read_probe_waves gives each wave one contiguous region
// and sixteen loads per lane per step, the access pattern of the decode
// kernel, whose four waves each walk their own range of keys (bytes must be
// a multiple of workgroups x 4 x 16).  Every thread folds what it read into
// one 32-bit value and stores it to `sink` (device memory of at least
// workgroups x 256 x 4 bytes), so no load is dead.  Asynchronous on
// `stream`.  Returns 0, 1 for an invalid argument (checked before any
// device access), or the HIP error code of the launch.

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <bool NT>
__global__ __launch_bounds__(kThreads) void read_probe_kernel(const u32x4* __restrict__ src, int64_t n,
                                                              uint32_t* __restrict__ sink) {
  uint32_t acc = 0;
  const int64_t step = (int64_t)gridDim.x * kThreads * kUnroll;
  for (int64_t i = (int64_t)blockIdx.x * kThreads * kUnroll + threadIdx.x; i < n; i += step) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t j = i + (int64_t)kThreads * u;
      if (j < n)
        v[u] = NT ? __builtin_nontemporal_load(src + j) : src[j];
      else
        v[u] = u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  sink[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

// One contiguous region per wave, 16 loads in flight per lane.
template <bool NT>
__global__ __launch_bounds__(kThreads) void read_probe_waves_kernel(const u32x4* __restrict__ src, int64_t n,
                                                                    uint32_t* __restrict__ sink) {
  constexpr int kLoads = 16;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t per = n / ((int64_t)gridDim.x * (kThreads / 64));
  const int64_t b = ((int64_t)blockIdx.x * (kThreads / 64) + wave) * per, e = b + per;
  uint32_t acc = 0;
  for (int64_t i = b + lane; i < e; i += 64 * kLoads) {
    u32x4 v[kLoads];
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      const int64_t j = i + 64 * u;
      if (j < e)
        v[u] = NT ? __builtin_nontemporal_load(src + j) : src[j];
      else
        v[u] = u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kLoads; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  sink[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

}  // namespace

extern "C" int hbm_read_probe_waves(const void* src, int64_t bytes, void* sink, int64_t sink_bytes, int workgroups,
                                    int nontemporal, hipStream_t stream) {
  if (!src || !sink || bytes <= 0 || bytes % 16 != 0 || workgroups <= 0 || workgroups > (1 << 20) ||
      sink_bytes < (int64_t)workgroups * kThreads * 4 || (nontemporal != 0 && nontemporal != 1) ||
      (bytes / 16) % ((int64_t)workgroups * (kThreads / 64)) != 0)
    return 1;
  const int64_t n = bytes / 16;
  if (nontemporal)
    hipLaunchKernelGGL(read_probe_waves_kernel<true>, dim3(workgroups), dim3(kThreads), 0, stream,
                       static_cast<const u32x4*>(src), n, static_cast<uint32_t*>(sink));
  else
    hipLaunchKernelGGL(read_probe_waves_kernel<false>, dim3(workgroups), dim3(kThreads), 0, stream,
                       static_cast<const u32x4*>(src), n, static_cast<uint32_t*>(sink));
  return (int)hipGetLastError();
}

extern "C" int hbm_read_probe(const void* src, int64_t bytes, void* sink, int64_t sink_bytes, int workgroups,
                              int nontemporal, hipStream_t stream) {
  if (!src || !sink || bytes <= 0 || bytes % 16 != 0 || workgroups <= 0 || workgroups > (1 << 20) ||
      sink_bytes < (int64_t)workgroups * kThreads * 4 || (nontemporal != 0 && nontemporal != 1))
    return 1;
  const int64_t n = bytes / 16;
  if (nontemporal)
    hipLaunchKernelGGL(read_probe_kernel<true>, dim3(workgroups), dim3(kThreads), 0, stream,
                       static_cast<const u32x4*>(src), n, static_cast<uint32_t*>(sink));
  else
    hipLaunchKernelGGL(read_probe_kernel<false>, dim3(workgroups), dim3(kThreads), 0, stream,
                       static_cast<const u32x4*>(src), n, static_cast<uint32_t*>(sink));
  return (int)hipGetLastError();
}
