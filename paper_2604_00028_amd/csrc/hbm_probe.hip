// A plain streaming-read kernel: the HBM read rate a kernel that does
// nothing but read can reach on this GPU, the practical ceiling the decode
// kernels' achieved bandwidth is set against (next to the published 8 TB/s).
// Measurement tooling, built into its own library (libhbm_probe.so) and
// loaded only by the benchmark; not part of the decode-attention boundary.
//
//   int hbm_read_probe(const void* src, int64_t bytes, void* sink, int64_t sink_bytes,
//                      int workgroups, int loads, int nontemporal, hipStream_t stream);
//   int hbm_read_probe_waves(const void* src, int64_t bytes, void* sink, int64_t sink_bytes,
//                            int workgroups, int loads, int nontemporal, hipStream_t stream);
//
// Reads `bytes` (a multiple of 16) from device memory `src` with 16-byte
// vector loads by `workgroups` workgroups of 256 threads; with `nontemporal`
// the loads carry the nontemporal hint.  hbm_read_probe walks the buffer in
// grid-stride order, each thread `loads` loads per step (4, 8 or 16): the
// whole grid reads one front.  hbm_read_probe_waves gives each wave one
// contiguous region and `loads` loads per lane per step (8 or 16), the
// access pattern of the decode kernel, whose waves each walk their own range
// of keys (bytes must be a multiple of workgroups x 4 x 16).  Every thread
// folds what it read into one 32-bit value and stores it to `sink` (device
// memory of at least workgroups x 256 x 4 bytes), so no load is dead.
// Asynchronous on `stream`.  Returns 0, 1 for an invalid argument (checked
// before any device access), or the HIP error code of the launch.

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 256;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ u32x4 load16(const u32x4* p) {
  return NT ? __builtin_nontemporal_load(p) : *p;
}

template <int U, bool NT>
__global__ __launch_bounds__(kThreads) void read_probe_kernel(const u32x4* __restrict__ src, int64_t n,
                                                              uint32_t* __restrict__ sink) {
  uint32_t acc = 0;
  const int64_t step = (int64_t)gridDim.x * kThreads * U;
  for (int64_t i = (int64_t)blockIdx.x * kThreads * U + threadIdx.x; i < n; i += step) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = i + (int64_t)kThreads * u;
      v[u] = j < n ? load16<NT>(src + j) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  sink[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

// One contiguous region per wave, U loads in flight per lane.
template <int U, bool NT>
__global__ __launch_bounds__(kThreads) void read_probe_waves_kernel(const u32x4* __restrict__ src, int64_t n,
                                                                    uint32_t* __restrict__ sink) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t per = n / ((int64_t)gridDim.x * (kThreads / 64));
  const int64_t b = ((int64_t)blockIdx.x * (kThreads / 64) + wave) * per, e = b + per;
  uint32_t acc = 0;
  for (int64_t i = b + lane; i < e; i += 64 * U) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t j = i + 64 * u;
      v[u] = j < e ? load16<NT>(src + j) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  sink[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

template <int U, bool NT>
void launch_gs(int wgs, hipStream_t st, const u32x4* s, int64_t n, uint32_t* o) {
  hipLaunchKernelGGL((read_probe_kernel<U, NT>), dim3(wgs), dim3(kThreads), 0, st, s, n, o);
}

template <int U, bool NT>
void launch_waves(int wgs, hipStream_t st, const u32x4* s, int64_t n, uint32_t* o) {
  hipLaunchKernelGGL((read_probe_waves_kernel<U, NT>), dim3(wgs), dim3(kThreads), 0, st, s, n, o);
}

bool common_args_ok(const void* src, int64_t bytes, const void* sink, int64_t sink_bytes, int workgroups,
                    int nontemporal) {
  return src && sink && bytes > 0 && bytes % 16 == 0 && workgroups > 0 && workgroups <= (1 << 20) &&
         sink_bytes >= (int64_t)workgroups * kThreads * 4 && (nontemporal == 0 || nontemporal == 1);
}

}  // namespace

extern "C" int hbm_read_probe(const void* src, int64_t bytes, void* sink, int64_t sink_bytes, int workgroups,
                              int loads, int nontemporal, hipStream_t stream) {
  if (!common_args_ok(src, bytes, sink, sink_bytes, workgroups, nontemporal) ||
      (loads != 4 && loads != 8 && loads != 16))
    return 1;
  const int64_t n = bytes / 16;
  auto* s = static_cast<const u32x4*>(src);
  auto* o = static_cast<uint32_t*>(sink);
  if (nontemporal) {
    if (loads == 4) launch_gs<4, true>(workgroups, stream, s, n, o);
    else if (loads == 8) launch_gs<8, true>(workgroups, stream, s, n, o);
    else launch_gs<16, true>(workgroups, stream, s, n, o);
  } else {
    if (loads == 4) launch_gs<4, false>(workgroups, stream, s, n, o);
    else if (loads == 8) launch_gs<8, false>(workgroups, stream, s, n, o);
    else launch_gs<16, false>(workgroups, stream, s, n, o);
  }
  return (int)hipGetLastError();
}

extern "C" int hbm_read_probe_waves(const void* src, int64_t bytes, void* sink, int64_t sink_bytes, int workgroups,
                                    int loads, int nontemporal, hipStream_t stream) {
  if (!common_args_ok(src, bytes, sink, sink_bytes, workgroups, nontemporal) || (loads != 8 && loads != 16) ||
      (bytes / 16) % ((int64_t)workgroups * (kThreads / 64)) != 0)
    return 1;
  const int64_t n = bytes / 16;
  auto* s = static_cast<const u32x4*>(src);
  auto* o = static_cast<uint32_t*>(sink);
  if (nontemporal) {
    if (loads == 8) launch_waves<8, true>(workgroups, stream, s, n, o);
    else launch_waves<16, true>(workgroups, stream, s, n, o);
  } else {
    if (loads == 8) launch_waves<8, false>(workgroups, stream, s, n, o);
    else launch_waves<16, false>(workgroups, stream, s, n, o);
  }
  return (int)hipGetLastError();
}
