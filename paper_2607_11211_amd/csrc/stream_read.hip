// Streaming read of device memory with 16-byte loads, plain or with the
// non-temporal cache policy: the measured HBM read rates next to which the
// layer's kernels are reported.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fasttps_probe.h"

namespace {

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256;

template <int U, bool NT>
__global__ __launch_bounds__(kThreads) void stream_read_kernel(const v4u* __restrict__ p, size_t n, unsigned* sink) {
  unsigned acc = 0;
  const size_t stride = (size_t)gridDim.x * kThreads * U;
  for (size_t i = (size_t)blockIdx.x * kThreads * U + threadIdx.x; i < n; i += stride) {
    v4u v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const size_t j = i + (size_t)u * kThreads;
      if constexpr (NT)
        v[u] = j < n ? __builtin_nontemporal_load(p + j) : v4u{0, 0, 0, 0};
      else
        v[u] = j < n ? p[j] : v4u{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (acc == 0x9E3779B9u) sink[threadIdx.x] = acc;
}

template <int U>
hipError_t launch(const void* src, size_t n, unsigned* sink, int blocks, bool nt, hipStream_t s) {
  if (nt)
    hipLaunchKernelGGL((stream_read_kernel<U, true>), dim3(blocks), dim3(kThreads), 0, s,
                       static_cast<const v4u*>(src), n, sink);
  else
    hipLaunchKernelGGL((stream_read_kernel<U, false>), dim3(blocks), dim3(kThreads), 0, s,
                       static_cast<const v4u*>(src), n, sink);
  return hipGetLastError();
}

}  // namespace

extern "C" int fasttps_probe_stream_read(const void* src, size_t bytes, void* sink, int blocks, int unroll,
                                         int nontemporal, void* stream, float* ms) {
  if (!src || !sink || !ms || bytes == 0 || bytes % 16 || reinterpret_cast<uintptr_t>(src) % 16 ||
      reinterpret_cast<uintptr_t>(sink) % 4 || blocks < 1 || blocks > 65536 ||
      !(unroll == 1 || unroll == 2 || unroll == 4 || unroll == 8) || (nontemporal != 0 && nontemporal != 1))
    return -1;
  const bool nt = nontemporal == 1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess) return -6;
  if (hipEventCreate(&e1) != hipSuccess) {
    (void)hipEventDestroy(e0);
    return -6;
  }
  const size_t n = bytes / 16;
  unsigned* k = static_cast<unsigned*>(sink);
  hipError_t err = hipEventRecord(e0, s);
  if (err == hipSuccess) {
    switch (unroll) {
      case 1: err = launch<1>(src, n, k, blocks, nt, s); break;
      case 2: err = launch<2>(src, n, k, blocks, nt, s); break;
      case 4: err = launch<4>(src, n, k, blocks, nt, s); break;
      default: err = launch<8>(src, n, k, blocks, nt, s); break;
    }
  }
  if (err == hipSuccess) err = hipEventRecord(e1, s);
  if (err == hipSuccess) err = hipEventSynchronize(e1);
  if (err == hipSuccess) err = hipEventElapsedTime(ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return err == hipSuccess ? 0 : -6;
}
