// HBM read-bandwidth probe: the ceiling against which the decode kernel's
// achieved bandwidth is reported. Not part of the attention method.
//
// Every byte of the buffer is read once with the same 16-byte non-temporal
// loads the decode kernel uses for K and V; each thread keeps kUnroll loads in
// flight. The XOR of everything read goes to sink[0] only when it equals a
// value the caller passes (so the loads cannot be elided, and the sink is
// normally left alone).
#include "resa_device.h"
#include "resa_internal.h"

namespace resa {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kUnroll = 8;

__global__ __launch_bounds__(kProbeThreads) void k_stream_read(const uint8_t* p, size_t n16,
                                                               uint32_t* sink, uint32_t match) {
  const size_t stride = (size_t)gridDim.x * kProbeThreads;
  size_t i = (size_t)blockIdx.x * kProbeThreads + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (kUnroll - 1) * stride < n16; i += kUnroll * stride) {
    U4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = ld16_stream(p + 16 * (i + u * stride));
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const U4 v = ld16_stream(p + 16 * i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == match) sink[0] = acc;
}

}  // namespace

hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, uint32_t match,
                              int32_t workgroups, hipStream_t stream) {
  hipLaunchKernelGGL(k_stream_read, dim3(workgroups), dim3(kProbeThreads), 0, stream,
                     static_cast<const uint8_t*>(buf), bytes / 16, sink, match);
  return hipGetLastError();
}

}  // namespace resa
