// Streaming-read probe for gfx950: a plain pass over a buffer with 16-byte
// non-temporal loads (the attention kernels' load type), grid-stride, four
// loads in flight per thread.  Its rate is the box's practical HBM read
// ceiling, against which the attention kernels' achieved bandwidth is read.
// Each workgroup writes the XOR of the 32-bit words it read (so the loads
// cannot be dropped, and a test can check the pass covered every word).

#include "../../include/wmtp.h"
#include "common.h"
#include "launch.h"

namespace wmtp {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 4;

__global__ __launch_bounds__(kProbeThreads) void hbm_read_kernel(const u32x4* __restrict__ p, int64_t n_vec,
                                                                 uint32_t* sink) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kProbeThreads;
  int64_t i = static_cast<int64_t>(blockIdx.x) * kProbeThreads + threadIdx.x;
  uint32_t acc = 0;
  for (; i + (kProbeUnroll - 1) * stride < n_vec; i += kProbeUnroll * stride) {
    u32x4 v[kProbeUnroll];
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n_vec; i += stride) {
    const u32x4 v = __builtin_nontemporal_load(p + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off);
  __shared__ uint32_t s_acc[kProbeThreads / kWave];
  const int lane = threadIdx.x & (kWave - 1);
  if (lane == 0) s_acc[threadIdx.x / kWave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t r = 0;
#pragma unroll
    for (int w = 0; w < kProbeThreads / kWave; ++w) r ^= s_acc[w];
    sink[blockIdx.x] = r;
  }
}

}  // namespace

hipError_t launch_hbm_read(const void* buf, int64_t bytes, uint32_t* sink, hipStream_t stream) {
  hipLaunchKernelGGL(hbm_read_kernel, dim3(WMTP_PROBE_BLOCKS), dim3(kProbeThreads), 0, stream,
                     static_cast<const u32x4*>(buf), bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace wmtp
