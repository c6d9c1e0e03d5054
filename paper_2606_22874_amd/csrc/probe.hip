// Streaming-read probe: the practical HBM read ceiling for 16-byte coalesced
// loads, measured with the same kind of loads the decode kernels issue.
#include "spot_internal.h"

namespace {

constexpr int kProbeWGs = 2048;
constexpr int kProbeThreads = 256;

__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const spot::u32x4* __restrict__ buf,
                                                                   size_t n16, float* __restrict__ sink) {
  uint32_t acc = 0;
  const size_t stride = (size_t)gridDim.x * kProbeThreads;
  size_t i = (size_t)blockIdx.x * kProbeThreads + threadIdx.x;
  // 4 independent loads in flight per thread per iteration.
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const spot::u32x4 a = __builtin_nontemporal_load(buf + i);
    const spot::u32x4 b = __builtin_nontemporal_load(buf + i + stride);
    const spot::u32x4 c = __builtin_nontemporal_load(buf + i + 2 * stride);
    const spot::u32x4 d = __builtin_nontemporal_load(buf + i + 3 * stride);
    acc ^= (a.x ^ a.y ^ a.z ^ a.w) ^ (b.x ^ b.y ^ b.z ^ b.w) ^ (c.x ^ c.y ^ c.z ^ c.w) ^
           (d.x ^ d.y ^ d.z ^ d.w);
  }
  for (; i < n16; i += stride) {
    const spot::u32x4 a = __builtin_nontemporal_load(buf + i);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  // One word per workgroup: xor over the wave, lane 0 of wave 0 writes.
  for (int off = 1; off < 64; off <<= 1) acc ^= (uint32_t)__shfl_xor((int)acc, off, 64);
  if (threadIdx.x == 0) sink[blockIdx.x] = __uint_as_float(acc & 0x3fffffffu);
}

}  // namespace

extern "C" {

int spot_probe_sink_words(void) { return kProbeWGs; }

spot_status spot_probe_stream_read(const void* buf, size_t bytes, float* sink, void* stream) {
  if (!buf || !sink) return SPOT_ERR_NULL;
  if (bytes % 16 || reinterpret_cast<uintptr_t>(buf) % 16) return SPOT_ERR_SHAPE;
  if (bytes == 0) return SPOT_OK;
  hipLaunchKernelGGL(stream_read_kernel, dim3(kProbeWGs), dim3(kProbeThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const spot::u32x4*>(buf),
                     bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? SPOT_OK : SPOT_ERR_HIP;
}

}  // extern "C"
