// libspdp_peak: a plain streaming-read kernel for gfx950, the measured read
// roof that the benchmark sets the spMspV kernel against (and a known-size
// reference for the hardware byte counters). Not part of the spMspV path.
//
//   int spdp_peak_read(const void* src, size_t bytes, unsigned* sink,
//                      int blocks, void* stream)
//
// Reads every byte of src (device, 16-byte aligned, bytes a multiple of 16)
// once with 16-byte vector loads, grid-stride over `blocks` workgroups of 256
// threads, four loads in flight per lane; each workgroup stores one word to
// sink[blockIdx.x] (device, `blocks` words) so that the loads are live.
// Enqueued on `stream` (hipStream_t); returns 0, or -1 for bad arguments,
// -4 if the launch fails.

#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

__global__ __launch_bounds__(256) void read_kernel(const uint4* __restrict__ src, size_t n16, unsigned* sink) {
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  unsigned acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc ^= (a.x ^ a.y ^ a.z ^ a.w) ^ (b.x ^ b.y ^ b.z ^ b.w) ^ (c.x ^ c.y ^ c.z ^ c.w) ^ (d.x ^ d.y ^ d.z ^ d.w);
  }
  for (; i < n16; i += stride) {
    const uint4 a = src[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  __shared__ unsigned red[4];
  for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

}  // namespace

extern "C" int spdp_peak_read(const void* src, size_t bytes, unsigned* sink, int blocks, void* stream) {
  if (!src || !sink || blocks < 1 || (bytes & 15) || (reinterpret_cast<uintptr_t>(src) & 15)) return -1;
  hipLaunchKernelGGL(read_kernel, dim3((unsigned)blocks), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const uint4*>(src), bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
