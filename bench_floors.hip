// Measurement floors for bench.py (not part of the inference library): a plain
// streaming read of a device buffer, the same read restricted to a given
// number of bytes, and an empty kernel. They give the achievable HBM read
// bandwidth and the fixed cost of one launch on the machine the benchmark
// runs on, reported beside the published peak.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

// Reads n 16-byte elements of src once (grid-stride) and writes one value per
// workgroup to sink[blockIdx.x], so the loads cannot be removed.
__global__ __launch_bounds__(256) void stream_read_kernel(const uint4* __restrict__ src,
                                                          int64_t n, float* __restrict__ sink) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^
           d.z ^ d.w;
  }
  for (; i < n; i += stride) {
    const uint4 a = src[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  __shared__ uint32_t red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t v = 0;
    for (int t = 0; t < 256; ++t) v ^= red[t];
    sink[blockIdx.x] = __uint_as_float(v & 0x3fffffffu);
  }
}

__global__ void empty_kernel() {}

}  // namespace

extern "C" {

// src: device buffer of n16 16-byte elements; sink: device buffer of at least
// `blocks` floats. Returns the hipError_t of the launch.
int floors_stream_read(const void* src, int64_t n16, float* sink, int blocks, hipStream_t stream) {
  if (!src || !sink || n16 < 0 || blocks < 1) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(256), 0, stream,
                     static_cast<const uint4*>(src), n16, sink);
  return (int)hipGetLastError();
}

int floors_empty(hipStream_t stream) {
  hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, stream);
  return (int)hipGetLastError();
}

}  // extern "C"
