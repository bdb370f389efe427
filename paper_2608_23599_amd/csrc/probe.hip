// Streaming-read probe: the HBM read rate a plain kernel reaches on this GPU, the
// second denominator beside the 8 TB/s peak for the decode kernels' achieved rates.
#include <hip/hip_runtime.h>

#include "gkv_internal.h"

namespace {

// Every workgroup reads its share of the buffer with 16-byte loads, four in flight
// per thread, and folds what it read into one word (so that no load can be dropped).
__global__ void __launch_bounds__(256) stream_read_kernel(const uint4 *__restrict__ src, int64_t n16,
                                                          uint32_t *__restrict__ sink) {
  uint32_t acc = 0;
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n16; i += stride) {
    const uint4 a = src[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  __shared__ uint32_t red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] ^= red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0];
}

}  // namespace

extern "C" gkv_status gkv_stream_read_probe(const void *src, int64_t bytes, uint32_t *sink, int32_t nsink,
                                            void *stream) {
  if (!src || !sink || bytes <= 0 || bytes % 16 || nsink <= 0) return GKV_E_ARG;
  if (((uintptr_t)src & 15) != 0) return GKV_E_ARG;
  hipLaunchKernelGGL(stream_read_kernel, dim3(nsink), dim3(256), 0, (hipStream_t)stream, (const uint4 *)src,
                     bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}
