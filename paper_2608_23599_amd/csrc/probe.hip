// Streaming-read probe: the HBM read rate a plain kernel reaches on this GPU, the
// second denominator beside the 8 TB/s peak for the decode kernels' achieved rates.
#include <hip/hip_runtime.h>

#include "gkv_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Every workgroup reads one contiguous share of the buffer with 16-byte nontemporal
// loads (each byte is read once, so it need not stay in the caches), eight in flight
// per thread, and folds what it read into one word (so that no load can be dropped).
// On gfx950 the nontemporal hint lifts a plain streaming read from about 6.2 to about
// 7.0 TB/s; the decode kernels issue their streaming loads with the same hint.
__global__ void __launch_bounds__(256) stream_read_kernel(const u32x4 *__restrict__ src, int64_t n16,
                                                          uint32_t *__restrict__ sink) {
  constexpr int U = 8;
  const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = lo + per < n16 ? lo + per : n16;
  uint32_t acc = 0;
  int64_t i = lo + threadIdx.x;
  for (; i + (U - 1) * 256 < hi; i += U * 256) {
    u32x4 a[U];
#pragma unroll
    for (int u = 0; u < U; ++u) a[u] = __builtin_nontemporal_load(src + i + u * 256);
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= a[u].x ^ a[u].y ^ a[u].z ^ a[u].w;
  }
  for (; i < hi; i += 256) {
    const u32x4 a = __builtin_nontemporal_load(src + i);
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
  hipLaunchKernelGGL(stream_read_kernel, dim3(nsink), dim3(256), 0, (hipStream_t)stream, (const u32x4 *)src,
                     bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? GKV_OK : GKV_E_HIP;
}
