// A measurement reference, not part of the product: one launch that streams
// a device buffer (include/celty_bench.h).  The benchmark times it on the
// byte count of a product's call to show what the memory system gives a
// single launch of that size.

#include <hip/hip_runtime.h>

#include <cstdint>

#include "celty_bench.h"

namespace {

typedef unsigned v4u __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(1024) void stream_read_kernel(const v4u* __restrict__ p, size_t n16, uint32_t* sink) {
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  unsigned acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {   // four 16-byte loads in flight per lane
    const v4u a = __builtin_nontemporal_load(p + i);
    const v4u b = __builtin_nontemporal_load(p + i + stride);
    const v4u c = __builtin_nontemporal_load(p + i + 2 * stride);
    const v4u d = __builtin_nontemporal_load(p + i + 3 * stride);
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n16; i += stride) {
    const v4u a = __builtin_nontemporal_load(p + i);
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  __shared__ unsigned word;
  if (threadIdx.x == 0) word = 0u;
  __syncthreads();
  atomicXor(&word, acc);
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = word;
}

}  // namespace

extern "C" celty_status celty_bench_stream_read(const void* p, size_t bytes, uint32_t* sink, int32_t blocks,
                                                int32_t threads, void* stream) {
  if (!sink || (reinterpret_cast<uintptr_t>(sink) & 3u)) return CELTY_EINVAL;
  if (bytes % 16 != 0 || (bytes > 0 && (!p || (reinterpret_cast<uintptr_t>(p) & 15u)))) return CELTY_EINVAL;
  if (blocks < 1 || blocks > 65535 || threads < 64 || threads > 1024 || threads % 64 != 0) return CELTY_EINVAL;
  hipLaunchKernelGGL(stream_read_kernel, dim3(static_cast<unsigned>(blocks)), dim3(static_cast<unsigned>(threads)), 0,
                     static_cast<hipStream_t>(stream), static_cast<const v4u*>(p), bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? CELTY_OK : CELTY_EHIP;
}
