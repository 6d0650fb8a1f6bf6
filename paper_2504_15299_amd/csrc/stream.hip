// Measurement helper: the HBM read ceiling of this GPU, measured with the
// simplest kernel that streams a buffer once (16-byte nontemporal loads, a
// grid-stride loop, nothing else).  The expert kernels' achieved bandwidth is
// reported next to it.
#include "internal.h"

namespace d2moe {
namespace {

constexpr int kStreamThreads = 256;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline uint32_t fold(u32x4 v) { return v.x ^ v.y ^ v.z ^ v.w; }

// Each thread reads 16-byte words i, i + stride, ... of the buffer and folds
// them into an XOR that it writes once per workgroup, so the loads cannot be
// removed.  n16 = number of 16-byte words; sink has one word per workgroup.
__global__ __launch_bounds__(kStreamThreads) void stream_read_kernel(
    const u32x4* __restrict__ buf, size_t n16, uint32_t* __restrict__ sink) {
  __shared__ uint32_t part[kStreamThreads / 64];
  const size_t stride = (size_t)gridDim.x * kStreamThreads;
  uint32_t acc = 0;
  size_t i = (size_t)blockIdx.x * kStreamThreads + threadIdx.x;
  // four loads in flight per thread per iteration
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 a = __builtin_nontemporal_load(buf + i);
    const u32x4 b = __builtin_nontemporal_load(buf + i + stride);
    const u32x4 c = __builtin_nontemporal_load(buf + i + 2 * stride);
    const u32x4 d = __builtin_nontemporal_load(buf + i + 3 * stride);
    acc ^= fold(a) ^ fold(b) ^ fold(c) ^ fold(d);
  }
  for (; i < n16; i += stride) {
    acc ^= fold(__builtin_nontemporal_load(buf + i));
  }
  for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

}  // namespace

hipError_t launch_stream_read(const void* buf, size_t bytes, uint32_t* sink, int blocks,
                              hipStream_t s) {
  stream_read_kernel<<<blocks, kStreamThreads, 0, s>>>((const u32x4*)buf, bytes / 16, sink);
  return hipGetLastError();
}

}  // namespace d2moe
