// HBM read stream: reads a device buffer once, as fast as the device allows,
// to measure the practical read-bandwidth ceiling that the decode kernels'
// achieved bandwidth is reported against (next to the published peak).
//
// Every load instruction of a wave reads one whole kilobyte (64 lanes x 16
// consecutive bytes), nontemporal: the stream is read once and every line it
// touches is consumed by a single instruction, the access pattern for which
// that hint pays.  Each thread keeps kStUnroll loads in flight per round.
#include "entry.h"
#include "internal.h"

namespace dwkv {
namespace {

typedef uint32_t u4v __attribute__((ext_vector_type(4)));

constexpr int kStThreads = 256;
constexpr int kStUnroll = 8;

// Block b reads rounds b, b + grid, b + 2 grid, ... of kStThreads * kStUnroll
// consecutive 16-byte words and writes the xor of every 32-bit word it read
// to sink[b]: the xor over the sink is the xor over the buffer.
__global__ __launch_bounds__(kStThreads) void stream_read_kernel(const u4v* __restrict__ p, uint64_t n16,
                                                                 uint32_t* __restrict__ sink) {
  constexpr uint64_t kRound = (uint64_t)kStThreads * kStUnroll;
  const uint64_t step = (uint64_t)gridDim.x * kRound;
  uint32_t acc = 0;
  for (uint64_t base = (uint64_t)blockIdx.x * kRound; base < n16; base += step) {
    u4v v[kStUnroll];
#pragma unroll
    for (int u = 0; u < kStUnroll; ++u) {
      const uint64_t i = base + (uint64_t)u * kStThreads + threadIdx.x;
      v[u] = i < n16 ? __builtin_nontemporal_load(p + i) : u4v{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kStUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o);
  __shared__ uint32_t wx[kStThreads / 64];
  if ((threadIdx.x & 63) == 0) wx[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t a = 0;
#pragma unroll
    for (int i = 0; i < kStThreads / 64; ++i) a ^= wx[i];
    sink[blockIdx.x] = a;
  }
}

}  // namespace

hipError_t launch_stream_read(const void* buf, uint64_t n16, uint32_t* sink, hipStream_t s) {
  hipLaunchKernelGGL(stream_read_kernel, dim3(kStreamBlocks), dim3(kStThreads), 0, s,
                     static_cast<const u4v*>(buf), n16, sink);
  return hipGetLastError();
}

}  // namespace dwkv
