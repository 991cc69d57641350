// Read-rate calibration: one pass over a device buffer with the load type of
// the HBM-bound kernels (16-byte non-temporal loads), eight loads in flight
// per lane, nothing else.  Not part of the method: the rate it reaches on a
// buffer of the decode's size is the practical read ceiling that the
// kernels' fractions of the 8 TB/s peak are set against.
#include <hip/hip_runtime.h>

#include "jfkv_internal.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kUnroll = 8;
constexpr int kThreads = 512;

// Block b reads the 16-byte vectors [b * chunk, min((b + 1) * chunk, n16)).
__global__ __launch_bounds__(kThreads) void read_stream_kernel(const u32x4* __restrict__ p,
                                                               size_t n16, size_t chunk,
                                                               uint32_t* __restrict__ sink) {
  const size_t lo = (size_t)blockIdx.x * chunk;
  const size_t hi = lo + chunk < n16 ? lo + chunk : n16;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (size_t i = lo + threadIdx.x; i < hi; i += (size_t)kThreads * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const size_t j = i + (size_t)u * kThreads;
      v[u] = j < hi ? __builtin_nontemporal_load(p + j) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u];
  }
  // (keeps the loads; true for no buffer the calibration fills)
  if (acc.x == 0x9E3779B9u && acc.y == 0x7F4A7C15u && acc.z == 0xF39CC060u) sink[0] = acc.w;
}

}  // namespace

namespace jfkv {

hipError_t launch_read_stream(const void* buf, size_t bytes, int32_t blocks, uint32_t* sink,
                              hipStream_t stream) {
  const size_t n16 = bytes / 16;
  const size_t chunk = (n16 + blocks - 1) / blocks;
  hipLaunchKernelGGL(read_stream_kernel, dim3(blocks), dim3(kThreads), 0, stream,
                     static_cast<const u32x4*>(buf), n16, chunk, sink);
  return hipGetLastError();
}

}  // namespace jfkv
