// Practical HBM ceiling for the benchmark: an in-place copy that reads and
// writes back every 16-byte piece of a buffer with non-temporal accesses,
// the same access kinds the state update uses on its tiles. Not part of the
// library's interface; built beside it for bench.py only.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Each thread moves U pieces per trip, spaced by the grid's thread count so
// that every wave instruction covers 1 KB of consecutive bytes; all loads of
// a trip are issued before its stores. `key` (0 from the host) keeps the
// stored data a function of the loaded data. The fastest copy keeps about
// 4 MB in flight (grid x 256 x U x 16 bytes).
template <int U>
__global__ __launch_bounds__(256) void copy_inplace_nt(u32x4* __restrict__ buf, size_t n16,
                                                       unsigned key) {
  const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
  size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  for (; i + (U - 1) * stride < n16; i += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(buf + i + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u) __builtin_nontemporal_store(v[u] ^ key, buf + i + u * stride);
  }
  for (; i < n16; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(buf + i) ^ key, buf + i);
}

}  // namespace

// bytes: a multiple of 16; buf 16-byte aligned; unroll 1, 2 or 4. Returns 0,
// or -1 for a bad argument, or the HIP error code of the launch.
extern "C" int copy_ceiling_inplace(void* buf, size_t bytes, int grid, int unroll, void* stream) {
  if (!buf || bytes % 16 != 0 || reinterpret_cast<uintptr_t>(buf) % 16 != 0 || grid <= 0)
    return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  u32x4* b = static_cast<u32x4*>(buf);
  const size_t n16 = bytes / 16;
  switch (unroll) {
    case 1: hipLaunchKernelGGL(copy_inplace_nt<1>, dim3(grid), dim3(256), 0, s, b, n16, 0u); break;
    case 2: hipLaunchKernelGGL(copy_inplace_nt<2>, dim3(grid), dim3(256), 0, s, b, n16, 0u); break;
    case 4: hipLaunchKernelGGL(copy_inplace_nt<4>, dim3(grid), dim3(256), 0, s, b, n16, 0u); break;
    default: return -1;
  }
  return static_cast<int>(hipGetLastError());
}
