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
// a trip are issued before its stores. Loads are non-temporal, stores
// non-temporal at device (sc1) scope, as the update kernels' state accesses;
// this copy was 0.2 us faster with those stores than with plain
// non-temporal ones. `key` (0 from the host) keeps the stored data a function
// of the loaded data. The fastest copy keeps about 4 MB in flight (grid x
// 256 x U x 16 bytes).
constexpr int kLoadPolicy = 2, kStorePolicy = 2 | 16;

template <int U>
__global__ __launch_bounds__(256) void copy_inplace_nt(uint8_t* buf, uint32_t bytes, unsigned key) {
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(buf, 0, bytes, 0x00020000);
  const uint32_t stride = gridDim.x * blockDim.x * 16u;
  uint32_t i = (blockIdx.x * blockDim.x + threadIdx.x) * 16u;
  for (; i + (U - 1) * stride < bytes; i += U * stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      v[u] = __builtin_amdgcn_raw_buffer_load_b128(r, i + u * stride, 0, kLoadPolicy);
#pragma unroll
    for (int u = 0; u < U; ++u)
      __builtin_amdgcn_raw_buffer_store_b128(v[u] ^ key, r, i + u * stride, 0, kStorePolicy);
  }
  for (; i < bytes; i += stride)
    __builtin_amdgcn_raw_buffer_store_b128(
        __builtin_amdgcn_raw_buffer_load_b128(r, i, 0, kLoadPolicy) ^ key, r, i, 0, kStorePolicy);
}

}  // namespace

// bytes: a multiple of 16 below 2^31; buf 16-byte aligned; unroll 1, 2 or 4.
// Returns 0, or -1 for a bad argument, or the HIP error code of the launch.
extern "C" int copy_ceiling_inplace(void* buf, size_t bytes, int grid, int unroll, void* stream) {
  if (!buf || bytes % 16 != 0 || bytes >= (size_t(1) << 31) ||
      reinterpret_cast<uintptr_t>(buf) % 16 != 0 || grid <= 0)
    return -1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* b = static_cast<uint8_t*>(buf);
  const uint32_t n = static_cast<uint32_t>(bytes);
  switch (unroll) {
    case 1: hipLaunchKernelGGL(copy_inplace_nt<1>, dim3(grid), dim3(256), 0, s, b, n, 0u); break;
    case 2: hipLaunchKernelGGL(copy_inplace_nt<2>, dim3(grid), dim3(256), 0, s, b, n, 0u); break;
    case 4: hipLaunchKernelGGL(copy_inplace_nt<4>, dim3(grid), dim3(256), 0, s, b, n, 0u); break;
    default: return -1;
  }
  return static_cast<int>(hipGetLastError());
}
