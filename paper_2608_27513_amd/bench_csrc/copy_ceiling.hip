// Practical HBM ceilings for the benchmark: in-place copies that read and
// write back every 16-byte piece of a buffer (copy_inplace_nt), or of the
// tiles a decode step touches in the update's own order (copy_tiles_nt), with
// the access kinds the state update uses on its tiles. Not part of the
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

// The update's own walk over the pool, as an in-place copy: each of the
// `grid` workgroups (a multiple of HV) keeps one value head h = blockIdx mod
// HV and takes requests b = blockIdx / HV + k grid / HV, so at any moment the
// chip works on the same few dozen requests the update does, at the same
// slots. A tile (at most kMaxPieces x 4 KB) is read whole into registers,
// the next tile's loads are issued, and then it is written back; a padded
// slot (id < 0 or >= num_slots) gets a zero-size resource, so its accesses
// are dropped. Loads and stores carry the update's cache policies.
constexpr int kMaxPieces = 5;

__global__ __launch_bounds__(256) void copy_tiles_nt(uint8_t* base, const int32_t* slots, int B,
                                                     int HV, uint64_t slot_stride,
                                                     uint64_t tile_stride, uint32_t tile_bytes,
                                                     int num_slots, unsigned key) {
  const int h = blockIdx.x % HV;
  const int step = gridDim.x / HV;
  auto rsrc = [&](int b) {
    const int s = slots[b];
    const bool live = s >= 0 && s < num_slots;
    uint8_t* t = base + static_cast<uint64_t>(live ? s : 0) * slot_stride +
                 static_cast<uint64_t>(h) * tile_stride;
    return __builtin_amdgcn_make_buffer_rsrc(t, 0, live ? tile_bytes : 0u, 0x00020000);
  };
  const uint32_t off0 = threadIdx.x * 16u;
  int b = blockIdx.x / HV;
  if (b >= B) return;
  __amdgpu_buffer_rsrc_t rc = rsrc(b);
  u32x4 cur[kMaxPieces];
#pragma unroll
  for (int q = 0; q < kMaxPieces; ++q)
    cur[q] = __builtin_amdgcn_raw_buffer_load_b128(rc, off0 + q * 4096u, 0, kLoadPolicy);
  for (;;) {
    const int bn = b + step;
    u32x4 nxt[kMaxPieces];
    __amdgpu_buffer_rsrc_t rn = rc;
    if (bn < B) {
      rn = rsrc(bn);
#pragma unroll
      for (int q = 0; q < kMaxPieces; ++q)
        nxt[q] = __builtin_amdgcn_raw_buffer_load_b128(rn, off0 + q * 4096u, 0, kLoadPolicy);
    }
#pragma unroll
    for (int q = 0; q < kMaxPieces; ++q)
      __builtin_amdgcn_raw_buffer_store_b128(cur[q] ^ key, rc, off0 + q * 4096u, 0, kStorePolicy);
    if (bn >= B) break;
#pragma unroll
    for (int q = 0; q < kMaxPieces; ++q) cur[q] = nxt[q];
    rc = rn;
    b = bn;
  }
}

}  // namespace

// slots: device int32 [B]; tile_bytes: a multiple of 16, at most 20 480;
// grid: a positive multiple of HV. Returns 0, -1 for a bad argument, or the
// HIP error code of the launch.
extern "C" int copy_tiles_inplace(void* base, const int32_t* slots, int B, int HV,
                                  uint64_t slot_stride, uint64_t tile_stride, int tile_bytes,
                                  int num_slots, int grid, void* stream) {
  if (!base || !slots || B < 0 || HV <= 0 || tile_bytes <= 0 || tile_bytes % 16 != 0 ||
      tile_bytes > kMaxPieces * 4096 || grid <= 0 || grid % HV != 0 ||
      static_cast<uint64_t>(tile_bytes) > tile_stride || tile_stride * HV > slot_stride)
    return -1;
  if (B == 0) return 0;
  hipLaunchKernelGGL(copy_tiles_nt, dim3(grid), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<uint8_t*>(base), slots, B, HV, slot_stride, tile_stride,
                     static_cast<uint32_t>(tile_bytes), num_slots, 0u);
  return static_cast<int>(hipGetLastError());
}

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
