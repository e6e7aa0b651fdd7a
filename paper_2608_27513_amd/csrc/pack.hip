// Pack, unpack and reset of packed pool tiles (section 5.2 and App. A.5,
// Eq. (17)): conversion between natural-order fp32 states and the persistent
// mixed-precision representation. Uses the same row encoder as the update.
#include "device.hpp"
#include "internal.hpp"

namespace damp {
namespace {

struct TileParams {
  uint8_t* layer_base;
  uint64_t slot_stride;
  uint64_t tile_stride;
  uint64_t layer_stride;
  const int32_t* slot_idx;
  const uint8_t* perm;
  float* S;          // [B, HV, D, D] natural order
  int32_t num_slots;
  int32_t HV;
  int32_t k_hi;
  int32_t had;  // block-32 Hadamard on the low tier (paper layout only)
};

template <int D>
struct Shape {
  static constexpr int NT = D >= 32 ? 2 * D : 64;
  static constexpr int CPT = D >= 32 ? 16 : 4;
  static constexpr int TPR = D / CPT;
  static constexpr int RG = NT / TPR;
  static constexpr int RPT = D / RG;
};

template <int KIND, int D>
__global__ __launch_bounds__(Shape<D>::NT) void pack_kernel(const TileParams p) {
  using Sh = Shape<D>;
  const int t = threadIdx.x, h = blockIdx.x, b = blockIdx.y;
  const int cg = t % Sh::TPR, rg = t / Sh::TPR, col0 = cg * Sh::CPT;
  const int slot = p.slot_idx[b];
  if (slot < 0 || slot >= p.num_slots) return;
  uint8_t* tile = p.layer_base + static_cast<size_t>(slot) * p.slot_stride +
                  static_cast<size_t>(h) * p.tile_stride;
  const int k_hi = KIND == kFp32 ? D : p.k_hi;
  uint8_t* codes = tile + static_cast<size_t>(k_hi) * D * 2;
  uint8_t* meta = codes + static_cast<size_t>(D - k_hi) * code_row_bytes<KIND, D>();
  const float* src = p.S + (static_cast<size_t>(b) * p.HV + h) * D * D;
  float s_g = 1.0f;
  if constexpr (KIND == kNvfp4) {  // the global scale of the tile's low tier
    float amax = 0.0f;
    for (int i = 0; i < Sh::RPT; ++i) {
      const int r = rg + Sh::RG * i;
      if (r < k_hi) continue;
      const int u = p.perm ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + r]) & (D - 1)) : r;
      for (int j = 0; j < Sh::CPT; ++j) amax = fmaxf(amax, fabsf(src[static_cast<size_t>(u) * D + col0 + j]));
    }
    s_g = nvfp4_global(block_max<Sh::NT>(amax));
    if (t == 0) store_global_scale<D>(meta, k_hi, s_g);
  }
  // every row slice of the thread is loaded before the first store: the
  // compiler cannot move a load of the state above a store into the tile
  // (the pointers may alias), so loading slot by slot would wait for the
  // memory once per slot
  float x[Sh::RPT][Sh::CPT];
#pragma unroll
  for (int i = 0; i < Sh::RPT; ++i) {
    const int r = rg + Sh::RG * i;
    const int u = p.perm ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + r]) & (D - 1)) : r;
    uint32_t w[Sh::CPT];
    load_words<Sh::CPT * 4>(reinterpret_cast<const uint8_t*>(src + static_cast<size_t>(u) * D + col0), w);
#pragma unroll
    for (int j = 0; j < Sh::CPT; ++j) x[i][j] = __uint_as_float(w[j]);
  }
#pragma unroll
  for (int i = 0; i < Sh::RPT; ++i)
    encode_row<KIND, D, Sh::CPT, Sh::TPR>(x[i], rg + Sh::RG * i, k_hi, cg, col0, tile, codes, meta,
                                          p.had != 0, s_g);
}

template <int KIND, int D>
__global__ __launch_bounds__(Shape<D>::NT) void unpack_kernel(const TileParams p) {
  using Sh = Shape<D>;
  // d = 128: per wave, its 8 rows of one row slot in transit to the stores
  __shared__ float ubuf[D == 128 ? Sh::NT / 64 : 1][D == 128 ? 8 * D : 1];
  const int t = threadIdx.x, h = blockIdx.x, b = blockIdx.y;
  const int cg = t % Sh::TPR, rg = t / Sh::TPR, col0 = cg * Sh::CPT;
  const int slot = p.slot_idx[b];
  float* dst = p.S + (static_cast<size_t>(b) * p.HV + h) * D * D;
  const bool live = slot >= 0 && slot < p.num_slots;
  const uint8_t* tile = p.layer_base + static_cast<size_t>(live ? slot : 0) * p.slot_stride +
                        static_cast<size_t>(h) * p.tile_stride;
  const int k_hi = KIND == kFp32 ? D : p.k_hi;
  const uint8_t* codes = tile + static_cast<size_t>(k_hi) * D * 2;
  const uint8_t* meta_bytes = codes + static_cast<size_t>(D - k_hi) * code_row_bytes<KIND, D>();
  const float2* meta = reinterpret_cast<const float2*>(meta_bytes);
  const uint32_t* meta16 = reinterpret_cast<const uint32_t*>(meta_bytes);
  // FP32 state and the default tiers: the bytes of every row slice are
  // loaded before the first store (the tile and the state may alias as far
  // as the compiler knows, so it would not move a later slot's loads above
  // an earlier slot's stores)
  constexpr bool kPre = KIND == kFp32 || KIND == kMixed;
  uint32_t pre[kPre ? Sh::RPT : 1][kPre ? Sh::CPT : 1];
  float2 presz[kPre ? Sh::RPT : 1];
  if constexpr (kPre) {
    if (live) {
#pragma unroll
      for (int i = 0; i < Sh::RPT; ++i) {
        const int r = rg + Sh::RG * i;
        if (KIND == kFp32) {
          load_words<Sh::CPT * 4>(tile + (static_cast<size_t>(r) * D + col0) * 4, pre[i]);
        } else if (r < k_hi) {
          load_words<Sh::CPT * 2>(tile + (static_cast<size_t>(r) * D + col0) * 2, pre[i]);
        } else {
          load_words<Sh::CPT>(codes + static_cast<size_t>(r - k_hi) * D + col0, pre[i]);
          presz[i] = meta[r - k_hi];
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < Sh::RPT; ++i) {
    const int r = rg + Sh::RG * i;
    const int u = p.perm ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + r]) & (D - 1)) : r;
    uint32_t out[Sh::CPT];
    if constexpr (KIND >= kInt4) {
      // FP16 rows; low rows as Eq. (16) or NVFP4 reconstruct (one product),
      // INT4 as s * (c - z) then the inverse transform
      float y[Sh::CPT];
      if (!live) {
#pragma unroll
        for (int j = 0; j < Sh::CPT; ++j) y[j] = 0.0f;
      } else if (r < k_hi) {
        decode_row<KIND, D, Sh::CPT>(tile, codes, meta_bytes, r, k_hi, cg, col0, false, y);
      } else if constexpr (KIND == kInt4) {
        const size_t l = static_cast<size_t>(r - k_hi);
        uint32_t w[2];
        load_words<8>(codes + l * code_row_bytes<KIND, D>() + col0 / 2, w);
        const uint32_t m = reinterpret_cast<const uint32_t*>(
            meta_bytes + l * meta_row_bytes<KIND, D>())[col0 >> 5];
        const float s16 = f16_lo(m), z16 = f16_hi(m);
#pragma unroll
        for (int j = 0; j < Sh::CPT; ++j)
          y[j] = __fmul_rn(s16, __fsub_rn(static_cast<float>((w[j >> 3] >> (4 * (j & 7))) & 0xfu), z16));
        if (p.had) {
          fwht32_pair(y, (cg & 1) != 0);
#pragma unroll
          for (int j = 0; j < Sh::CPT; ++j) y[j] *= kInvSqrt32;
        }
      } else {
        decode_row<KIND, D, Sh::CPT>(tile, codes, meta_bytes, r, k_hi, cg, col0, false, y);
      }
#pragma unroll
      for (int j = 0; j < Sh::CPT; ++j) out[j] = __float_as_uint(y[j]);
    } else if constexpr (KIND == kPaper) {
      // FP16 rows; low rows: s * (c - z) per group of 32, then the inverse
      // transform (the lane pair holds the group)
      float y[Sh::CPT];
      if (r < k_hi) {
        uint32_t w[Sh::CPT / 2];
        load_words<Sh::CPT * 2>(tile + (static_cast<size_t>(r) * D + col0) * 2, w);
#pragma unroll
        for (int j = 0; j < Sh::CPT / 2; ++j) {
          y[2 * j] = f16_lo(w[j]);
          y[2 * j + 1] = f16_hi(w[j]);
        }
      } else {
        uint32_t w[Sh::CPT / 4];
        load_words<Sh::CPT>(codes + static_cast<size_t>(r - k_hi) * D + col0, w);
        const uint32_t m = meta16[static_cast<size_t>(r - k_hi) * (D / 32) + (col0 >> 5)];
        const float s16 = f16_lo(m), z16 = f16_hi(m);
#pragma unroll
        for (int j = 0; j < Sh::CPT / 4; ++j) {
          y[4 * j + 0] = __fmul_rn(s16, __fsub_rn(ubyte<0>(w[j]), z16));
          y[4 * j + 1] = __fmul_rn(s16, __fsub_rn(ubyte<1>(w[j]), z16));
          y[4 * j + 2] = __fmul_rn(s16, __fsub_rn(ubyte<2>(w[j]), z16));
          y[4 * j + 3] = __fmul_rn(s16, __fsub_rn(ubyte<3>(w[j]), z16));
        }
        if (p.had) {
          fwht32_pair(y, (cg & 1) != 0);
#pragma unroll
          for (int j = 0; j < Sh::CPT; ++j) y[j] *= kInvSqrt32;
        }
      }
#pragma unroll
      for (int j = 0; j < Sh::CPT; ++j) out[j] = live ? __float_as_uint(y[j]) : 0u;
    } else if (!live) {
#pragma unroll
      for (int j = 0; j < Sh::CPT; ++j) out[j] = 0u;
    } else if (KIND == kFp32) {
#pragma unroll
      for (int j = 0; j < Sh::CPT; ++j) out[j] = pre[i][j];
    } else if (r < k_hi) {
      const uint32_t(&w)[Sh::CPT] = pre[i];
#pragma unroll
      for (int j = 0; j < Sh::CPT / 2; ++j) {
        out[2 * j] = w[j] << 16;
        out[2 * j + 1] = w[j] & 0xffff0000u;
      }
    } else {
      const uint32_t(&w)[Sh::CPT] = pre[i];
      const float2 sz = presz[i];
      // x_hat = s * (c - z), exactly as Eq. (3) reconstructs
#pragma unroll
      for (int j = 0; j < Sh::CPT / 4; ++j) {
        out[4 * j + 0] = __float_as_uint(__fmul_rn(sz.x, __fsub_rn(ubyte<0>(w[j]), sz.y)));
        out[4 * j + 1] = __float_as_uint(__fmul_rn(sz.x, __fsub_rn(ubyte<1>(w[j]), sz.y)));
        out[4 * j + 2] = __float_as_uint(__fmul_rn(sz.x, __fsub_rn(ubyte<2>(w[j]), sz.y)));
        out[4 * j + 3] = __float_as_uint(__fmul_rn(sz.x, __fsub_rn(ubyte<3>(w[j]), sz.y)));
      }
    }
    if constexpr (D == 128 && Sh::NT == 256) {
      // through the wave's LDS slice, so that every store instruction writes
      // two whole 512-byte rows: lane l writes 16 bytes at chunk l (+ 64 m)
      // of the wave's 8 rows of this slot
      const int lane = t & 63, wv = t >> 6;
      float4* rows = reinterpret_cast<float4*>(&ubuf[wv][0]);
#pragma unroll
      for (int k = 0; k < Sh::CPT / 4; ++k)
        rows[(rg & 7) * (D / 4) + cg * (Sh::CPT / 4) + k] =
            make_float4(__uint_as_float(out[4 * k]), __uint_as_float(out[4 * k + 1]),
                        __uint_as_float(out[4 * k + 2]), __uint_as_float(out[4 * k + 3]));
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const int c = lane + 64 * m;  // chunk: row c / 32 of the wave, columns 4 (c % 32) ..
        const int rr = 8 * wv + (c >> 5) + Sh::RG * i;
        const int uu =
            p.perm ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + rr]) & (D - 1)) : rr;
        *reinterpret_cast<float4*>(dst + static_cast<size_t>(uu) * D + 4 * (c & 31)) = rows[c];
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
    } else {
      store_words<Sh::CPT * 4>(reinterpret_cast<uint8_t*>(dst + static_cast<size_t>(u) * D + col0),
                               out);
    }
  }
}

// Packed zero state: zero high tier and codes, (s, z) = (1, 0) per row or group.
template <int KIND, int D>
__global__ __launch_bounds__(Shape<D>::NT) void reset_kernel(const TileParams p) {
  using Sh = Shape<D>;
  const int t = threadIdx.x, h = blockIdx.x, i_slot = blockIdx.y, layer = blockIdx.z;
  const int cg = t % Sh::TPR, rg = t / Sh::TPR, col0 = cg * Sh::CPT;
  const int slot = p.slot_idx[i_slot];
  if (slot < 0 || slot >= p.num_slots) return;
  uint8_t* tile = p.layer_base + static_cast<size_t>(layer) * p.layer_stride +
                  static_cast<size_t>(slot) * p.slot_stride + static_cast<size_t>(h) * p.tile_stride;
  const int k_hi = KIND == kFp32 ? D : p.k_hi;
  uint8_t* codes = tile + static_cast<size_t>(k_hi) * D * 2;
  uint8_t* meta = codes + static_cast<size_t>(D - k_hi) * code_row_bytes<KIND, D>();
  if constexpr (KIND == kNvfp4) {
    if (t == 0) store_global_scale<D>(meta, k_hi, nvfp4_global(0.0f));
  }
  float x[Sh::CPT];
#pragma unroll
  for (int j = 0; j < Sh::CPT; ++j) x[j] = 0.0f;
#pragma unroll
  for (int i = 0; i < Sh::RPT; ++i)
    encode_row<KIND, D, Sh::CPT, Sh::TPR>(x, rg + Sh::RG * i, k_hi, cg, col0, tile, codes, meta,
                                          p.had != 0);
}

enum class Op { kPack, kUnpack, kReset };

template <int KIND, int D>
void launch(Op op, const TileParams& p, dim3 grid, hipStream_t s) {
  const dim3 block(Shape<D>::NT);
  switch (op) {
    case Op::kPack: hipLaunchKernelGGL((pack_kernel<KIND, D>), grid, block, 0, s, p); break;
    case Op::kUnpack: hipLaunchKernelGGL((unpack_kernel<KIND, D>), grid, block, 0, s, p); break;
    case Op::kReset: hipLaunchKernelGGL((reset_kernel<KIND, D>), grid, block, 0, s, p); break;
  }
}

template <int KIND>
void launch_d(Op op, int D, const TileParams& p, dim3 grid, hipStream_t s) {
  switch (D) {
    case 16:
      if constexpr (KIND < kPaper) launch<KIND, 16>(op, p, grid, s);  // groups need d_v >= 32
      break;
    case 32: launch<KIND, 32>(op, p, grid, s); break;
    case 64: launch<KIND, 64>(op, p, grid, s); break;
    default: launch<KIND, 128>(op, p, grid, s); break;
  }
}

damp_status run(Op op, const char* name, const damp_pool* pool, int32_t layer,
                const int32_t* slot_idx, int32_t B, const uint8_t* perm, float* S,
                void* stream) {
  clear_error();
  damp_status st = check_pool(pool);
  if (st != DAMP_OK) return st;
  const bool all_layers = op == Op::kReset && layer == -1;
  if (!all_layers && (layer < 0 || layer >= pool->num_layers))
    return fail(DAMP_ERR_INVALID_ARG, "%s: layer %d outside [0, %d)", name, layer,
                pool->num_layers);
  if (B < 0 || B > 65535) return fail(DAMP_ERR_INVALID_ARG, "%s: count %d outside [0, 65535]", name, B);
  if (B == 0) return DAMP_OK;
  if (!slot_idx || (op != Op::kReset && !S))
    return fail(DAMP_ERR_INVALID_ARG, "%s: a required pointer is NULL", name);
  if (!layout_has_kernels(&pool->layout))
    return fail(DAMP_ERR_UNSUPPORTED, "%s: no kernel for this layout", name);
  if (op != Op::kUnpack) {
    st = debug_check_slots(pool, slot_idx, B, as_stream(stream), name);
    if (st != DAMP_OK) return st;
  }
  TileParams p;
  p.tile_stride = pool->tile_stride;
  p.slot_stride = pool->tile_stride * static_cast<uint64_t>(pool->num_v_heads);
  p.layer_stride = p.slot_stride * static_cast<uint64_t>(pool->num_slots);
  p.layer_base = layer_base(pool, all_layers ? 0 : layer);
  p.slot_idx = slot_idx;
  p.perm = perm;
  p.S = S;
  p.num_slots = pool->num_slots;
  p.HV = pool->num_v_heads;
  p.k_hi = pool->layout.kind == DAMP_STATE_FP32 ? 0 : pool->layout.k_hi;
  p.had = pool->layout.hadamard;
  const dim3 grid(pool->num_v_heads, B, all_layers ? pool->num_layers : 1);
  const int D = pool->layout.d_k;
  hipStream_t s = as_stream(stream);
  switch (layout_codec(&pool->layout)) {
    case kCodecFp32: launch_d<kFp32>(op, D, p, grid, s); break;
    case kCodecPaper: launch_d<kPaper>(op, D, p, grid, s); break;
    case kCodecInt4: launch_d<kInt4>(op, D, p, grid, s); break;
    case kCodecFp8: launch_d<kFp8>(op, D, p, grid, s); break;
    case kCodecNvfp4: launch_d<kNvfp4>(op, D, p, grid, s); break;
    default: launch_d<kMixed>(op, D, p, grid, s); break;
  }
  return check_launch(name);
}

}  // namespace
}  // namespace damp

extern "C" {

damp_status damp_state_pack(const damp_pool* pool, int32_t layer, const int32_t* slot_idx,
                            int32_t B, const float* S, const uint8_t* perm, void* stream) {
  return damp::run(damp::Op::kPack, "damp_state_pack", pool, layer, slot_idx, B, perm,
                   const_cast<float*>(S), stream);
}

damp_status damp_state_unpack(const damp_pool* pool, int32_t layer, const int32_t* slot_idx,
                              int32_t B, const uint8_t* perm, float* S_out, void* stream) {
  return damp::run(damp::Op::kUnpack, "damp_state_unpack", pool, layer, slot_idx, B, perm,
                   S_out, stream);
}

damp_status damp_pool_reset_slots(const damp_pool* pool, int32_t layer, const int32_t* slots,
                                  int32_t n, void* stream) {
  return damp::run(damp::Op::kReset, "damp_pool_reset_slots", pool, layer, slots, n, nullptr,
                   nullptr, stream);
}

}  // extern "C"
