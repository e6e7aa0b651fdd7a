// Fused decode-step state update for GDN and KDA heads on gfx950.
//
// One workgroup owns one (request, value head) tile and makes one pass over
// it in HBM: load the packed tile (dequantize), decay, key read-out and
// delta-rule residual, rank-1 update, read-out of o, re-encode in place
// (section 3.1 Eq. (1)-(2); section 3.2 Eq. (3); section 5.2 and App. A.5).
//
// Thread mapping (D = d_k = d_v, NT threads, CPT columns per thread): a row
// of the tile is split over TPR = D / CPT consecutive lanes, so a low-tier
// row slice is one 16-byte load of codes; row group rg = t / TPR handles rows
// rg, rg + RG, rg + 2 RG, ... (RPT rows per thread, RG = NT / TPR). With
// D = 128 and NT = 256 that is 4 rows x 16 columns = 64 state values per
// thread, all held in registers between the load and the store.
//
// The two key-axis reductions share one LDS pass: every thread writes its
// partial column sums of k~ . S_bar and q~ . S_bar, and thread t < 2D sums
// column t over the RG row groups. The output uses
//   o = scale (S_bar^T q~ + beta (q~ . k~) delta),
// which equals scale * S'^T q~ for the updated S' = S_bar + beta k~ delta^T,
// so no second reduction over S' is needed.
#include "device.hpp"
#include "internal.hpp"
#include "update.hpp"

namespace damp {
namespace {

__device__ __forceinline__ void write_o(const UpdateParams& p, size_t idx, float val) {
  if (p.o_bf16)
    static_cast<uint16_t*>(p.o)[idx] = f32_to_bf16(val);
  else
    static_cast<float*>(p.o)[idx] = val;
}

template <int KIND, bool KDA, int D, int NT, int CPT>
__global__ __launch_bounds__(NT) void update_kernel(const UpdateParams p) {
  constexpr int TPR = D / CPT;  // lanes per row
  constexpr int RG = NT / TPR;  // row groups
  constexpr int RPT = D / RG;   // rows per thread
  constexpr int EB = KIND == kFp32 ? 4 : 2;  // bytes per full-precision value
  static_assert(D % CPT == 0 && NT % TPR == 0 && D % RG == 0, "bad tiling");
  static_assert(NT >= 2 * D, "one reducing thread per output column");
  static_assert(TPR <= 16 && 64 % TPR == 0, "row lanes must sit in one DPP row");

  __shared__ float red[RG][2 * D];
  __shared__ float dsh[D];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int h = blockIdx.x;
  const int b = blockIdx.y;
  const int cg = t % TPR, rg = t / TPR, col0 = cg * CPT;
  const size_t bh = static_cast<size_t>(b) * p.HV + h;

  const int slot = p.slot_idx[b];
  if (slot < 0 || slot >= p.num_slots) {  // padded request: o = 0, state untouched
    for (int j = t; j < D; j += NT) write_o(p, bh * D + j, 0.0f);
    return;
  }

  uint8_t* tile = p.layer_base + static_cast<size_t>(slot) * p.slot_stride +
                  static_cast<size_t>(h) * p.tile_stride;
  const int k_hi = KIND == kFp32 ? D : p.k_hi;
  uint8_t* codes = tile + static_cast<size_t>(k_hi) * D * 2;
  uint8_t* meta_bytes = codes + static_cast<size_t>(D - k_hi) * code_row_bytes<KIND, D>();
  const float2* meta = reinterpret_cast<const float2*>(meta_bytes);
  // paper tiers: one word (FP16 s, FP16 z) per row and group of 32
  const uint32_t* meta16 = reinterpret_cast<const uint32_t*>(meta_bytes);

  // ---- issue the tile loads (the dominant HBM traffic) ---------------------
  uint32_t raw[RPT][CPT * EB / 4];
  float2 sz[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = rg + RG * i;
    if constexpr (KIND >= kInt4) {
      // the table formats decode through decode_row below
    } else if (r < k_hi) {
      load_words<CPT * EB>(tile + (static_cast<size_t>(r) * D + col0) * EB, raw[i]);
      sz[i] = make_float2(0.0f, 0.0f);
    } else {
      load_words<CPT>(codes + static_cast<size_t>(r - k_hi) * D + col0, raw[i]);
      if constexpr (KIND == kPaper) {
        const uint32_t m = meta16[static_cast<size_t>(r - k_hi) * (D / 32) + (col0 >> 5)];
        sz[i] = make_float2(f16_lo(m), f16_hi(m));
      } else {
        sz[i] = meta[r - k_hi];
      }
    }
  }

  // ---- operands in tile-row order (gathered through the permutation) ------
  const int hk = h / (p.HV / p.HK);
  const uint16_t* kb = p.k + (static_cast<size_t>(b) * p.HK + hk) * D;
  const uint16_t* qb = p.q + (static_cast<size_t>(b) * p.HK + hk) * D;
  const float beta = bf16_to_f32(p.beta[bh]);
  float alpha = 1.0f;
  if (!KDA) alpha = expf(bf16_to_f32(p.g[bh]));
  float kk[RPT], qq[RPT], aa[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = rg + RG * i;
    const int u = p.perm ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + r]) & (D - 1)) : r;
    kk[i] = bf16_to_f32(kb[u]);
    qq[i] = bf16_to_f32(qb[u]);
    aa[i] = KDA ? expf(bf16_to_f32(p.g[bh * D + u])) : alpha;
  }
  // q~ . k~ is permutation invariant: natural order, reduced over the wave.
  float qk = 0.0f;
  for (int e = lane; e < D; e += 64) qk = fmaf(bf16_to_f32(qb[e]), bf16_to_f32(kb[e]), qk);
  qk = wave_sum(qk);

  // ---- dequantize and decay: S_bar = Lambda S -----------------------------
  float x[RPT][CPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = rg + RG * i;
    if constexpr (KIND >= kInt4) {
      decode_row<KIND, D, CPT>(tile, codes, meta_bytes, r, k_hi, cg, col0, p.had != 0, x[i]);
#pragma unroll
      for (int j = 0; j < CPT; ++j) x[i][j] *= aa[i];
    } else if (r < k_hi) {
      if (KIND == kFp32) {
#pragma unroll
        for (int j = 0; j < CPT; ++j) x[i][j] = aa[i] * __uint_as_float(raw[i][j]);
      } else if (KIND == kPaper) {
#pragma unroll
        for (int j = 0; j < CPT / 2; ++j) {
          x[i][2 * j] = aa[i] * f16_lo(raw[i][j]);
          x[i][2 * j + 1] = aa[i] * f16_hi(raw[i][j]);
        }
      } else {
#pragma unroll
        for (int j = 0; j < CPT / 2; ++j) {
          x[i][2 * j] = aa[i] * bf16_lo(raw[i][j]);
          x[i][2 * j + 1] = aa[i] * bf16_hi(raw[i][j]);
        }
      }
    } else {
      // a * s * (c - z) as one FMA per value: (a s) c + (-(a s) z); with the
      // transform, its normalization folds into the same factor
      const float A = aa[i] * sz[i].x * ((KIND == kPaper && p.had) ? kInvSqrt32 : 1.0f);
      const float B0 = -A * sz[i].y;
#pragma unroll
      for (int j = 0; j < CPT / 4; ++j) {
        x[i][4 * j + 0] = fmaf(A, ubyte<0>(raw[i][j]), B0);
        x[i][4 * j + 1] = fmaf(A, ubyte<1>(raw[i][j]), B0);
        x[i][4 * j + 2] = fmaf(A, ubyte<2>(raw[i][j]), B0);
        x[i][4 * j + 3] = fmaf(A, ubyte<3>(raw[i][j]), B0);
      }
      if constexpr (KIND == kPaper) {
        if (p.had) fwht32_pair(reinterpret_cast<float(&)[16]>(x[i]), (cg & 1) != 0);
      }
    }
  }

  // ---- partial key and query read-outs over this thread's rows ------------
  {
    float pw[CPT], pq[CPT];
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
      pw[j] = kk[0] * x[0][j];
      pq[j] = qq[0] * x[0][j];
    }
#pragma unroll
    for (int i = 1; i < RPT; ++i)
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        pw[j] = fmaf(kk[i], x[i][j], pw[j]);
        pq[j] = fmaf(qq[i], x[i][j], pq[j]);
      }
#pragma unroll
    for (int j = 0; j < CPT; j += 4) {
      *reinterpret_cast<float4*>(&red[rg][col0 + j]) =
          make_float4(pw[j], pw[j + 1], pw[j + 2], pw[j + 3]);
      *reinterpret_cast<float4*>(&red[rg][D + col0 + j]) =
          make_float4(pq[j], pq[j + 1], pq[j + 2], pq[j + 3]);
    }
  }
  __syncthreads();

  // ---- column totals: w = S_bar^T k~ (t < D), S_bar^T q~ (D <= t < 2D) ----
  float tot = 0.0f;
  if (t < 2 * D) {
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int g = 0; g < RG; ++g) acc[g & 3] += red[g][t];
    tot = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  if (t < D) dsh[t] = bf16_to_f32(p.v[bh * D + t]) - tot;  // delta = v - S_bar^T k~
  __syncthreads();
  if (t >= D && t < 2 * D) {
    const int j = t - D;
    write_o(p, bh * D + j, p.scale * fmaf(beta * qk, dsh[j], tot));
  }

  // ---- rank-1 update S' = S_bar + beta k~ delta^T, re-encode, store -------
  float dl[CPT];
#pragma unroll
  for (int j = 0; j < CPT; j += 4) {
    const float4 d4 = *reinterpret_cast<const float4*>(&dsh[col0 + j]);
    dl[j] = d4.x;
    dl[j + 1] = d4.y;
    dl[j + 2] = d4.z;
    dl[j + 3] = d4.w;
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const float bk = beta * kk[i];
#pragma unroll
    for (int j = 0; j < CPT; ++j) x[i][j] = fmaf(bk, dl[j], x[i][j]);
  }
  float s_g = 1.0f;
  if constexpr (KIND == kNvfp4) {  // the global scale of the updated low tier
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < RPT; ++i)
      if (rg + RG * i >= k_hi)
#pragma unroll
        for (int j = 0; j < CPT; ++j) amax = fmaxf(amax, fabsf(x[i][j]));
    s_g = nvfp4_global(block_max<NT>(amax));
    if (t == 0) store_global_scale<D>(meta_bytes, k_hi, s_g);
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i)
    encode_row<KIND, D, CPT, TPR>(x[i], rg + RG * i, k_hi, cg, col0, tile, codes, meta_bytes,
                                  p.had != 0, s_g);
}

template <int KIND, bool KDA, int D>
void launch(const UpdateParams& p, int B, hipStream_t stream) {
  constexpr int NT = D >= 32 ? 2 * D : 64;
  constexpr int CPT = D >= 32 ? 16 : 4;
  hipLaunchKernelGGL((update_kernel<KIND, KDA, D, NT, CPT>), dim3(p.HV, B), dim3(NT), 0, stream,
                     p);
}

template <int KIND, bool KDA>
void launch_d(int D, const UpdateParams& p, int B, hipStream_t stream) {
  switch (D) {
    case 16:
      if constexpr (KIND < kPaper) launch<KIND, KDA, 16>(p, B, stream);  // groups need d_v >= 32
      break;
    case 32: launch<KIND, KDA, 32>(p, B, stream); break;
    case 64: launch<KIND, KDA, 64>(p, B, stream); break;
    default: launch<KIND, KDA, 128>(p, B, stream); break;
  }
}

template <bool KDA>
void launch_codec(int codec, int D, const UpdateParams& p, int B, hipStream_t s) {
  switch (codec) {
    case kCodecFp32: launch_d<kFp32, KDA>(D, p, B, s); break;
    case kCodecPaper: launch_d<kPaper, KDA>(D, p, B, s); break;
    case kCodecInt4: launch_d<kInt4, KDA>(D, p, B, s); break;
    case kCodecFp8: launch_d<kFp8, KDA>(D, p, B, s); break;
    case kCodecNvfp4: launch_d<kNvfp4, KDA>(D, p, B, s); break;
    default: launch_d<kMixed, KDA>(D, p, B, s); break;
  }
}

damp_status update(bool kda, const damp_pool* pool, int32_t layer, const int32_t* slot_idx,
                   int32_t B, int32_t num_k_heads, const uint16_t* q, const uint16_t* k,
                   const uint16_t* v, const uint16_t* g, const uint16_t* beta,
                   const uint8_t* perm, float scale, void* o, int32_t o_dtype, void* stream) {
  clear_error();
  const char* name = kda ? "damp_state_update_kda" : "damp_state_update_gdn";
  damp_status st = check_pool(pool);
  if (st != DAMP_OK) return st;
  if (layer < 0 || layer >= pool->num_layers)
    return fail(DAMP_ERR_INVALID_ARG, "%s: layer %d outside [0, %d)", name, layer,
                pool->num_layers);
  if (B < 0 || B > 65535) return fail(DAMP_ERR_INVALID_ARG, "%s: B = %d outside [0, 65535]", name, B);
  if (num_k_heads <= 0 || pool->num_v_heads % num_k_heads != 0)
    return fail(DAMP_ERR_INVALID_ARG, "%s: num_v_heads %d is not a multiple of num_k_heads %d",
                name, pool->num_v_heads, num_k_heads);
  if (o_dtype != DAMP_DT_FP32 && o_dtype != DAMP_DT_BF16)
    return fail(DAMP_ERR_INVALID_ARG, "%s: o_dtype must be FP32 or BF16", name);
  if (B == 0) return DAMP_OK;
  if (!slot_idx || !q || !k || !v || !g || !beta || !o)
    return fail(DAMP_ERR_INVALID_ARG, "%s: a required pointer is NULL", name);
  if (!layout_has_kernels(&pool->layout))
    return fail(DAMP_ERR_UNSUPPORTED, "%s: no kernel for this layout", name);
  st = debug_check_slots(pool, slot_idx, B, as_stream(stream), name);
  if (st != DAMP_OK) return st;

  UpdateParams p;
  p.layer_base = layer_base(pool, layer);
  p.tile_stride = pool->tile_stride;
  p.slot_stride = pool->tile_stride * static_cast<uint64_t>(pool->num_v_heads);
  p.slot_idx = slot_idx;
  p.q = q;
  p.k = k;
  p.v = v;
  p.g = g;
  p.beta = beta;
  p.perm = perm;
  p.o = o;
  p.scale = scale;
  p.num_slots = pool->num_slots;
  p.HK = num_k_heads;
  p.HV = pool->num_v_heads;
  p.k_hi = pool->layout.kind == DAMP_STATE_FP32 ? 0 : pool->layout.k_hi;
  p.o_bf16 = o_dtype == DAMP_DT_BF16;
  p.had = pool->layout.hadamard;
  const int D = pool->layout.d_k;
  hipStream_t s = as_stream(stream);
  // the persistent kernel numbers the B * HV tiles with 32-bit integers
  const bool tiles_fit = static_cast<int64_t>(B) * p.HV <= INT32_MAX;
  const int codec = layout_codec(&pool->layout);
  const int sfmt = codec == kCodecDefault ? kMixed
                   : codec == kCodecPaper ? kPaper
                   : codec == kCodecInt4  ? kInt4
                   : codec == kCodecFp8   ? kFp8
                   : codec == kCodecNvfp4 ? kNvfp4
                                          : -1;
  if (sfmt >= 0 && D == 128 && p.k_hi <= 32 && tiles_fit) {
    if (!launch_stream128(kda, sfmt, p, B, s))
      return fail(DAMP_ERR_HIP, "%s: occupancy query or launch failed", name);
    return check_launch(name);
  }
  if (codec == kCodecFp32 && D == 128) {
    launch_fp32_128(kda, p, B, s);
    return check_launch(name);
  }
  if (kda) launch_codec<true>(layout_codec(&pool->layout), D, p, B, s);
  else launch_codec<false>(layout_codec(&pool->layout), D, p, B, s);
  return check_launch(name);
}

}  // namespace
}  // namespace damp

extern "C" {

damp_status damp_state_update_gdn(const damp_pool* pool, int32_t layer, const int32_t* slot_idx,
                                  int32_t B, int32_t num_k_heads, const uint16_t* q,
                                  const uint16_t* k, const uint16_t* v, const uint16_t* g,
                                  const uint16_t* beta, const uint8_t* perm, float scale,
                                  void* o, int32_t o_dtype, void* stream) {
  return damp::update(false, pool, layer, slot_idx, B, num_k_heads, q, k, v, g, beta, perm,
                      scale, o, o_dtype, stream);
}

damp_status damp_state_update_kda(const damp_pool* pool, int32_t layer, const int32_t* slot_idx,
                                  int32_t B, int32_t num_k_heads, const uint16_t* q,
                                  const uint16_t* k, const uint16_t* v, const uint16_t* g,
                                  const uint16_t* beta, const uint8_t* perm, float scale,
                                  void* o, int32_t o_dtype, void* stream) {
  return damp::update(true, pool, layer, slot_idx, B, num_k_heads, q, k, v, g, beta, perm,
                      scale, o, o_dtype, stream);
}

}  // extern "C"
