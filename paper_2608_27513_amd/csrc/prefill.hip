// Prefill of one chunk of tokens per request into the packed pool (App. A.5,
// prefill path; section 3.1 Eq. (1)).
//
// One workgroup owns one (request, value head) tile: it decodes the stored
// state once into registers, runs the recurrence of Eq. (1) in fp32 for the
// chunk's T tokens (emitting o for every token), and re-encodes only the
// chunk-final state. The thread mapping is that of the decode update: a row
// of the tile is split over TPR lanes, each holding CPT columns of RPT rows.
//
// Per token, threads t < d_k stage the token's operands (k~, q~ gathered
// through the permutation, the row decay, v) in LDS, double-buffered: the
// next token's operands are loaded into registers while the current token
// computes. Both key-axis reductions share one LDS pass, and
//   o = scale (S_bar^T q~ + beta (q~ . k~) delta)
// equals scale * S^T q~ for the updated state S.
#include <climits>

#include "device.hpp"
#include "internal.hpp"

namespace damp {
namespace {

struct PrefillParams {
  uint8_t* layer_base;
  uint64_t slot_stride;
  uint64_t tile_stride;
  const int32_t* slot_idx;
  const uint16_t* q;  // [B, t_pitch, HK, D]
  const uint16_t* k;
  const uint16_t* v;  // [B, t_pitch, HV, D]
  const uint16_t* g;  // [B, t_pitch, HV] or [B, t_pitch, HV, D]
  const uint16_t* beta;  // [B, t_pitch, HV]
  const uint8_t* perm;
  void* o;  // [B, T, HV, D], or NULL: no outputs
  float scale;
  int32_t T;        // tokens run by this launch
  int32_t t_pitch;  // tokens per request in the input arrays
  int32_t t0;       // first input token of this launch
  int32_t num_slots;
  int32_t HK;
  int32_t HV;
  int32_t k_hi;
  int32_t o_bf16;
  int32_t had;
};

struct TokRegs {
  uint32_t k = 0u, q = 0u, g = 0u, v = 0u, beta = 0u;
};

template <int KIND, bool KDA, int D, int NT, int CPT>
__global__ __launch_bounds__(NT) void prefill_kernel(const PrefillParams p) {
  constexpr int TPR = D / CPT;  // lanes per row
  constexpr int RG = NT / TPR;  // row groups
  constexpr int RPT = D / RG;   // rows per thread
  constexpr int NQK = (D + 63) / 64;  // waves holding operand rows
  static_assert(NT >= 2 * D, "one reducing thread per output column");

  __shared__ float red[RG][2 * D];
  __shared__ float dsh[D];
  __shared__ float4 opr[2][D];   // per token parity, row r: (k~_r, q~_r, a~_r, v_r)
  __shared__ float opsc[2][4];   // per token parity: beta, alpha (GDN), partial sums of q~ . k~

  const int t = threadIdx.x;
  const int h = blockIdx.x;
  const int b = blockIdx.y;
  const int cg = t % TPR, rg = t / TPR, col0 = cg * CPT;
  const int T = p.T;
  const int hk = h / (p.HV / p.HK);
  const int o_esize = p.o_bf16 ? 2 : 4;
  auto o_at = [&](int tok, int j) {
    return static_cast<uint8_t*>(p.o) +
           ((static_cast<size_t>(b) * T + tok) * p.HV + h) * D * o_esize +
           static_cast<size_t>(j) * o_esize;
  };
  auto write_o = [&](int tok, int j, float val) {
    if (!p.o) return;
    if (p.o_bf16) *reinterpret_cast<uint16_t*>(o_at(tok, j)) = f32_to_bf16(val);
    else *reinterpret_cast<float*>(o_at(tok, j)) = val;
  };

  const int slot = p.slot_idx[b];
  if (slot < 0 || slot >= p.num_slots) {  // padded request: o = 0, state untouched
    for (int tok = 0; tok < T; ++tok)
      for (int j = t; j < D; j += NT) write_o(tok, j, 0.0f);
    return;
  }
  uint8_t* tile = p.layer_base + static_cast<size_t>(slot) * p.slot_stride +
                  static_cast<size_t>(h) * p.tile_stride;
  const int k_hi = KIND == kFp32 ? D : p.k_hi;
  uint8_t* codes = tile + static_cast<size_t>(k_hi) * D * 2;
  uint8_t* meta_bytes = codes + static_cast<size_t>(D - k_hi) * code_row_bytes<KIND, D>();
  const bool had = p.had != 0;

  // ---- decode the stored state once
  float x[RPT][CPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i)
    decode_row<KIND, D, CPT>(tile, codes, meta_bytes, rg + RG * i, k_hi, cg, col0, had, x[i]);

  // ---- operands of one token, gathered by threads t < D
  const int my_u = (t < D && p.perm) ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + t]) & (D - 1)) : t;
  auto load_tok = [&](TokRegs& r, int tok) {
    if (t < D) {
      const size_t bt = static_cast<size_t>(b) * p.t_pitch + p.t0 + tok;
      const size_t kq = (bt * p.HK + hk) * D;
      const size_t bth = bt * p.HV + h;
      r.k = p.k[kq + my_u];
      r.q = p.q[kq + my_u];
      r.g = KDA ? p.g[bth * D + my_u] : p.g[bth];
      r.v = p.v[bth * D + t];
      r.beta = p.beta[bth];
    }
  };
  auto publish = [&](const TokRegs& r, int par) {
    float kq = 0.0f;
    float gf = 0.0f;
    if (t < D) {
      const float kf = bf16_to_f32(static_cast<uint16_t>(r.k));
      const float qf = bf16_to_f32(static_cast<uint16_t>(r.q));
      gf = bf16_to_f32(static_cast<uint16_t>(r.g));
      opr[par][t] = make_float4(kf, qf, KDA ? __expf(gf) : 1.0f,
                                bf16_to_f32(static_cast<uint16_t>(r.v)));
      kq = kf * qf;
    }
    if (t < 64 * NQK) {  // whole waves, lanes past D contribute 0
      kq = wave_sum_dpp(kq);
      if ((t & 63) == 0) opsc[par][2 + (t >> 6)] = kq;
    }
    if (t == 0) {
      opsc[par][0] = bf16_to_f32(static_cast<uint16_t>(r.beta));
      opsc[par][1] = KDA ? 1.0f : __expf(gf);
      if (NQK == 1) opsc[par][3] = 0.0f;
    }
  };

  TokRegs cur, nxt;
  if (T > 0) {
    load_tok(cur, 0);
    publish(cur, 0);
  }
  __syncthreads();

  for (int tok = 0; tok < T; ++tok) {
    const int par = tok & 1;
    if (tok + 1 < T) load_tok(nxt, tok + 1);
    // -- decay S_bar = Lambda S, partial read-outs over this thread's rows
    float kk[RPT];
    {
      const float alpha = opsc[par][1];
      float qq[RPT];
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        const float4 o4 = opr[par][rg + RG * i];
        kk[i] = o4.x;
        qq[i] = o4.y;
        const float a = KDA ? o4.z : alpha;
#pragma unroll
        for (int j = 0; j < CPT; ++j) x[i][j] *= a;
      }
#pragma unroll
      for (int j = 0; j < CPT; ++j) {
        float pw = kk[0] * x[0][j], pq = qq[0] * x[0][j];
#pragma unroll
        for (int i = 1; i < RPT; ++i) {
          pw = fmaf(kk[i], x[i][j], pw);
          pq = fmaf(qq[i], x[i][j], pq);
        }
        red[rg][col0 + j] = pw;
        red[rg][D + col0 + j] = pq;
      }
    }
    __syncthreads();
    // -- column totals: w = S_bar^T k~ (t < D), S_bar^T q~ (D <= t < 2D)
    float tot = 0.0f;
    if (t < 2 * D) {
      float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int gg = 0; gg < RG; ++gg) acc[gg & 3] += red[gg][t];
      tot = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    }
    if (t < D) dsh[t] = opr[par][t].w - tot;  // delta = v - S_bar^T k~
    if (tok + 1 < T) publish(nxt, par ^ 1);
    __syncthreads();
    const float beta = opsc[par][0], qk = opsc[par][2] + opsc[par][3];
    if (t >= D && t < 2 * D) write_o(tok, t - D, p.scale * fmaf(beta * qk, dsh[t - D], tot));
    // -- rank-1 update S = S_bar + beta k~ delta^T
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const float bk = beta * kk[i];
#pragma unroll
      for (int j = 0; j < CPT; ++j) x[i][j] = fmaf(bk, dsh[col0 + j], x[i][j]);
    }
  }

  // ---- store the chunk-final state per its tier
  float s_g = 1.0f;
  if constexpr (KIND == kNvfp4) {  // the global scale of the final low tier
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
    encode_row<KIND, D, CPT, TPR>(x[i], rg + RG * i, k_hi, cg, col0, tile, codes, meta_bytes, had,
                                  s_g);
}

template <int KIND, bool KDA, int D>
void launch(const PrefillParams& p, int B, hipStream_t stream) {
  constexpr int NT = D >= 32 ? 2 * D : 64;
  constexpr int CPT = D >= 32 ? 16 : 4;
  hipLaunchKernelGGL((prefill_kernel<KIND, KDA, D, NT, CPT>), dim3(p.HV, B), dim3(NT), 0, stream,
                     p);
}

template <int KIND, bool KDA>
void launch_d(int D, const PrefillParams& p, int B, hipStream_t stream) {
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
void launch_kind(const damp_pool* pool, int D, const PrefillParams& p, int B, hipStream_t s) {
  switch (layout_codec(&pool->layout)) {
    case kCodecFp32: launch_d<kFp32, KDA>(D, p, B, s); break;
    case kCodecPaper: launch_d<kPaper, KDA>(D, p, B, s); break;
    case kCodecInt4: launch_d<kInt4, KDA>(D, p, B, s); break;
    case kCodecFp8: launch_d<kFp8, KDA>(D, p, B, s); break;
    case kCodecNvfp4: launch_d<kNvfp4, KDA>(D, p, B, s); break;
    default: launch_d<kMixed, KDA>(D, p, B, s); break;
  }
}

}  // namespace

void prefill_window(bool kda, const damp_pool* pool, int32_t layer, const int32_t* slot_idx,
                    int32_t B, int32_t t0, int32_t T, int32_t t_pitch, int32_t num_k_heads,
                    const uint16_t* q, const uint16_t* k, const uint16_t* v, const uint16_t* g,
                    const uint16_t* beta, const uint8_t* perm, float scale, void* o,
                    bool o_bf16, hipStream_t stream) {
  PrefillParams p;
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
  p.T = T;
  p.t_pitch = t_pitch;
  p.t0 = t0;
  p.num_slots = pool->num_slots;
  p.HK = num_k_heads;
  p.HV = pool->num_v_heads;
  p.k_hi = pool->layout.kind == DAMP_STATE_FP32 ? 0 : pool->layout.k_hi;
  p.o_bf16 = o_bf16 ? 1 : 0;
  p.had = pool->layout.hadamard;
  if (kda) launch_kind<true>(pool, pool->layout.d_k, p, B, stream);
  else launch_kind<false>(pool, pool->layout.d_k, p, B, stream);
}

namespace {

damp_status prefill(bool kda, const damp_pool* pool, int32_t layer, const int32_t* slot_idx,
                    int32_t B, int32_t T, int32_t num_k_heads, const uint16_t* q,
                    const uint16_t* k, const uint16_t* v, const uint16_t* g, const uint16_t* beta,
                    const uint8_t* perm, float scale, void* o, int32_t o_dtype, void* stream) {
  clear_error();
  const char* name = kda ? "damp_state_prefill_kda" : "damp_state_prefill_gdn";
  damp_status st = check_pool(pool);
  if (st != DAMP_OK) return st;
  if (layer < 0 || layer >= pool->num_layers)
    return fail(DAMP_ERR_INVALID_ARG, "%s: layer %d outside [0, %d)", name, layer,
                pool->num_layers);
  if (B < 0 || B > 65535) return fail(DAMP_ERR_INVALID_ARG, "%s: B = %d outside [0, 65535]", name, B);
  if (T < 0) return fail(DAMP_ERR_INVALID_ARG, "%s: T = %d is negative", name, T);
  if (num_k_heads <= 0 || pool->num_v_heads % num_k_heads != 0)
    return fail(DAMP_ERR_INVALID_ARG, "%s: num_v_heads %d is not a multiple of num_k_heads %d",
                name, pool->num_v_heads, num_k_heads);
  if (o_dtype != DAMP_DT_FP32 && o_dtype != DAMP_DT_BF16)
    return fail(DAMP_ERR_INVALID_ARG, "%s: o_dtype must be FP32 or BF16", name);
  if (B == 0 || T == 0) return DAMP_OK;
  if (!slot_idx || !q || !k || !v || !g || !beta || !o)
    return fail(DAMP_ERR_INVALID_ARG, "%s: a required pointer is NULL", name);
  if (!layout_has_kernels(&pool->layout))
    return fail(DAMP_ERR_UNSUPPORTED, "%s: no kernel for this layout", name);

  prefill_window(kda, pool, layer, slot_idx, B, 0, T, T, num_k_heads, q, k, v, g, beta, perm,
                 scale, o, o_dtype == DAMP_DT_BF16, as_stream(stream));
  return check_launch(name);
}

}  // namespace
}  // namespace damp

extern "C" {

damp_status damp_state_prefill_gdn(const damp_pool* pool, int32_t layer,
                                   const int32_t* slot_idx, int32_t B, int32_t T,
                                   int32_t num_k_heads, const uint16_t* q, const uint16_t* k,
                                   const uint16_t* v, const uint16_t* g, const uint16_t* beta,
                                   const uint8_t* perm, float scale, void* o, int32_t o_dtype,
                                   void* stream) {
  return damp::prefill(false, pool, layer, slot_idx, B, T, num_k_heads, q, k, v, g, beta, perm,
                       scale, o, o_dtype, stream);
}

damp_status damp_state_prefill_kda(const damp_pool* pool, int32_t layer,
                                   const int32_t* slot_idx, int32_t B, int32_t T,
                                   int32_t num_k_heads, const uint16_t* q, const uint16_t* k,
                                   const uint16_t* v, const uint16_t* g, const uint16_t* beta,
                                   const uint8_t* perm, float scale, void* o, int32_t o_dtype,
                                   void* stream) {
  return damp::prefill(true, pool, layer, slot_idx, B, T, num_k_heads, q, k, v, g, beta, perm,
                       scale, o, o_dtype, stream);
}

}  // extern "C"
