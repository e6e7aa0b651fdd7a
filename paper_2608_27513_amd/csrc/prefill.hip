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

// d = 128 chunks run one lane pair per state column: a workgroup of four
// waves holds the tile transposed, lane l of wave w keeping rows
// 64 (l >> 5) .. 64 (l >> 5) + 63 of column 32 w + (l & 31) in registers, the
// other half of the column in lane l ^ 32. Both key-axis read-outs,
// sum_u k~_u S_bar_uj and sum_u q~_u S_bar_uj, are then sums within the
// lane plus one exchange with the partner lane, so a token needs no LDS
// reduction and no workgroup barrier. The token's per-row operands (k~, q~,
// the decay a~, gathered through the permutation) are staged by each wave in
// its own LDS slice, double-buffered across tokens, and read as broadcasts
// (the upper half's rows padded onto other banks). The stored tile is
// decoded and encoded once per chunk with the row-slice codecs, 16 rows at a
// time through an LDS transpose buffer, so every storage format is handled.
struct ColOps {
  uint32_t k[2] = {0u, 0u}, q[2] = {0u, 0u}, g[2] = {0u, 0u};
  uint32_t gs = 0u, beta = 0u, v = 0u;
};

template <int KIND, bool KDA>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3))) void prefill_col128(const PrefillParams p) {
  constexpr int D = 128, CPT = 16, TPR = 8, RH = 64;  // rows per lane
  constexpr int OPN = D + 4;                           // padded operand rows
  __shared__ float tbuf[16][D + 4];        // 16 tile rows (padded against bank conflicts)
  __shared__ float4 opk[4][2][OPN / 4];    // [wave][parity] k~ (row u at u + 4 (u >= 64))
  __shared__ float4 opq[4][2][OPN / 4];    // q~
  __shared__ float4 opa[4][2][KDA ? OPN / 4 : 1];  // a~ = exp(g~) per row (KDA)

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int hh = lane >> 5;                 // which half of the column
  const int col = 32 * wave + (lane & 31);  // this lane's column
  const int h = blockIdx.x, b = blockIdx.y;
  const int rr = (t >> 3) & 15, cg = t & 7, col0 = cg * CPT;  // row-slice role (t < 128)
  const int T = p.T;
  const int hk = h / (p.HV / p.HK);
  const int o_esize = p.o_bf16 ? 2 : 4;
  auto write_o = [&](int tok, float val) {
    if (!p.o || hh) return;
    uint8_t* at = static_cast<uint8_t*>(p.o) +
                  (((static_cast<size_t>(b) * T + tok) * p.HV + h) * D + col) * o_esize;
    if (p.o_bf16) *reinterpret_cast<uint16_t*>(at) = f32_to_bf16(val);
    else *reinterpret_cast<float*>(at) = val;
  };

  const int slot = p.slot_idx[b];
  if (slot < 0 || slot >= p.num_slots) {  // padded request: o = 0, state untouched
    for (int tok = 0; tok < T; ++tok) write_o(tok, 0.0f);
    return;
  }
  uint8_t* tile = p.layer_base + static_cast<size_t>(slot) * p.slot_stride +
                  static_cast<size_t>(h) * p.tile_stride;
  const int k_hi = KIND == kFp32 ? D : p.k_hi;
  uint8_t* codes = tile + static_cast<size_t>(k_hi) * D * 2;
  uint8_t* meta_bytes = codes + static_cast<size_t>(D - k_hi) * code_row_bytes<KIND, D>();
  const bool had = p.had != 0;

  // ---- decode the stored state once, transposing 16 rows at a time
  float x[RH];
#pragma unroll
  for (int c = 0; c < D / 16; ++c) {
    if (t < 128) {  // waves 0 and 1 decode the 16 rows as row slices
      float sl[CPT];
      decode_row<KIND, D, CPT>(tile, codes, meta_bytes, 16 * c + rr, k_hi, cg, col0, had, sl);
#pragma unroll
      for (int q4 = 0; q4 < CPT / 4; ++q4)
        *reinterpret_cast<float4*>(&tbuf[rr][col0 + 4 * q4]) =
            make_float4(sl[4 * q4], sl[4 * q4 + 1], sl[4 * q4 + 2], sl[4 * q4 + 3]);
    }
    __syncthreads();
    if (hh == c / 4) {
#pragma unroll
      for (int r = 0; r < 16; ++r) x[16 * (c % 4) + r] = tbuf[r][col];
    }
    __syncthreads();
  }

  // ---- per-token operands: lane stages rows lane and lane + 64. Inputs are
  // read through buffer resources based at this request, with the token's
  // offset wave-uniform and the row's per lane.
  int urow2[2];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int r = lane + 64 * e;
    urow2[e] = 2 * (p.perm ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + r]) & (D - 1)) : r);
  }
  const size_t tp = static_cast<size_t>(p.t_pitch);
  constexpr int kCfg = 0x00020000;  // raw 32-bit buffer
  auto rsrc = [&](const uint16_t* base, size_t per_token) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base) + b * tp * per_token, 0,
                                             static_cast<int>(tp * per_token * 2), kCfg);
  };
  const __amdgpu_buffer_rsrc_t rk = rsrc(p.k, static_cast<size_t>(p.HK) * D);
  const __amdgpu_buffer_rsrc_t rq = rsrc(p.q, static_cast<size_t>(p.HK) * D);
  const __amdgpu_buffer_rsrc_t rv = rsrc(p.v, static_cast<size_t>(p.HV) * D);
  const __amdgpu_buffer_rsrc_t rg = rsrc(p.g, static_cast<size_t>(p.HV) * (KDA ? D : 1));
  const __amdgpu_buffer_rsrc_t rb = rsrc(p.beta, static_cast<size_t>(p.HV));
  auto load_ops = [&](ColOps& o, int tok) {
    const int tt = p.t0 + tok;
    const int kq = ((tt * p.HK + hk) * D) * 2;
    const int th = tt * p.HV + h;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      o.k[e] = __builtin_amdgcn_raw_buffer_load_b16(rk, urow2[e], kq, 0);
      o.q[e] = __builtin_amdgcn_raw_buffer_load_b16(rq, urow2[e], kq, 0);
      if (KDA) o.g[e] = __builtin_amdgcn_raw_buffer_load_b16(rg, urow2[e], th * D * 2, 0);
    }
    if (!KDA) o.gs = __builtin_amdgcn_raw_buffer_load_b16(rg, 0, th * 2, 0);
    o.beta = __builtin_amdgcn_raw_buffer_load_b16(rb, 0, th * 2, 0);
    o.v = __builtin_amdgcn_raw_buffer_load_b16(rv, 2 * col, th * D * 2, 0);
  };
  // converts the staged words and writes this wave's operand slice; returns
  // q~ . k~ over all rows (every lane)
  auto publish = [&](const ColOps& o, int par) {
    float kq = 0.0f;
    float* fk = reinterpret_cast<float*>(opk[wave][par]);
    float* fq = reinterpret_cast<float*>(opq[wave][par]);
    float* fa = reinterpret_cast<float*>(opa[wave][KDA ? par : 0]);
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int at = lane + 68 * e;  // row lane + 64 e, the upper half shifted by 4
      const float kf = bf16_to_f32(static_cast<uint16_t>(o.k[e]));
      const float qf = bf16_to_f32(static_cast<uint16_t>(o.q[e]));
      fk[at] = kf;
      fq[at] = qf;
      if (KDA) fa[at] = __expf(bf16_to_f32(static_cast<uint16_t>(o.g[e])));
      kq = fmaf(kf, qf, kq);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
    return wave_sum_dpp(kq);
  };
  // the partner lane's copy of v (the other half of the column)
  auto partner = [&](float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false,
                                                    false);
    return __uint_as_float(hh ? r[0] : r[1]);
  };

  __builtin_amdgcn_sched_barrier(0);
  ColOps cur, nxt;
  float qk = 0.0f, beta = 0.0f, vj = 0.0f, alpha = 1.0f;
  if (T > 0) {
    load_ops(cur, 0);
    qk = publish(cur, 0);
    beta = bf16_to_f32(static_cast<uint16_t>(cur.beta));
    vj = bf16_to_f32(static_cast<uint16_t>(cur.v));
    if (!KDA) alpha = __expf(bf16_to_f32(static_cast<uint16_t>(cur.gs)));
  }
  const int ob = 17 * hh;  // this half's first float4 of the operand rows
#pragma unroll 1
  for (int tok = 0; tok < T; ++tok) {
    const int par = tok & 1;
    if (tok + 1 < T) load_ops(nxt, tok + 1);
    // decay and both read-outs over this lane's 64 rows
    float w[4] = {0.0f, 0.0f, 0.0f, 0.0f}, pq[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int i = 0; i < RH / 4; ++i) {
      const float4 k4 = opk[wave][par][ob + i], q4 = opq[wave][par][ob + i];
      float4 a4 = make_float4(alpha, alpha, alpha, alpha);
      if (KDA) a4 = opa[wave][KDA ? par : 0][ob + i];
      const float kk[4] = {k4.x, k4.y, k4.z, k4.w}, qq[4] = {q4.x, q4.y, q4.z, q4.w};
      const float aa[4] = {a4.x, a4.y, a4.z, a4.w};
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        float& xv = x[4 * i + m];
        xv *= aa[m];
        w[m] = fmaf(kk[m], xv, w[m]);
        pq[m] = fmaf(qq[m], xv, pq[m]);
      }
    }
    float wt = (w[0] + w[1]) + (w[2] + w[3]);
    float pt = (pq[0] + pq[1]) + (pq[2] + pq[3]);
    wt += partner(wt);  // the column's other 64 rows
    pt += partner(pt);
    const float delta = vj - wt;  // delta = v - S_bar^T k~
    write_o(tok, p.scale * fmaf(beta * qk, delta, pt));
    // rank-1 update S = S_bar + beta k~ delta^T
    const float bd = beta * delta;
#pragma unroll
    for (int i = 0; i < RH / 4; ++i) {
      const float4 k4 = opk[wave][par][ob + i];
      x[4 * i + 0] = fmaf(k4.x, bd, x[4 * i + 0]);
      x[4 * i + 1] = fmaf(k4.y, bd, x[4 * i + 1]);
      x[4 * i + 2] = fmaf(k4.z, bd, x[4 * i + 2]);
      x[4 * i + 3] = fmaf(k4.w, bd, x[4 * i + 3]);
    }
    if (tok + 1 < T) {
      qk = publish(nxt, par ^ 1);
      beta = bf16_to_f32(static_cast<uint16_t>(nxt.beta));
      vj = bf16_to_f32(static_cast<uint16_t>(nxt.v));
      if (!KDA) alpha = __expf(bf16_to_f32(static_cast<uint16_t>(nxt.gs)));
    }
  }

  // ---- store the chunk-final state per its tier, 16 rows at a time
  float s_g = 1.0f;
  if constexpr (KIND == kNvfp4) {  // the global scale of the final low tier
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < RH; ++i)
      if (RH * hh + i >= k_hi) amax = fmaxf(amax, fabsf(x[i]));
    s_g = nvfp4_global(block_max<256>(amax));
    if (t == 0) store_global_scale<D>(meta_bytes, k_hi, s_g);
  }
#pragma unroll
  for (int c = 0; c < D / 16; ++c) {
    if (hh == c / 4) {
#pragma unroll
      for (int r = 0; r < 16; ++r) tbuf[r][col] = x[16 * (c % 4) + r];
    }
    __syncthreads();
    if (t < 128) {
      float sl[CPT];
#pragma unroll
      for (int q4 = 0; q4 < CPT / 4; ++q4) {
        const float4 v4 = *reinterpret_cast<const float4*>(&tbuf[rr][col0 + 4 * q4]);
        sl[4 * q4] = v4.x;
        sl[4 * q4 + 1] = v4.y;
        sl[4 * q4 + 2] = v4.z;
        sl[4 * q4 + 3] = v4.w;
      }
      encode_row<KIND, D, CPT, TPR>(sl, 16 * c + rr, k_hi, cg, col0, tile, codes, meta_bytes,
                                    had, s_g);
    }
    __syncthreads();
  }
}

// GDN chunks at d = 128 take their per-row operands from scalar registers:
// a workgroup of two waves holds the tile transposed with rows in natural
// key-channel order (the permutation is applied when the tile is decoded and
// encoded), lane l of wave w keeping column 64 w + l of all 128 rows. The
// token's k~ and q~ rows then come straight from the inputs by scalar loads,
// shared by every lane at no LDS cost. The head's scalar decay is deferred:
// the lane keeps P with S = gamma P, gamma the product of the decays since the
// last renormalization, so a token costs one FMA per state value for each
// read-out and one for the update:
//   w = gamma sum_u k_u P_u,  P_u += k_u (beta delta / gamma).
template <int KIND>
__global__ __launch_bounds__(128) void prefill_gdn_sgpr128(const PrefillParams p) {
  constexpr int D = 128, CPT = 16, TPR = 8;
  __shared__ float tbuf[16][D + 4];  // 16 rows in transit (padded against bank conflicts)
  __shared__ int inv[D];             // tile row of each natural key channel

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int col = 64 * wave + lane;
  const int h = blockIdx.x, b = blockIdx.y;
  const int rr = t >> 3, cg = t & 7, col0 = cg * CPT;  // row-slice role of the codecs
  const int T = p.T;
  const int hk = h / (p.HV / p.HK);
  const int o_esize = p.o_bf16 ? 2 : 4;
  auto write_o = [&](int tok, float val) {
    if (!p.o) return;
    uint8_t* at = static_cast<uint8_t*>(p.o) +
                  (((static_cast<size_t>(b) * T + tok) * p.HV + h) * D + col) * o_esize;
    if (p.o_bf16) *reinterpret_cast<uint16_t*>(at) = f32_to_bf16(val);
    else *reinterpret_cast<float*>(at) = val;
  };

  const int slot = p.slot_idx[b];
  if (slot < 0 || slot >= p.num_slots) {  // padded request: o = 0, state untouched
    for (int tok = 0; tok < T; ++tok) write_o(tok, 0.0f);
    return;
  }
  uint8_t* tile = p.layer_base + static_cast<size_t>(slot) * p.slot_stride +
                  static_cast<size_t>(h) * p.tile_stride;
  const int k_hi = KIND == kFp32 ? D : p.k_hi;
  uint8_t* codes = tile + static_cast<size_t>(k_hi) * D * 2;
  uint8_t* meta_bytes = codes + static_cast<size_t>(D - k_hi) * code_row_bytes<KIND, D>();
  const bool had = p.had != 0;

  inv[p.perm ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + t]) & (D - 1)) : t] = t;
  __syncthreads();

  // ---- decode: natural rows 16 c .. 16 c + 15 at a time
  float x[D];
#pragma unroll
  for (int c = 0; c < D / 16; ++c) {
    __builtin_amdgcn_sched_barrier(0);
    float sl[CPT];
    decode_row<KIND, D, CPT>(tile, codes, meta_bytes, inv[16 * c + rr], k_hi, cg, col0, had, sl);
#pragma unroll
    for (int q4 = 0; q4 < CPT / 4; ++q4)
      *reinterpret_cast<float4*>(&tbuf[rr][col0 + 4 * q4]) =
          make_float4(sl[4 * q4], sl[4 * q4 + 1], sl[4 * q4 + 2], sl[4 * q4 + 3]);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r) x[16 * c + r] = tbuf[r][col];
    __syncthreads();
  }

  const size_t req = static_cast<size_t>(b) * p.t_pitch + p.t0;
  const uint16_t* __restrict__ vb = p.v;
  float gamma = 1.0f;
#pragma unroll 1
  for (int tok = 0; tok < T; ++tok) {
    const size_t bt = req + tok;
    const size_t bth = bt * p.HV + h;
    const uint32_t* __restrict__ kr =
        reinterpret_cast<const uint32_t*>(p.k + (bt * p.HK + hk) * D);
    const uint32_t* __restrict__ qr =
        reinterpret_cast<const uint32_t*>(p.q + (bt * p.HK + hk) * D);
    const float alpha = __expf(bf16_to_f32(p.g[bth]));
    const float beta = bf16_to_f32(p.beta[bth]);
    const float vj = bf16_to_f32(vb[bth * D + col]);
    // q~ . k~ over the channels (permutation invariant), two per lane
    float kq = 0.0f;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const uint16_t* kk = p.k + (bt * p.HK + hk) * D;
      const uint16_t* qq = p.q + (bt * p.HK + hk) * D;
      kq = fmaf(bf16_to_f32(kk[lane + 64 * e]), bf16_to_f32(qq[lane + 64 * e]), kq);
    }
    const float qk = wave_sum_dpp(kq);
    gamma *= alpha;
    // both read-outs: one FMA per state value each, k and q from SGPRs
    float w0 = 0.0f, w1 = 0.0f, p0 = 0.0f, p1 = 0.0f;
#pragma unroll
    for (int d = 0; d < D / 2; ++d) {
      const uint32_t pk = kr[d], pq = qr[d];
      w0 = fmaf(__uint_as_float(pk << 16), x[2 * d], w0);
      w1 = fmaf(__uint_as_float(pk & 0xffff0000u), x[2 * d + 1], w1);
      p0 = fmaf(__uint_as_float(pq << 16), x[2 * d], p0);
      p1 = fmaf(__uint_as_float(pq & 0xffff0000u), x[2 * d + 1], p1);
    }
    const float wt = gamma * (w0 + w1);
    const float pt = gamma * (p0 + p1);
    const float delta = vj - wt;  // delta = v - S_bar^T k~
    write_o(tok, p.scale * fmaf(beta * qk, delta, pt));
    // S = S_bar + beta k~ delta^T, i.e. P += k~ (beta delta / gamma)
    const float cf = beta * delta / gamma;
#pragma unroll
    for (int d = 0; d < D / 2; ++d) {
      const uint32_t pk = kr[d];
      x[2 * d] = fmaf(__uint_as_float(pk << 16), cf, x[2 * d]);
      x[2 * d + 1] = fmaf(__uint_as_float(pk & 0xffff0000u), cf, x[2 * d + 1]);
    }
    if (!(gamma >= 9.094947e-13f && gamma <= 1.0995116e12f)) {  // outside [2^-40, 2^40]
#pragma unroll
      for (int u = 0; u < D; ++u) x[u] *= gamma;
      gamma = 1.0f;
    }
  }
#pragma unroll
  for (int u = 0; u < D; ++u) x[u] *= gamma;

  // ---- store the chunk-final state per its tier, natural rows 16 at a time
  float s_g = 1.0f;
  if constexpr (KIND == kNvfp4) {  // the global scale of the final low tier
    float amax = 0.0f;
#pragma unroll
    for (int u = 0; u < D; ++u)
      if (inv[u] >= k_hi) amax = fmaxf(amax, fabsf(x[u]));
    s_g = nvfp4_global(block_max<128>(amax));
    if (t == 0) store_global_scale<D>(meta_bytes, k_hi, s_g);
  }
#pragma unroll
  for (int c = 0; c < D / 16; ++c) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int r = 0; r < 16; ++r) tbuf[r][col] = x[16 * c + r];
    __syncthreads();
    float sl[CPT];
#pragma unroll
    for (int q4 = 0; q4 < CPT / 4; ++q4) {
      const float4 v4 = *reinterpret_cast<const float4*>(&tbuf[rr][col0 + 4 * q4]);
      sl[4 * q4] = v4.x;
      sl[4 * q4 + 1] = v4.y;
      sl[4 * q4 + 2] = v4.z;
      sl[4 * q4 + 3] = v4.w;
    }
    encode_row<KIND, D, CPT, TPR>(sl, inv[16 * c + rr], k_hi, cg, col0, tile, codes, meta_bytes,
                                  had, s_g);
    __syncthreads();
  }
}

template <int KIND, bool KDA, int D>
void launch(const PrefillParams& p, int B, hipStream_t stream) {
  // the column kernel addresses one request's inputs with 32-bit offsets
  const int64_t span = static_cast<int64_t>(p.t_pitch) * (p.HK > p.HV ? p.HK : p.HV) * D * 2;
  if constexpr (D == 128 && !KDA) {
    (void)span;
    hipLaunchKernelGGL((prefill_gdn_sgpr128<KIND>), dim3(p.HV, B), dim3(128), 0, stream, p);
    return;
  } else if constexpr (D == 128) {
    if (span <= INT32_MAX) {
      hipLaunchKernelGGL((prefill_col128<KIND, KDA>), dim3(p.HV, B), dim3(256), 0, stream, p);
      return;
    }
  }
  {
    constexpr int NT = D >= 32 ? 2 * D : 64;
    constexpr int CPT = D >= 32 ? 16 : 4;
    hipLaunchKernelGGL((prefill_kernel<KIND, KDA, D, NT, CPT>), dim3(p.HV, B), dim3(NT), 0,
                       stream, p);
  }
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
