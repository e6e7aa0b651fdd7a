// Prefill of one chunk of tokens per request into the packed pool (App. A.5,
// prefill path; section 3.1 Eq. (1)).
//
// One workgroup owns one (request, value head) tile: it decodes the stored
// state once into registers, runs the recurrence of Eq. (1) in fp32 for the
// chunk's T tokens (emitting o for every token), and re-encodes only the
// chunk-final state. At d = 128 the block kernel below does this; for the
// smaller head sizes (and inputs too long for its 32-bit offsets) the
// generic kernel keeps the mapping of the decode update: a row of the tile
// is split over TPR lanes, each holding CPT columns of RPT rows.
//
// In the generic kernel, per token, threads t < d_k stage the token's
// operands (k~, q~ gathered through the permutation, the row decay, v) in
// LDS, double-buffered: the next token's operands are loaded into registers
// while the current token computes. Both key-axis reductions share one LDS
// pass. In both kernels
//   o = scale (S_bar^T q~ + beta (q~ . k~) delta)
// equals scale * S^T q~ for the updated state S.
#include <climits>
#include <cstdint>

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
// d = 128 chunks in blocks of tokens. A workgroup of four waves owns one
// tile; thread (wave w, lane l = 8 cl + rb) keeps tile rows 16 rb .. 16 rb +
// 15 of columns 32 w + 4 cl .. + 3, 64 values. The operands of TB tokens
// (k~, q~ gathered through the permutation, KDA's a~ = exp(g~), v, beta, the
// scalar decay, q~ . k~) are converted to fp32 once per block by the whole
// workgroup into LDS, double-buffered: the next block's inputs are loaded
// into registers while the current block runs, and one barrier per block
// publishes them. Per token a lane reads its 16 rows' operands as LDS
// broadcasts (eight distinct addresses per wave), forms 8 partial read-outs
// (S_bar^T k~ and S_bar^T q~ over its rows, for its 4 columns) and sums them
// over the 8 row blocks with three DPP butterfly steps (lane bits 0..2), so
// every lane holds its columns' totals: the update needs no other exchange
// and the waves do not wait for each other within a block. GDN's scalar
// decay is deferred: the lane keeps P with S = gamma P, gamma the product of
// the decays since the last renormalization, so a token costs one FMA per
// state value for each read-out and one for the update:
//   w = gamma sum_u k_u P_u,  P_u += k_u (beta delta / gamma).
// A token whose decay would take gamma outside [2^-40, 2^40] (a zero decay
// included) scales P by gamma and its decay instead and resets gamma to 1.
struct BlkOps {
  uint32_t k[4], q[4], v[4], g[4];
  uint32_t beta[4];
};

template <int KIND, bool KDA>
__global__ __launch_bounds__(256) void prefill_blk128(const PrefillParams p) {
  constexpr int D = 128, TB = 8, CPT = 16, TPR = 8, NA = KDA ? TB : 1;
  // operand blocks by parity; the decode/encode transit buffer (32 rows)
  // aliases them outside the token loop
  struct OpBuf {
    float4 k[TB][D / 4];
    float4 q[TB][D / 4];
    float4 v[TB][D / 4];
    float4 a[NA][D / 4];
    float4 sc[TB];  // beta, alpha (GDN), q~ . k~ over rows 0..63 and 64..127
    float4 ge[KDA ? D / 4 : 1];  // KDA, deferred decay: each row's product over the block
    float4 os[TB][D / 4];        // o of the block's tokens, stored as whole rows at its end
  };
  constexpr int kTbufFloats = 32 * (D + 4);
  constexpr int kOpFloats = 2 * static_cast<int>(sizeof(OpBuf) / 4);
  __shared__ float4 lds4[(kOpFloats > kTbufFloats ? kOpFloats : kTbufFloats) / 4];
  OpBuf* ob = reinterpret_cast<OpBuf*>(lds4);
  float(*tbuf)[D + 4] = reinterpret_cast<float(*)[D + 4]>(lds4);

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int rb = lane & 7, cl = lane >> 3;
  const int c0 = 32 * wave + 4 * cl;  // this lane's first column
  const int rr = t >> 3, cg = t & 7, col0 = cg * CPT;  // row-slice role in transit
  const int h = blockIdx.x, b = blockIdx.y;
  const int T = p.T;
  const int hk = h / (p.HV / p.HK);

  // o of token tok at o_lane + tok * o_step (the token part is wave-uniform)
  const size_t o_esize = p.o_bf16 ? 2 : 4;
  uint8_t* const o_lane = static_cast<uint8_t*>(p.o) +
                          ((static_cast<size_t>(b) * T * p.HV + h) * D + c0) * o_esize;
  const size_t o_step = static_cast<size_t>(p.HV) * D * o_esize;
  auto o_ptr = [&](int tok) { return o_lane + static_cast<size_t>(tok) * o_step; };
  auto write_o = [&](int tok, const float (&ov)[4]) {
    if (!p.o || rb != 0) return;
    if (p.o_bf16) {
      *reinterpret_cast<uint2*>(o_ptr(tok)) =
          make_uint2(pack_bf16x2(ov[0], ov[1]), pack_bf16x2(ov[2], ov[3]));
    } else {
      *reinterpret_cast<float4*>(o_ptr(tok)) = make_float4(ov[0], ov[1], ov[2], ov[3]);
    }
  };

  const int slot = p.slot_idx[b];
  if (slot < 0 || slot >= p.num_slots) {  // padded request: o = 0, state untouched
    const float z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int tok = 0; tok < T; ++tok) write_o(tok, z);
    return;
  }
  uint8_t* tile = p.layer_base + static_cast<size_t>(slot) * p.slot_stride +
                  static_cast<size_t>(h) * p.tile_stride;
  const int k_hi = KIND == kFp32 ? D : p.k_hi;
  uint8_t* codes = tile + static_cast<size_t>(k_hi) * D * 2;
  uint8_t* meta_bytes = codes + static_cast<size_t>(D - k_hi) * code_row_bytes<KIND, D>();
  const bool had = p.had != 0;

  // ---- decode: pass c moves tile rows 16 j + 4 c + m (j < 8, m < 4), which
  // the row-slice threads decode and lane (rb, cl) reads as x[4 c + m]
  float x[16][4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    {
      float sl[CPT];
      decode_row<KIND, D, CPT>(tile, codes, meta_bytes, 16 * (rr >> 2) + 4 * c + (rr & 3), k_hi,
                               cg, col0, had, sl);
#pragma unroll
      for (int q4 = 0; q4 < CPT / 4; ++q4)
        *reinterpret_cast<float4*>(&tbuf[rr][col0 + 4 * q4]) =
            make_float4(sl[4 * q4], sl[4 * q4 + 1], sl[4 * q4 + 2], sl[4 * q4 + 3]);
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const float4 v4 = *reinterpret_cast<const float4*>(&tbuf[4 * rb + m][c0]);
      x[4 * c + m][0] = v4.x;
      x[4 * c + m][1] = v4.y;
      x[4 * c + m][2] = v4.z;
      x[4 * c + m][3] = v4.w;
    }
    __syncthreads();
  }

  // ---- operand staging: thread t handles tile row (and column) r of the
  // tokens 2 i + (wave >> 1) of a block, i < 4
  const int r = 64 * (wave & 1) + lane;
  // The per-row operands (k~, q~, a~ and KDA's block products) sit at
  // position ((r / 4) % 4) 32 + (r / 16) 4 + r % 4 of their 128 floats: a
  // lane of row block rb reads the float4 of rows 16 rb + 4 j .. + 3 at
  // index 8 j + rb, so for each j the eight row blocks of a wave read 128
  // consecutive bytes (one bank each) instead of eight float4 64 bytes apart.
  const int rsw = ((r >> 2) & 3) * 32 + (r >> 4) * 4 + (r & 3);
  const int u2 = 2 * (p.perm ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + r]) & (D - 1))
                             : r);
  const int half = wave >> 1;
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
  const __amdgpu_buffer_rsrc_t rbt = rsrc(p.beta, static_cast<size_t>(p.HV));
  auto load_blk = [&](BlkOps& o, int blk) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tok = TB * blk + 2 * i + half;
      if (tok < T) {
        const int tt = p.t0 + tok;
        const int kq = ((tt * p.HK + hk) * D) * 2;
        const int th = tt * p.HV + h;
        o.k[i] = __builtin_amdgcn_raw_buffer_load_b16(rk, u2, kq, 0);
        o.q[i] = __builtin_amdgcn_raw_buffer_load_b16(rq, u2, kq, 0);
        o.v[i] = __builtin_amdgcn_raw_buffer_load_b16(rv, 2 * r, th * D * 2, 0);
        o.g[i] = KDA ? __builtin_amdgcn_raw_buffer_load_b16(rg, u2, th * D * 2, 0)
                     : __builtin_amdgcn_raw_buffer_load_b16(rg, 0, th * 2, 0);
        o.beta[i] = __builtin_amdgcn_raw_buffer_load_b16(rbt, 0, th * 2, 0);
      }
    }
  };
  auto publish_blk = [&](const BlkOps& o, int blk, int par) {
    OpBuf& B_ = ob[par];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int tb = 2 * i + half;
      if (TB * blk + tb < T) {
        const float kf = bf16_to_f32(static_cast<uint16_t>(o.k[i]));
        const float qf = bf16_to_f32(static_cast<uint16_t>(o.q[i]));
        reinterpret_cast<float*>(B_.k[tb])[rsw] = kf;
        reinterpret_cast<float*>(B_.q[tb])[rsw] = qf;
        reinterpret_cast<float*>(B_.v[tb])[r] = bf16_to_f32(static_cast<uint16_t>(o.v[i]));
        if (KDA)
          reinterpret_cast<float*>(B_.a[KDA ? tb : 0])[rsw] =
              __expf(bf16_to_f32(static_cast<uint16_t>(o.g[i])));
        const float kq = wave_sum_dpp(kf * qf);
        float* sc = reinterpret_cast<float*>(&B_.sc[tb]);
        if (lane == 0) {
          sc[2 + (wave & 1)] = kq;
          if ((wave & 1) == 0) {
            sc[0] = bf16_to_f32(static_cast<uint16_t>(o.beta[i]));
            sc[1] = KDA ? 1.0f : __expf(bf16_to_f32(static_cast<uint16_t>(o.g[i])));
          }
        }
      }
    }
  };

  // KDA: the decays of a block are deferred per row. The lanes keep P with
  // S = G P, G_r(t) the product of row r's decays over the block's tokens up
  // to t; the staged operands become k~ G, q~ G (read-outs) and k~ / G (the
  // update), and the block ends with x *= G_r(end). A block in which some
  // G leaves [2^-60, 2^60] keeps the per-token decay (returns 1).
  auto cumulate = [&](int par, int ntok_) -> int {
    OpBuf& B_ = ob[par];
    bool ok = true;
    if (t < D) {
      float G = 1.0f;
      for (int tb = 0; tb < ntok_; ++tb) {
        G *= reinterpret_cast<const float*>(B_.a[tb])[t];
        ok = ok && G >= 8.6736174e-19f && G <= 1.1529215e18f;
      }
    }
    const int slow = __syncthreads_or(ok ? 0 : 1);
    if (!slow && t < D) {
      float G = 1.0f;
      for (int tb = 0; tb < ntok_; ++tb) {
        float* kk_ = reinterpret_cast<float*>(B_.k[tb]);
        float* qq_ = reinterpret_cast<float*>(B_.q[tb]);
        float* aa_ = reinterpret_cast<float*>(B_.a[tb]);
        G *= aa_[t];
        const float kf = kk_[t];
        kk_[t] = kf * G;
        qq_[t] = qq_[t] * G;
        aa_[t] = kf * refined_rcp(G);
      }
      reinterpret_cast<float*>(B_.ge)[t] = G;
    }
    return slow;
  };
  const int nblk = (T + TB - 1) / TB;
  BlkOps cur;
  int slow_cur = 1;
  if (nblk > 0) {
    load_blk(cur, 0);
    publish_blk(cur, 0, 0);
    if constexpr (KDA) {
      __syncthreads();
      slow_cur = cumulate(0, T < TB ? T : TB);
    }
  }
  __syncthreads();
  float gamma = 1.0f;
#pragma unroll 1
  for (int blk = 0; blk < nblk; ++blk) {
    const int par = blk & 1;
    if (blk + 1 < nblk) load_blk(cur, blk + 1);
    const OpBuf& B_ = ob[par];
    const int ntok = T - TB * blk < TB ? T - TB * blk : TB;
#pragma unroll 1
    for (int tb = 0; tb < ntok; ++tb) {
      const int tok = TB * blk + tb;
      float kr[16];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 k4 = B_.k[tb][8 * j + rb];
        kr[4 * j] = k4.x;
        kr[4 * j + 1] = k4.y;
        kr[4 * j + 2] = k4.z;
        kr[4 * j + 3] = k4.w;
      }
      if (KDA && slow_cur) {  // the decay of each row, per token
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float4 a4 = B_.a[KDA ? tb : 0][8 * j + rb];
          const float aj[4] = {a4.x, a4.y, a4.z, a4.w};
#pragma unroll
          for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int c = 0; c < 4; ++c) x[4 * j + m][c] *= aj[m];
        }
      }
      // partial read-outs over this lane's 16 rows
      float w[4], pq[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) w[c] = kr[0] * x[0][c];
#pragma unroll
      for (int i = 1; i < 16; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) w[c] = fmaf(kr[i], x[i][c], w[c]);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 q4 = B_.q[tb][8 * j + rb];
        const float qj[4] = {q4.x, q4.y, q4.z, q4.w};
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
          for (int c = 0; c < 4; ++c)
            pq[c] = (j == 0 && m == 0) ? qj[0] * x[0][c] : fmaf(qj[m], x[4 * j + m][c], pq[c]);
      }
      // sums over the 8 row blocks: lane bits 0, 1 (quad_perm) and 2
      // (row_half_mirror pairs each lane with one of the other quad)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        w[c] += dpp_mov<0xb1>(w[c]);
        pq[c] += dpp_mov<0xb1>(pq[c]);
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        w[c] += dpp_mov<0x4e>(w[c]);
        pq[c] += dpp_mov<0x4e>(pq[c]);
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        w[c] += dpp_mov<0x141>(w[c]);
        pq[c] += dpp_mov<0x141>(pq[c]);
      }
      // per token: g = gamma (1 for KDA), o = scale (g p + beta (q~.k~) delta),
      // delta = v - g w, and the update's factor (beta / g) delta. GDN keeps
      // gamma within [2^-40, 2^40]: when this token's decay would take it out
      // (a vanishing or zero alpha included), the read-outs still take the
      // exact factor, but the update runs on S_bar itself (P scaled by the old
      // gamma and this alpha, gamma reset to 1), so 1 / gamma stays finite
      const float4 sc = B_.sc[tb];
      float gw = 1.0f, bg = sc.x;
      bool fold = false;
      if (!KDA) {
        gw = gamma * sc.y;
        fold = !(gw >= 9.094947e-13f && gw <= 1.0995116e12f);
        if (!fold) bg = sc.x * refined_rcp(gw);
      }
      const float sg = p.scale * gw, sbq = p.scale * sc.x * (sc.z + sc.w);
      const float4 v4 = B_.v[tb][c0 / 4];
      const float vv[4] = {v4.x, v4.y, v4.z, v4.w};
      float ov[4], cf[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float delta = fmaf(-gw, w[c], vv[c]);  // delta = v - S_bar^T k~
        ov[c] = fmaf(sbq, delta, sg * pq[c]);
        cf[c] = bg * delta;
      }
      if (rb == 0) ob[par].os[tb][c0 / 4] = make_float4(ov[0], ov[1], ov[2], ov[3]);
      // rank-1 update S = S_bar + beta k~ delta^T (GDN: on P = S / gamma;
      // KDA with deferred decay: on P = S / G with k~ / G)
      if (KDA && !slow_cur) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float4 b4 = B_.a[KDA ? tb : 0][8 * j + rb];
          kr[4 * j] = b4.x;
          kr[4 * j + 1] = b4.y;
          kr[4 * j + 2] = b4.z;
          kr[4 * j + 3] = b4.w;
        }
      }
      if (!KDA) {
        if (fold) {
#pragma unroll
          for (int i = 0; i < 16; ++i)
#pragma unroll
            for (int c = 0; c < 4; ++c) x[i][c] = (x[i][c] * gamma) * sc.y;
          gamma = 1.0f;
        } else {
          gamma = gw;
        }
      }
#pragma unroll
      for (int i = 0; i < 16; ++i)
#pragma unroll
        for (int c = 0; c < 4; ++c) x[i][c] = fmaf(kr[i], cf[c], x[i][c]);
    }
    if (KDA && !slow_cur) {  // S = G P at the end of the block
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float4 g4 = B_.ge[KDA ? 8 * j + rb : 0];
        const float gj[4] = {g4.x, g4.y, g4.z, g4.w};
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
          for (int c = 0; c < 4; ++c) x[4 * j + m][c] *= gj[m];
      }
    }
    int slow_next = 1;
    if (blk + 1 < nblk) {
      publish_blk(cur, blk + 1, par ^ 1);
      if constexpr (KDA) {
        __syncthreads();
        const int left = T - TB * (blk + 1);
        slow_next = cumulate(par ^ 1, left < TB ? left : TB);
      }
    }
    __syncthreads();
    slow_cur = slow_next;
    // the block's o, a 16-byte piece per thread: 128 threads for bf16 rows
    // (8 columns each), all 256 for fp32 rows (4 columns each)
    if (p.o) {
      const OpBuf& O_ = ob[par];
      uint8_t* const o_row = static_cast<uint8_t*>(p.o) +
                             ((static_cast<size_t>(b) * T * p.HV + h) * D) * o_esize;
      if (p.o_bf16) {
        const int tb = t >> 4, q8 = t & 15;
        if (tb < ntok) {
          const float4 lo = O_.os[tb][2 * q8], hi = O_.os[tb][2 * q8 + 1];
          *reinterpret_cast<uint4*>(o_row + static_cast<size_t>(TB * blk + tb) * o_step +
                                    16 * q8) =
              make_uint4(pack_bf16x2(lo.x, lo.y), pack_bf16x2(lo.z, lo.w),
                         pack_bf16x2(hi.x, hi.y), pack_bf16x2(hi.z, hi.w));
        }
      } else {
        const int tb = t >> 5, q4 = t & 31;
        if (tb < ntok)
          *reinterpret_cast<float4*>(o_row + static_cast<size_t>(TB * blk + tb) * o_step +
                                     16 * q4) = O_.os[tb][q4];
      }
    }
  }
  __syncthreads();  // the last block's o is read before the transit buffer reuses it
  if (!KDA) {
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int c = 0; c < 4; ++c) x[i][c] *= gamma;
  }

  // ---- store the chunk-final state per its tier, in the decode's passes
  float s_g = 1.0f;
  if constexpr (KIND == kNvfp4) {  // the global scale of the final low tier
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (16 * rb + i >= k_hi)
#pragma unroll
        for (int c = 0; c < 4; ++c) amax = fmaxf(amax, fabsf(x[i][c]));
    s_g = nvfp4_global(block_max<256>(amax));
    if (t == 0) store_global_scale<D>(meta_bytes, k_hi, s_g);
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) {
#pragma unroll
    for (int m = 0; m < 4; ++m)
      *reinterpret_cast<float4*>(&tbuf[4 * rb + m][c0]) =
          make_float4(x[4 * c + m][0], x[4 * c + m][1], x[4 * c + m][2], x[4 * c + m][3]);
    __syncthreads();
    {
      float sl[CPT];
#pragma unroll
      for (int q4 = 0; q4 < CPT / 4; ++q4) {
        const float4 v4 = *reinterpret_cast<const float4*>(&tbuf[rr][col0 + 4 * q4]);
        sl[4 * q4] = v4.x;
        sl[4 * q4 + 1] = v4.y;
        sl[4 * q4 + 2] = v4.z;
        sl[4 * q4 + 3] = v4.w;
      }
      encode_row<KIND, D, CPT, TPR>(sl, 16 * (rr >> 2) + 4 * c + (rr & 3), k_hi, cg, col0, tile,
                                    codes, meta_bytes, had, s_g);
    }
    __syncthreads();
  }
}

template <int KIND, bool KDA, int D>
void launch(const PrefillParams& p, int B, hipStream_t stream) {
  // the block kernel addresses one request's inputs with 32-bit offsets
  const int64_t span = static_cast<int64_t>(p.t_pitch) * (p.HK > p.HV ? p.HK : p.HV) * D * 2;
  if constexpr (D == 128) {
    if (span <= INT32_MAX) {
      hipLaunchKernelGGL((prefill_blk128<KIND, KDA>), dim3(p.HV, B), dim3(256), 0, stream, p);
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
  if (reinterpret_cast<uintptr_t>(o) % 16 != 0)
    return fail(DAMP_ERR_INVALID_ARG, "%s: o is not 16-byte aligned", name);
  if (!layout_has_kernels(&pool->layout))
    return fail(DAMP_ERR_UNSUPPORTED, "%s: no kernel for this layout", name);
  st = debug_check_slots(pool, slot_idx, B, as_stream(stream), name);
  if (st != DAMP_OK) return st;

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
