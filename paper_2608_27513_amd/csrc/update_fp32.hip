// Decode-step update of an FP32 state at d_k = d_v = 128 (the deployment
// baseline the paper compares DAMP against: section 6, one FP32 state per
// request), for GDN and KDA heads (section 3.1 Eq. (1)-(2)).
//
// The tile is 64 KB of fp32 and the arithmetic is four FMAs per value, so the
// kernel is an HBM stream: what matters is that every load and store moves
// whole 128-byte lines and that enough of them are in flight. One workgroup
// (4 wave64) owns one tile; thread t (row group rg = t / 8, column group
// cg = t % 8) holds rows rg + 32 i (i = 0..3) and, in each quarter jj of the
// row, columns 32 jj + 4 cg .. 32 jj + 4 cg + 3. So for a fixed (i, jj) the 8
// lanes of a row group read one whole 128-byte line of their row, and a wave
// instruction moves 8 whole lines. The tile's 16 loads per thread are issued
// before anything waits on them; loads and stores are non-temporal, stores at
// device (sc1) scope.
//
// The two key-axis read-outs share one LDS pass (per-thread partial column
// sums, then one thread per (column, kind) adds the 32 row groups), and
//   o = scale (S_bar^T q~ + beta (q~ . k~) delta)
// equals scale * S'^T q~ for the updated S' = S_bar + beta k~ delta^T.
#include "device.hpp"
#include "internal.hpp"
#include "update.hpp"

namespace damp {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCachePolicyNT = 2;  // loads
constexpr int kStorePolicy = 2 | 16;  // stores: non-temporal, device (sc1) scope (190.0 against 193.3 us)
constexpr int kBufferConfig = 0x00020000;  // raw 32-bit buffer (gfx9 family)

template <bool KDA>
__global__ __launch_bounds__(256) void update_fp32_128(const UpdateParams p) {
  constexpr int D = 128, RG = 32, RPT = 4, CPT = 16;
  __shared__ float red[RG][2 * D];
  __shared__ float dsh[D];

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int h = blockIdx.x;
  const int b = blockIdx.y;
  const int cg = t % 8, rg = t / 8;
  const size_t bh = static_cast<size_t>(b) * p.HV + h;
  auto write_o = [&](int j, float val) {
    if (p.o_bf16)
      static_cast<uint16_t*>(p.o)[bh * D + j] = f32_to_bf16(val);
    else
      static_cast<float*>(p.o)[bh * D + j] = val;
  };

  const int slot = p.slot_idx[b];
  if (slot < 0 || slot >= p.num_slots) {  // padded request: o = 0, state untouched
    if (t < D) write_o(t, 0.0f);
    return;
  }
  uint8_t* tile = p.layer_base + static_cast<size_t>(slot) * p.slot_stride +
                  static_cast<size_t>(h) * p.tile_stride;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(tile, 0, D * D * 4,
                                                                      kBufferConfig);
  // byte offset of (row rg + 32 i, columns 32 jj + 4 cg ..)
  auto off = [&](int i, int jj) { return ((rg + RG * i) * D + 32 * jj + 4 * cg) * 4; };

  // ---- the whole tile in flight ------------------------------------------
  u32x4 raw[RPT][4];
#pragma unroll
  for (int i = 0; i < RPT; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      raw[i][jj] = __builtin_amdgcn_raw_buffer_load_b128(rs, off(i, jj), 0, kCachePolicyNT);

  // ---- operands in tile-row order (gathered through the permutation) ------
  const int hk = h / (p.HV / p.HK);
  const uint16_t* kb = p.k + (static_cast<size_t>(b) * p.HK + hk) * D;
  const uint16_t* qb = p.q + (static_cast<size_t>(b) * p.HK + hk) * D;
  const float beta = bf16_to_f32(p.beta[bh]);
  const float alpha = KDA ? 1.0f : expf(bf16_to_f32(p.g[bh]));
  float kk[RPT], qq[RPT], aa[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = rg + RG * i;
    const int u = p.perm ? (static_cast<int>(p.perm[static_cast<size_t>(h) * D + r]) & (D - 1)) : r;
    kk[i] = bf16_to_f32(kb[u]);
    qq[i] = bf16_to_f32(qb[u]);
    aa[i] = KDA ? expf(bf16_to_f32(p.g[bh * D + u])) : alpha;
  }
  float qk = 0.0f;  // q~ . k~ = q . k (permutation invariant)
  for (int e = lane; e < D; e += 64) qk = fmaf(bf16_to_f32(qb[e]), bf16_to_f32(kb[e]), qk);
  qk = wave_sum(qk);

  // ---- decay and the partial read-outs over this thread's 4 rows ----------
  float x[RPT][CPT];  // x[i][4 jj + e]: row rg + 32 i, column 32 jj + 4 cg + e
#pragma unroll
  for (int i = 0; i < RPT; ++i)
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
#pragma unroll
      for (int e = 0; e < 4; ++e) x[i][4 * jj + e] = aa[i] * __uint_as_float(raw[i][jj][e]);
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
    for (int jj = 0; jj < 4; ++jj) {
      const int c = 32 * jj + 4 * cg;
      *reinterpret_cast<float4*>(&red[rg][c]) =
          make_float4(pw[4 * jj], pw[4 * jj + 1], pw[4 * jj + 2], pw[4 * jj + 3]);
      *reinterpret_cast<float4*>(&red[rg][D + c]) =
          make_float4(pq[4 * jj], pq[4 * jj + 1], pq[4 * jj + 2], pq[4 * jj + 3]);
    }
  }
  __syncthreads();

  // ---- column totals: w = S_bar^T k~ (t < D), S_bar^T q~ (D <= t < 2D) ----
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int g = 0; g < RG; ++g) acc[g & 3] += red[g][t];
  const float tot = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  if (t < D) dsh[t] = bf16_to_f32(p.v[bh * D + t]) - tot;  // delta = v - S_bar^T k~
  __syncthreads();
  if (t >= D) write_o(t - D, p.scale * fmaf(beta * qk, dsh[t - D], tot));

  // ---- rank-1 update S' = S_bar + beta k~ delta^T and the store -----------
  float dl[CPT];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    const float4 d4 = *reinterpret_cast<const float4*>(&dsh[32 * jj + 4 * cg]);
    dl[4 * jj] = d4.x;
    dl[4 * jj + 1] = d4.y;
    dl[4 * jj + 2] = d4.z;
    dl[4 * jj + 3] = d4.w;
  }
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const float bk = beta * kk[i];
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      u32x4 w;
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = __float_as_uint(fmaf(bk, dl[4 * jj + e], x[i][4 * jj + e]));
      __builtin_amdgcn_raw_buffer_store_b128(w, rs, off(i, jj), 0, kStorePolicy);
    }
  }
}

}  // namespace

void launch_fp32_128(bool kda, const UpdateParams& p, int B, hipStream_t stream) {
  if (kda)
    hipLaunchKernelGGL(update_fp32_128<true>, dim3(p.HV, B), dim3(256), 0, stream, p);
  else
    hipLaunchKernelGGL(update_fp32_128<false>, dim3(p.HV, B), dim3(256), 0, stream, p);
}

}  // namespace damp
