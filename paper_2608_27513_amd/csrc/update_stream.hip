// Persistent, software-pipelined decode-step update for d_k = d_v = 128 mixed
// tiles with at most 32 high-precision rows (section 3.1 Eq. (1)-(2);
// section 3.2 Eq. (3); section 5.2 and App. A.5), in the default tiers or
// the UINT8, UINT4, FP8 and NVFP4 rows of App. A.1's format table.
//
// The state update moves ~2.4 bytes per state value and does ~11 VALU
// instructions per value, so on MI355X the memory time and the VALU time are
// of the same size; the kernel must overlap them. Each workgroup (4 wave64)
// is resident for the whole launch and walks the tiles (b, h) with a fixed
// value head h = blockIdx.x mod HV, so the channel permutation and the row
// offsets are computed once. While tile k is reduced, updated, re-encoded
// and stored, the packed bytes of the next one or two tiles are already in
// flight into registers.
//
// Tiles are read and written through buffer resources whose size is the tile
// size, or 0 for a padded request: then the loads return zeros and the
// stores are dropped by the hardware, so every thread issues the same
// memory instructions for every tile. Loads and stores of the state are
// non-temporal: each tile is touched once per step.
//
// Per tile: thread t (row group rg = t / 8, column group cg = t % 8) holds
// rows rg, rg+32, rg+64, rg+96, columns 16 cg .. 16 cg + 15. Row 0 of a thread
// can be in the high (16-bit) tier, the others are low rows (codes of one
// byte, or half a byte for UINT4).
// Operands are staged once per tile by two waves (one tile row per thread):
// k~, q~, the row decay a~ and v, in LDS; q~ . k~ is reduced there too.
#include <type_traits>

#include "device.hpp"
#include "internal.hpp"
#include "update.hpp"

namespace damp {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kCachePolicyNT = 2;           // non-temporal loads
// Stores of the state: non-temporal and at device (sc1) coherence scope.
// Measured against non-temporal alone in one run: GDN B=256 -0.6 us, KDA
// -0.5 us, B=1024 -1.8 us; without the non-temporal bit +2 to +7 us.
constexpr int kStorePolicy = 2 | 16;
constexpr int kBufferConfig = 0x00020000;   // raw 32-bit buffer (gfx9 family)

// Workgroup barrier ordering LDS only (global loads stay in flight). The
// scheduling fences keep the compiler from hoisting uses of prefetched
// values above it, which would wait on their latency here.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  __builtin_amdgcn_sched_barrier(0);
}

// voff: per-lane byte offset; soff: wave-uniform byte offset
__device__ __forceinline__ u32x4 ld16(__amdgpu_buffer_rsrc_t r, int voff, int soff = 0) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kCachePolicyNT);
}
__device__ __forceinline__ u32x2 ld8(__amdgpu_buffer_rsrc_t r, int voff, int soff = 0) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, kCachePolicyNT);
}
__device__ __forceinline__ void st16(u32x4 v, __amdgpu_buffer_rsrc_t r, int voff, int soff = 0) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, voff, soff, kStorePolicy);
}
__device__ __forceinline__ void st8(u32x2 v, __amdgpu_buffer_rsrc_t r, int voff, int soff = 0) {
  __builtin_amdgcn_raw_buffer_store_b64(v, r, voff, soff, kStorePolicy);
}

// Cross-lane sums used by the key-axis reduction. fold32(a, b) returns, on
// lanes 0..31, a summed over the lane pair (L, L + 32) and, on lanes 32..63,
// b summed over the pair; fold16 does the same for lane pairs (L, L ^ 16)
// (even 16-lane rows keep a, odd rows keep b) and fold8 for (L, L ^ 8)
// (lanes with bit 3 clear keep a). Each halves the number of live partial
// sums while it halves the number of lanes holding a partial of one value.
__device__ __forceinline__ float fold32(float a, float b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float fold16(float a, float b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float fold8(float a, float b, bool upper) {
  const float send = upper ? a : b, keep = upper ? b : a;
  // row_ror:8 reads lane L ^ 8 of the same 16-lane row
  return keep + __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(send), 0x128, 0xf, 0xf,
                                                        true));
}

// One butterfly stage between lanes L and L ^ 16: v_permlane16_swap of x
// with itself leaves (own, partner) on even 16-lane rows and (partner, own)
// on odd ones, so the lower lane keeps own + partner and the upper lane
// (`upper`, odd row) partner - own.
__device__ __forceinline__ float swap16_butterfly(float x, bool upper) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaf(__uint_as_float(r[1]), upper ? -1.0f : 1.0f, __uint_as_float(r[0]));
}

// Largest of a non-negative value over the 64 lanes of a wave, returned to
// every lane: butterflies within rows of 16 lanes, then row broadcasts (the
// lanes they do not write keep 0, the identity for non-negative values).
__device__ __forceinline__ float wave_max_nonneg(float x) {
  x = fmaxf(x, dpp_mov<0xb1>(x));   // quad_perm [1,0,3,2]
  x = fmaxf(x, dpp_mov<0x4e>(x));   // quad_perm [2,3,0,1]
  x = fmaxf(x, dpp_mov<0x141>(x));  // row_half_mirror
  x = fmaxf(x, dpp_mov<0x140>(x));  // row_mirror: every lane holds its row's max
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x142, 0xa, 0xf,
                                                          false)));
  x = fmaxf(x, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x143, 0xc, 0xf,
                                                          false)));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

// Packed bytes of one tile as loaded by one thread: row slot 0 (the first
// 16 bytes of a 16-bit row slice, or its codes: 16 bytes, 4-bit codes 8 in
// .xy), the codes of slots 1..3 (16 bytes, 4-bit codes 8), the second half
// of a 16-bit row slot 0, the metadata of one row of its wave (the (s, z)
// pair of the default tiers or NVFP4's eight block scales: 8 bytes; the four
// words of the groups of 32: 16 bytes) and NVFP4's global scale.
template <int FMT>
struct RawSetT {
  using Codes =
      typename std::conditional<FMT == kInt4 || FMT == kNvfp4, u32x2, u32x4>::type;
  u32x4 ra0;
  Codes rc[3];
  u32x4 rb0 = u32x4{0u, 0u, 0u, 0u};
  typename std::conditional<FMT == kMixed || FMT == kNvfp4, u32x2, u32x4>::type rm;
  uint32_t gs = 0u;
};

// Sixteen low-tier values of one row slice from their codes: A c + B0 for
// the integer codes (UINT8; UINT4 nibble j of word k is value 8 k + j), A c
// for E4M3 and E2M1 (B0 unused; E2M1 nibbles in the same order). A and B0
// fold the decay into the dequantization.
template <int FMT, typename W>
__device__ __forceinline__ void decode16(const W& w, float A, float B0, float (&x)[16]) {
  if constexpr (FMT == kInt4) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      uint32_t ev = w[k] & 0x0f0f0f0fu, od = (w[k] >> 4) & 0x0f0f0f0fu;
      // opaque to the optimizer, which would otherwise extract each nibble
      // with its own bit-field instruction instead of v_cvt_f32_ubyte{m}
      asm("" : "+v"(ev), "+v"(od));
      x[8 * k + 0] = fmaf(A, ubyte<0>(ev), B0);
      x[8 * k + 1] = fmaf(A, ubyte<0>(od), B0);
      x[8 * k + 2] = fmaf(A, ubyte<1>(ev), B0);
      x[8 * k + 3] = fmaf(A, ubyte<1>(od), B0);
      x[8 * k + 4] = fmaf(A, ubyte<2>(ev), B0);
      x[8 * k + 5] = fmaf(A, ubyte<2>(od), B0);
      x[8 * k + 6] = fmaf(A, ubyte<3>(ev), B0);
      x[8 * k + 7] = fmaf(A, ubyte<3>(od), B0);
    }
  } else if constexpr (FMT == kNvfp4) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      float e[8];
      e2m1_byte<0>(w[k], e[0], e[1]);
      e2m1_byte<1>(w[k], e[2], e[3]);
      e2m1_byte<2>(w[k], e[4], e[5]);
      e2m1_byte<3>(w[k], e[6], e[7]);
#pragma unroll
      for (int j = 0; j < 8; ++j) x[8 * k + j] = A * e[j];
    }
  } else if constexpr (FMT == kFp8) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const auto lo = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w[k]), false);
      const auto hi = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w[k]), true);
      x[4 * k + 0] = A * lo[0];
      x[4 * k + 1] = A * lo[1];
      x[4 * k + 2] = A * hi[0];
      x[4 * k + 3] = A * hi[1];
    }
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[4 * k + 0] = fmaf(A, ubyte<0>(w[k]), B0);
      x[4 * k + 1] = fmaf(A, ubyte<1>(w[k]), B0);
      x[4 * k + 2] = fmaf(A, ubyte<2>(w[k]), B0);
      x[4 * k + 3] = fmaf(A, ubyte<3>(w[k]), B0);
    }
  }
}

// A 16-bit value that is the same for the whole workgroup, through the scalar
// cache: the 4-byte word holding it (aligned down, so it never crosses a
// page the value is not on) and the value's half of it.
__device__ __forceinline__ uint32_t sload_u16(const uint16_t* base, size_t i) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(base + i);
  const __attribute__((address_space(4))) uint32_t* w =
      (const __attribute__((address_space(4))) uint32_t*)(a & ~static_cast<uintptr_t>(3));
  return (*w >> ((a & 2u) * 8u)) & 0xffffu;
}

// Operands of one tile as loaded by the operand threads (raw bf16 bits; beta
// and GDN's g are one value per tile, in scalar registers).
struct OpsRegs {
  uint32_t k, q, g, v, beta;
};

// FMT = kMixed: the default tiers (BF16 high rows, one fp32 (s, z) per low
// row). The group formats of App. A.1's table, each with FP16 high rows and
// one 4-byte word per group of 32 low values: FMT = kPaper (UINT8 codes, FP16
// (s, z)), kInt4 (UINT4 codes, FP16 (s, z)), kFp8 (E4M3 codes, one fp32 scale
// of Eq. (16)). FMT = kNvfp4: FP16 high rows, E2M1 codes in blocks of 16
// (one lane's slice) with an E4M3 scale each, and one fp32 global scale per
// tile from the largest magnitude of its updated low tier. With the block-32
// transform (p.had; UINT8 and UINT4 only) the recurrence runs in the
// transformed domain: H is symmetric and orthonormal, so a low row is used as
// stored (s (c - z) of the transformed values) and only the FP16 rows are
// transformed, on load and before the store; v is transformed on staging and
// o transformed back before it is written, both in registers (DPP and row
// swaps between the lanes of a group). Eq. (1) commutes with the
// transform: S H = Lambda S_prev H + beta k (H delta)^T, delta_H = H v - (S_bar
// H)^T k, o = H (S H)^T q.
//
// DEPTH = tiles of packed bytes prefetched into registers. DEPTH = 1 holds
// one raw tile set (168 VGPRs, three workgroups per CU): the shorter
// prologue and the larger resident front win on short streams. DEPTH = 2
// holds two (two workgroups per CU) and hides more latency on long streams.
template <bool KDA, int FMT, int DEPTH>
__global__ __launch_bounds__(256, DEPTH == 1 ? 3 : 2) void update_stream128(
    const UpdateParams p, const int ntiles, const int tile_bytes) {
  constexpr int D = 128, RG = 32, RPT = 4, CPT = 16, TPR = 8;
  constexpr bool kF16 = FMT != kMixed;  // FP16 high rows
  // 16 metadata bytes per low row (one word per group of 32); the default
  // tiers and NVFP4 have 8 (the (s, z) pair, or eight E4M3 block scales)
  constexpr bool kP = FMT == kPaper || FMT == kInt4 || FMT == kFp8;
  constexpr bool kNib = FMT == kInt4 || FMT == kNvfp4;  // two codes per byte
  constexpr int kCodeRow = kNib ? D / 2 : D;  // code bytes per low row
  constexpr int kSlice = kNib ? 8 : 16;       // code bytes per row slice
  using RawSet = RawSetT<FMT>;
  using Codes = typename RawSet::Codes;
  constexpr int kDrop = 0x40000000;  // buffer offset past any tile: the store is dropped
  // Per-wave partial column sums of k~ . S_bar (index c) and q~ . S_bar
  // (index D + c), in the slot order described at the reduction below;
  // double-buffered by tile parity.
  __shared__ float4 part[2][4][2 * D / 4];
  __shared__ float4 dwv[4][D / 4];  // per wave: delta, same slot order
  // Operands, triple-buffered: row r (k~_r, q~_r, a~_r), column c v_c, and
  // the scalars beta, alpha (GDN) and two partial sums of q~ . k~.
  __shared__ float4 opr[3][D];
  __shared__ float vsh[3][D];
  __shared__ float opsc[3][4];
  // Per wave: the metadata of its 32 rows (8 wave + j + 32 i at index j +
  // 8 i) of the next tile as loaded: 8 bytes per row ((s, z) pairs, NVFP4's
  // block scales), or ([0]) the four words of the groups, which also pass
  // through [1] as re-encoded.
  __shared__ float2 msh[4][kP ? 1 : 32];
  __shared__ u32x4 mshp[4][2][kP ? 32 : 1];
  // 8-byte metadata: the re-encoded rows of a tile, by tile parity, stored
  // after the next tile's workgroup barrier as whole lines.
  __shared__ float2 mout[2][kP ? 1 : D];
  // NVFP4: each wave's largest magnitude of the updated low tier, by tile
  // parity, for the tile's global scale
  __shared__ float amx[2][4];
  // Per wave: its 8 high rows (slot 0) in tile order, 2 KB, for the
  // exchange between the lane layout and whole 1 KB loads and stores.
  __shared__ u32x4 hsh[4][2 * 64];
  __shared__ float osh[D];  // o of the tile (output wave), staged for one whole-row store
  const bool had = (FMT == kPaper || FMT == kInt4) && p.had != 0;

  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int cg = t % TPR, rg = t / TPR, col0 = cg * CPT;
  const bool b3 = (lane & 8) != 0, b4 = (lane & 16) != 0, b5 = (lane & 32) != 0;
  const int HV = p.HV;
  const int G = gridDim.x;  // a multiple of HV
  const int h = blockIdx.x % HV;
  const int hk = h / (HV / p.HK);
  const int B = ntiles / HV;
  const int b_step = G / HV;
  const int k_hi = p.k_hi;
  const bool hi0 = rg < k_hi;  // row slot 0 of this thread is in the 16-bit tier
  const int lo0 = k_hi * D * 2;
  const int meta0 = lo0 + (D - k_hi) * kCodeRow;
  const int off_gs = meta0 + (D - k_hi) * 8;  // NVFP4: the tile's fp32 global scale
  constexpr int kMetaRow = kP ? 16 : 8;  // metadata bytes per low row
  const int o_esize = p.o_bf16 ? 2 : 4;
  // slot ids are read-only here: scalar loads through the constant address space
  const __attribute__((address_space(4))) int32_t* slots =
      (const __attribute__((address_space(4))) int32_t*)p.slot_idx;

  // every lane of this wave has a low row slot 0 (no 16-bit second half to
  // load or store), or every lane a high one
  const bool wave_lo = 8 * wave >= k_hi;
  const bool wave_hi = 8 * wave + 8 <= k_hi;
  // Byte offsets of this thread's row slices inside a tile (same for every
  // tile). Row slot 0 is a 16-bit row (two 16-byte halves at off_a0 and
  // off_b0) or a row of codes; rows 1..3 (always low) sit at off_a1 +
  // (i-1) * 32 rows of codes (scalar offsets). A wave whose slot-0 rows are
  // all high (rows 8 wave .. 8 wave + 7, 2 KB of the tile) loads them as two
  // whole 1 KB blocks instead, lane l taking bytes 16 l of each; the rows
  // reach the lane layout through the wave's LDS slice (stage_meta).
  const int off_a0 = wave_hi ? 2048 * wave + 16 * lane
                             : (hi0 ? (rg * D + col0) * 2 : lo0 + (rg - k_hi) * kCodeRow + cg * kSlice);
  const int off_b0 = wave_hi ? off_a0 + 1024 : off_a0 + 16;
  const int off_a1 = lo0 + (rg + RG - k_hi) * kCodeRow + cg * kSlice;
  constexpr int kStepA = RG * kCodeRow;
  const int st_b0 = hi0 ? off_b0 : kDrop;  // second half of a 16-bit row
  // The metadata of the wave's 32 rows moves with one 8-byte access per
  // lane: lane l < 32 handles row 8 wave + (l & 7) + 32 (l >> 3). Rows of
  // the high tier have no metadata: their loads read bytes of the tile that
  // are never used, their stores are dropped.
  const int mrow = 8 * wave + (lane & 7) + 32 * (lane >> 3);
  const int off_m = lane < 32 ? meta0 + (mrow - k_hi) * kMetaRow : kDrop;
  const int st_m = (lane < 32 && mrow >= k_hi) ? off_m : kDrop;
  const int rgw = lane >> 3;  // row group within the wave
  // Two waves stage the operands, one tile row per thread, and one wave writes
  // o. With the paper's tiers the waves holding the 16-bit rows (0 and 1 for
  // k_hi = 16) also transform them, so waves 2 and 3 stage and wave 2 writes
  // (with o transformed in registers: 0.1 us (GDN) and 0.6 us (KDA) faster
  // than wave 1, 1.3 us faster than wave 3 on KDA).
  constexpr int kOpsT = kF16 ? 128 : 0;  // first thread of the operand waves
  constexpr int kOutWave = kF16 ? 2 : 3;
  const int tr = t - kOpsT;            // tile row of an operand thread
  const bool ops_thread = tr >= 0 && tr < D;
  const int my_u =
      (ops_thread && p.perm) ? (static_cast<int>(p.perm[h * D + tr]) & (D - 1)) : (tr & (D - 1));

  // Reduction slots: after the in-wave folds, lane (cg, b3, b4, b5) holds the
  // wave's partial sums of kind b5 (0: k~, 1: q~) for the columns
  // col0 + 8 hf + 4 b4 + 2 b3 + i, hf, i in {0, 1}; they occupy the four
  // consecutive floats from slot s0 (position 2 hf + i).
  const int c_pair = col0 + 4 * (b4 ? 1 : 0) + 2 * (b3 ? 1 : 0);  // first column of hf = 0
  const int s0q = (b5 ? D / 4 : 0) + cg * 4 + 2 * (b4 ? 1 : 0) + (b3 ? 1 : 0);  // float4 index
  const int dq = cg * 4 + 2 * (b4 ? 1 : 0) + (b3 ? 1 : 0);  // float4 index of delta in dwv
  // o: the q-kind lanes of the output wave hold columns c_pair + {0, 1} and c_pair + 8 + {0, 1}
  auto wave_sync = [] {  // orders the wave's own LDS accesses
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
  };

  if (static_cast<int>(blockIdx.x) >= ntiles) return;

  // ---- operand staging: the operand threads gather one tile row each
  auto issue_ops = [&](OpsRegs& r, int b_) {
    const size_t bh = static_cast<size_t>(b_) * HV + h;
    r.beta = sload_u16(p.beta, bh);
    if (!KDA) r.g = sload_u16(p.g, bh);
    if (ops_thread) {
      const size_t kq = (static_cast<size_t>(b_) * p.HK + hk) * D;
      r.k = p.k[kq + my_u];
      r.q = p.q[kq + my_u];
      if (KDA) r.g = p.g[bh * D + my_u];
      r.v = p.v[bh * D + tr];
    }
  };
  auto publish_ops = [&](const OpsRegs& r, int buf) {
    if (ops_thread) {
      const float kf = bf16_to_f32(static_cast<uint16_t>(r.k));
      const float qf = bf16_to_f32(static_cast<uint16_t>(r.q));
      const float gf = bf16_to_f32(static_cast<uint16_t>(r.g));
      opr[buf][tr] = make_float4(kf, qf, KDA ? __expf(gf) : 1.0f, 0.0f);
      float vf = bf16_to_f32(static_cast<uint16_t>(r.v));
      if (had) {  // v in the transformed domain: 32 consecutive lanes hold a group
        // one butterfly per lane bit: the partner through DPP (lane ^ 1,
        // ^ 2, ^ 4 as two mirrors, ^ 8) or the row swap (^ 16); the lane
        // with the bit set keeps partner - own, the other own + partner
        vf = fmaf(vf, (tr & 1) ? -1.0f : 1.0f, dpp_mov<0xb1>(vf));
        vf = fmaf(vf, (tr & 2) ? -1.0f : 1.0f, dpp_mov<0x4e>(vf));
        vf = fmaf(vf, (tr & 4) ? -1.0f : 1.0f, dpp_mov<0x1b>(dpp_mov<0x141>(vf)));
        vf = fmaf(vf, (tr & 8) ? -1.0f : 1.0f, dpp_mov<0x128>(vf));
        vf = swap16_butterfly(vf, (tr & 16) != 0);
        vf *= kInvSqrt32;
      }
      vsh[buf][tr] = vf;
      const float kq = wave_sum_dpp(kf * qf);
      if ((tr & 63) == 0) opsc[buf][2 + (tr >> 6)] = kq;
      if (tr == 0) {
        opsc[buf][0] = bf16_to_f32(static_cast<uint16_t>(r.beta));
        opsc[buf][1] = KDA ? 1.0f : __expf(gf);
      }
    }
  };

  // ---- packed tile loads into registers -----------------------------------
  auto make_rsrc = [&](int slot_) {
    const bool live = slot_ >= 0 && slot_ < p.num_slots;
    uint8_t* base = p.layer_base + static_cast<size_t>(live ? slot_ : 0) * p.slot_stride +
                    static_cast<size_t>(h) * p.tile_stride;
    return __builtin_amdgcn_make_buffer_rsrc(base, 0, live ? tile_bytes : 0, kBufferConfig);
  };
  // The loads of a tile in four parts (metadata and row slot 0, then one
  // slot of codes each), issued at four points of the previous tile's
  // computation: a burst of them would stall the wave on the full
  // address queue while it has arithmetic to do.
  auto issue_raw_part = [&](RawSet& rs, __amdgpu_buffer_rsrc_t r, int part) {
    if (part == 0) {
      if constexpr (kP) rs.rm = ld16(r, off_m);
      else rs.rm = ld8(r, off_m);
      if constexpr (FMT == kNvfp4)
        rs.gs = __builtin_amdgcn_raw_buffer_load_b32(r, off_gs, 0, kCachePolicyNT);
      if (kNib && wave_lo) {
        const u32x2 c = ld8(r, off_a0);
        rs.ra0 = __builtin_shufflevector(c, c, 0, 1, -1, -1);
      } else {
        rs.ra0 = ld16(r, off_a0);
      }
      if (!wave_lo) rs.rb0 = ld16(r, off_b0);
    } else if constexpr (kNib) {
      rs.rc[part - 1] = ld8(r, off_a1, (part - 1) * kStepA);
    } else {
      rs.rc[part - 1] = ld16(r, off_a1, (part - 1) * kStepA);
    }
  };
  auto issue_raw = [&](RawSet& rs, __amdgpu_buffer_rsrc_t r) {
#pragma unroll
    for (int part = 0; part < RPT; ++part) issue_raw_part(rs, r, part);
  };
  // metadata of a prefetched tile into the wave's LDS slice; the high rows
  // of a wave_hi wave from whole blocks into the lane layout (row lane / 8,
  // columns 16 (lane % 8) ..)
  auto stage_meta = [&](RawSet& rs) {
    if (lane < 32) {
      if constexpr (kP) mshp[wave][0][lane] = rs.rm;
      else msh[wave][lane] = make_float2(__uint_as_float(rs.rm.x), __uint_as_float(rs.rm.y));
    }
    if (wave_hi) {
      hsh[wave][lane] = rs.ra0;
      hsh[wave][64 + lane] = rs.rb0;
    }
    wave_sync();
    if (wave_hi) {
      rs.ra0 = hsh[wave][2 * lane];
      rs.rb0 = hsh[wave][2 * lane + 1];
    }
  };
  auto slot_of = [&](int b_) { return b_ < B ? slots[b_] : -1; };

  // ---- one tile (request b): its packed bytes are in `cur`; with DEPTH = 2
  // those of the next tile are in flight in `oth` (with DEPTH = 1, `oth` is
  // `cur`). Once `cur` is dequantized it receives the bytes DEPTH tiles
  // ahead, in four parts over this tile's arithmetic. Its operands are in
  // buffer `buf`; those of the next tile are in flight in `pub` and are
  // published into buffer `buf_n`; those two tiles ahead are loaded into
  // `nxt`.
  int b = blockIdx.x / HV;
  int slot_cur = slot_of(b);
  int slot_n1 = slot_of(b + b_step);
  int slot_n2 = slot_of(b + 2 * b_step);
  __amdgpu_buffer_rsrc_t rs_cur = make_rsrc(slot_cur);
  __amdgpu_buffer_rsrc_t rs_n1 = make_rsrc(slot_n1);
  bool done = false;
  int buf = 0, pb = 0;
  // The re-encoded 8-byte metadata of a tile (the default tiers' (s, z),
  // NVFP4's block scales) are stored after the next tile's workgroup
  // barrier, when every wave's rows are in mout: wave w writes the 256
  // contiguous bytes of rows k_hi + 32 w ..
  __amdgpu_buffer_rsrc_t rs_prev = make_rsrc(-1);
  auto store_prev_meta = [&](int pbuf, int ln) {
    if constexpr (!kP) {
      const int r = k_hi + 32 * wave + ln;
      const bool on = ln < 32 && r < D;
      const float2 mo = mout[pbuf][on ? r : 0];
      st8(u32x2{__float_as_uint(mo.x), __float_as_uint(mo.y)}, rs_prev,
          on ? meta0 + (32 * wave + ln) * 8 : kDrop);
    }
  };
  int turn = b % 3;

  auto tile = [&](OpsRegs& pub, OpsRegs& nxt, RawSet& cur, RawSet& oth) {
    // The wave arbiter favours older waves, so the workgroups sharing a CU
    // would otherwise progress at very different rates and the last ones
    // would finish alone. Rotating the in-kernel wave priority every tile
    // lets them take turns.
    switch (turn) {
      case 0: __builtin_amdgcn_s_setprio(0); break;
      case 1: __builtin_amdgcn_s_setprio(1); break;
      default: __builtin_amdgcn_s_setprio(2); break;
    }
    turn = turn == 2 ? 0 : turn + 1;
    const int buf_n = buf == 2 ? 0 : buf + 1;
    const bool live = slot_cur >= 0 && slot_cur < p.num_slots;
    // -- operands of this tile; dequantize and decay: S_bar = Lambda S
    float kk[RPT], qq[RPT], aa[RPT];
    const float alpha = opsc[buf][1];
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const float4 o4 = opr[buf][rg + RG * i];
      kk[i] = o4.x;
      qq[i] = o4.y;
      aa[i] = KDA ? o4.z : alpha;
    }
    // per row slot: the dequantization of this lane's slice, A c + B0 (or A c
    // for E4M3 and E2M1), with the decay folded in
    float dA[RPT], dB[RPT];
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      if constexpr (FMT == kNvfp4) {  // this lane's block: its E4M3 scale times the global one
        const uint32_t sb =
            reinterpret_cast<const uint8_t*>(&msh[wave][0])[(rgw + 8 * i) * 8 + cg];
        dA[i] = aa[i] * (e4m3_byte<0>(sb) * __uint_as_float(cur.gs));
        dB[i] = 0.0f;
      } else if constexpr (kP) {  // this lane's group: one word
        const uint32_t m = reinterpret_cast<const uint32_t*>(&mshp[wave][0][0])[(rgw + 8 * i) * 4 +
                                                                               (cg >> 1)];
        if constexpr (FMT == kFp8) {
          dA[i] = aa[i] * __uint_as_float(m);
          dB[i] = 0.0f;
        } else {
          dA[i] = aa[i] * f16_lo(m);
          dB[i] = -dA[i] * f16_hi(m);
        }
      } else {
        const float2 sz = msh[wave][rgw + 8 * i];
        dA[i] = aa[i] * sz.x;
        dB[i] = -dA[i] * sz.y;
      }
    }
    float x[RPT][CPT];
    const u32x4 ra0 = cur.ra0;
    if (hi0) {
      if constexpr (kF16) {  // FP16 rows, into the transformed domain with had
        const float a0 = aa[0] * (had ? kInvSqrt32 : 1.0f);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          x[0][2 * j] = a0 * f16_lo(ra0[j]);
          x[0][2 * j + 1] = a0 * f16_hi(ra0[j]);
          x[0][8 + 2 * j] = a0 * f16_lo(cur.rb0[j]);
          x[0][8 + 2 * j + 1] = a0 * f16_hi(cur.rb0[j]);
        }
        if (had) fwht32_pair(x[0], (cg & 1) != 0);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          x[0][2 * j] = aa[0] * bf16_lo(ra0[j]);
          x[0][2 * j + 1] = aa[0] * bf16_hi(ra0[j]);
          x[0][8 + 2 * j] = aa[0] * bf16_lo(cur.rb0[j]);
          x[0][8 + 2 * j + 1] = aa[0] * bf16_hi(cur.rb0[j]);
        }
      }
    } else if constexpr (kNib) {
      decode16<FMT>(u32x2{ra0.x, ra0.y}, dA[0], dB[0], x[0]);
    } else {
      decode16<FMT>(ra0, dA[0], dB[0], x[0]);
    }
#pragma unroll
    for (int i = 1; i < RPT; ++i) decode16<FMT>(cur.rc[i - 1], dA[i], dB[i], x[i]);
    // the dequantized tile must exist before the next tile's loads are
    // issued, so that the waits for this tile's bytes precede the prefetch
#pragma unroll
    for (int i = 0; i < RPT; ++i)
      asm volatile("" ::"v"(x[i][0]), "v"(x[i][1]), "v"(x[i][2]), "v"(x[i][3]), "v"(x[i][4]),
                   "v"(x[i][5]), "v"(x[i][6]), "v"(x[i][7]), "v"(x[i][8]), "v"(x[i][9]),
                   "v"(x[i][10]), "v"(x[i][11]), "v"(x[i][12]), "v"(x[i][13]), "v"(x[i][14]),
                   "v"(x[i][15]));

    // -- prefetch: the packed bytes DEPTH tiles ahead (the first part here,
    // the others between the read-out halves and after the barrier) and the
    // operands two tiles ahead
    const int b_n = b + b_step;
    const bool has_next = b_n < B;
    const bool has_next2 = b_n + b_step < B;
    __amdgpu_buffer_rsrc_t rs_n2 = rs_n1;
    int slot_n3 = -1;
    if (has_next2) rs_n2 = make_rsrc(slot_n2);
    const bool pf = DEPTH == 1 ? has_next : has_next2;
    const __amdgpu_buffer_rsrc_t rs_pf = DEPTH == 1 ? rs_n1 : rs_n2;
    if (pf) issue_raw_part(cur, rs_pf, 0);
    if (has_next2) {
      issue_ops(nxt, b_n + b_step);
      slot_n3 = slot_of(b_n + 2 * b_step);
    }
    __builtin_amdgcn_sched_barrier(0);

    // -- partial key and query read-outs over this thread's 4 rows, folded
    // over the 8 row groups of the wave (lane bits 5, 4, 3), so each lane
    // keeps 4 of the wave's 256 partial sums
    float r3[4];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      float pw[8], pq[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        pw[j] = kk[0] * x[0][8 * hf + j];
        pq[j] = qq[0] * x[0][8 * hf + j];
      }
#pragma unroll
      for (int i = 1; i < RPT; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          pw[j] = fmaf(kk[i], x[i][8 * hf + j], pw[j]);
          pq[j] = fmaf(qq[i], x[i][8 * hf + j], pq[j]);
        }
      float r1[8], r2[4];
#pragma unroll
      for (int j = 0; j < 8; ++j) r1[j] = fold32(pw[j], pq[j]);  // kind b5, column 8 hf + j
#pragma unroll
      for (int j = 0; j < 4; ++j) r2[j] = fold16(r1[j], r1[j + 4]);  // column 8 hf + 4 b4 + j
#pragma unroll
      for (int j = 0; j < 2; ++j) r3[2 * hf + j] = fold8(r2[j], r2[j + 2], b3);
      __builtin_amdgcn_sched_barrier(0);
      if (pf) issue_raw_part(cur, rs_pf, 1 + hf);
      __builtin_amdgcn_sched_barrier(0);
    }
    part[pb][wave][s0q] = make_float4(r3[0], r3[1], r3[2], r3[3]);
    if (has_next) publish_ops(pub, buf_n);  // loaded a whole tile ago
    lds_barrier();
    store_prev_meta(pb ^ 1, lane);
    if (pf) issue_raw_part(cur, rs_pf, 3);

    // -- column totals of this lane's 4 slots over the 4 waves (the k lanes:
    // S_bar^T k~, the q lanes: S_bar^T q~); delta = v - S_bar^T k~ on the k
    // lanes
    float tot[4], dd[4];
    {
      const float4 p0 = part[pb][0][s0q], p1 = part[pb][1][s0q];
      const float4 p2 = part[pb][2][s0q], p3 = part[pb][3][s0q];
      tot[0] = (p0.x + p1.x) + (p2.x + p3.x);
      tot[1] = (p0.y + p1.y) + (p2.y + p3.y);
      tot[2] = (p0.z + p1.z) + (p2.z + p3.z);
      tot[3] = (p0.w + p1.w) + (p2.w + p3.w);
      const float2 v0 = *reinterpret_cast<const float2*>(&vsh[buf][c_pair]);
      const float2 v1 = *reinterpret_cast<const float2*>(&vsh[buf][c_pair + 8]);
      const float vv[4] = {v0.x, v0.y, v1.x, v1.y};
#pragma unroll
      for (int m = 0; m < 4; ++m) dd[m] = vv[m] - tot[m];
    }
    const float beta = opsc[buf][0];

    // -- output o = scale (S_bar^T q~ + beta (q~.k~) delta), by the output
    // wave: one swap gives its q lanes the delta of their 4 columns
    if (wave == kOutWave) {
      const float bqk = beta * (opsc[buf][2] + opsc[buf][3]);
      const float osc = had ? p.scale * kInvSqrt32 : p.scale;
      float ov[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const float val = b5 ? tot[m] : dd[m];
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(val),
                                                        __float_as_uint(val), false, false);
        ov[m] = live ? osc * fmaf(bqk, __uint_as_float(r[0]), __uint_as_float(r[1])) : 0.0f;
      }
      if (had) {
        // back from the transformed domain. Of a group's 32 columns a q lane
        // holds 4: column bits 0 and 3 are its own (m & 1, m >> 1), bits 4,
        // 1 and 2 are lane bits 0, 3 and 4 (the k lanes, lane bit 5 clear,
        // take part but are not used)
        float t0 = ov[0] + ov[1], t1 = ov[0] - ov[1], t2 = ov[2] + ov[3], t3 = ov[2] - ov[3];
        ov[0] = t0 + t2;
        ov[2] = t0 - t2;
        ov[1] = t1 + t3;
        ov[3] = t1 - t3;
        const float s0 = (lane & 1) ? -1.0f : 1.0f, s3 = b3 ? -1.0f : 1.0f;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          ov[m] = fmaf(ov[m], s0, dpp_mov<0xb1>(ov[m]));
          ov[m] = fmaf(ov[m], s3, dpp_mov<0x128>(ov[m]));
          ov[m] = swap16_butterfly(ov[m], b4);
        }
      }
      uint8_t* obase = static_cast<uint8_t*>(p.o) +
                       (static_cast<size_t>(b) * HV + h) * D * o_esize;
      const __amdgpu_buffer_rsrc_t ro =
          __builtin_amdgcn_make_buffer_rsrc(obase, 0, D * o_esize, kBufferConfig);
      {
        if (b5) {
          *reinterpret_cast<float2*>(&osh[c_pair]) = make_float2(ov[0], ov[1]);
          *reinterpret_cast<float2*>(&osh[c_pair + 8]) = make_float2(ov[2], ov[3]);
        }
        wave_sync();
        // one store writes the whole row: 16 lanes x 16 bytes (bf16) or 32
        // lanes x 16 bytes (fp32); the other lanes' offsets lie past the
        // buffer and are dropped
        const float4* o4 = reinterpret_cast<const float4*>(osh);
        u32x4 ow;
        if (p.o_bf16) {
          const float4 a = o4[2 * (lane & 15)], c = o4[2 * (lane & 15) + 1];
          ow = u32x4{pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w), pack_bf16x2(c.x, c.y),
                     pack_bf16x2(c.z, c.w)};
        } else {
          const float4 a = o4[lane & 31];
          ow = u32x4{__float_as_uint(a.x), __float_as_uint(a.y), __float_as_uint(a.z),
                     __float_as_uint(a.w)};
        }
        __builtin_amdgcn_raw_buffer_store_b128(ow, ro, lane * 16, 0, 0);
      }
    }

    // -- delta of this lane's 16 columns, through the wave's own LDS slice
    // (a wave's LDS accesses complete in order: no barrier)
    if (!b5) dwv[wave][dq] = make_float4(dd[0], dd[1], dd[2], dd[3]);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
    float dl[CPT];
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      // float4 q4 of the lane's block holds columns 4 (q4 >> 1) + 2 (q4 & 1)
      // + {0, 1} and the same + 8
      const float4 d4 = dwv[wave][cg * 4 + q4];
      const int c = 4 * (q4 >> 1) + 2 * (q4 & 1);
      dl[c] = d4.x;
      dl[c + 1] = d4.y;
      dl[c + 8] = d4.z;
      dl[c + 9] = d4.w;
    }

    // -- rank-1 update S' = S_bar + beta k~ delta^T, re-encode, store in place
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const float bk = beta * kk[i];
#pragma unroll
      for (int j = 0; j < CPT; ++j) x[i][j] = fmaf(bk, dl[j], x[i][j]);
    }
    // NVFP4: the tile's global scale from the largest magnitude of its
    // updated low tier, over the workgroup (one more barrier); the block
    // maxima are kept for the block scales
    float bmx[RPT];
    float s_g = 1.0f, d6 = 6.0f, rd6 = 1.0f;
    if constexpr (FMT == kNvfp4) {
      float am = 0.0f;
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        float m = fabsf(x[i][0]);
#pragma unroll
        for (int j = 1; j < CPT; ++j) m = fmaxf(m, fabsf(x[i][j]));
        bmx[i] = m;
        if (i > 0 || !hi0) am = fmaxf(am, m);
      }
      am = wave_max_nonneg(am);
      if (lane == 0) amx[pb][wave] = am;
      lds_barrier();
      s_g = nvfp4_global(fmaxf(fmaxf(amx[pb][0], amx[pb][1]), fmaxf(amx[pb][2], amx[pb][3])));
      d6 = 6.0f * s_g;
      rd6 = refined_rcp(d6);
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(s_g), rs_cur, t == 0 ? off_gs : kDrop,
                                            0, kStorePolicy);
    }
    u32x4 wa0, wb0;
    Codes wc[RPT];
    float2 wm[RPT];    // default tiers: the row's (s, z)
    uint32_t wg[RPT];  // group formats: the word of this lane's group
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      if (i == 0 && hi0) {
        if constexpr (kF16) {  // FP16 rows, back from the transformed domain with had
          if (had) {
            fwht32_pair(x[0], (cg & 1) != 0);
#pragma unroll
            for (int j = 0; j < CPT; ++j) x[0][j] *= kInvSqrt32;
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            wa0[j] = pack_f16x2(x[0][2 * j], x[0][2 * j + 1]);
            wb0[j] = pack_f16x2(x[0][8 + 2 * j], x[0][8 + 2 * j + 1]);
          }
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            wa0[j] = pack_bf16x2(x[0][2 * j], x[0][2 * j + 1]);
            wb0[j] = pack_bf16x2(x[0][8 + 2 * j], x[0][8 + 2 * j + 1]);
          }
        }
        wm[0] = make_float2(0.0f, 0.0f);
        wg[0] = 0u;
        continue;
      }
      if constexpr (FMT == kNvfp4) {
        // the block scale E4M3(min(amax / (6 s_g), 448)) (the quotient from
        // the refined reciprocal), codes E2M1(x / scale), zero codes under a
        // zero scale
        float tq = bmx[i] * rd6;
        tq = fmaf(fmaf(-tq, d6, bmx[i]), rd6, tq);
        const uint32_t sb = cvt_e4m3x2<false>(fminf(tq, 448.0f), 0.0f, 0u) & 0xffu;
        const float scale = e4m3_byte<0>(sb) * s_g;
        const bool nz = scale > 0.0f;
        const float inv = nz ? refined_rcp(scale) : 0.0f;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const float* y = &x[i][8 * k];
          uint32_t v = cvt_e2m1x2<0>(y[0] * inv, y[1] * inv, 0u);
          v = cvt_e2m1x2<1>(y[2] * inv, y[3] * inv, v);
          v = cvt_e2m1x2<2>(y[4] * inv, y[5] * inv, v);
          v = cvt_e2m1x2<3>(y[6] * inv, y[7] * inv, v);
          wc[i][k] = nz ? v : 0u;
        }
        wg[i] = sb;
      } else if constexpr (FMT == kFp8) {
        // Eq. (16): s = max |x| / 448 over the lane pair's group of 32
        float amax = fabsf(x[i][0]);
#pragma unroll
        for (int j = 1; j < CPT; ++j) amax = fmaxf(amax, fabsf(x[i][j]));
        amax = fmaxf(amax, dpp_mov<0xb1>(amax));
        // the quotient from a refined reciprocal (IEEE except in rare last-bit cases)
        const float am = amax > 1e-10f ? amax : 1e-10f;
        float s = am * (1.0f / 448.0f);
        s = fmaf(fmaf(-s, 448.0f, am), 1.0f / 448.0f, s);
        const float inv = refined_rcp(s);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t lo = cvt_e4m3x2<false>(x[i][4 * k] * inv, x[i][4 * k + 1] * inv, 0u);
          wc[i][k] = cvt_e4m3x2<true>(x[i][4 * k + 2] * inv, x[i][4 * k + 3] * inv, lo);
        }
        wg[i] = __float_as_uint(s);
      } else {
        float mn = x[i][0], mx = x[i][0];
#pragma unroll
        for (int j = 1; j < CPT; ++j) {
          mn = fminf(mn, x[i][j]);
          mx = fmaxf(mx, x[i][j]);
        }
        float s, z, inv;
        if constexpr (kP) {  // the lane pair's group of 32, FP16 (s, z)
          group_qparams_f16_rcp<kNib ? 15 : 255>(mn, mx, s, z, inv);
          wg[i] = pack_f16x2(s, z);
        } else {
          group_minmax<TPR>(mn, mx);
          row_qparams(mn, mx, s, z, inv);
          wm[i] = make_float2(s, z);
        }
        if constexpr (FMT == kInt4) {
          // codes clamped to [0, 15] before the conversion (it rounds to
          // nearest even), then values 2 m and 2 m + 1 into the nibbles of byte m
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            uint32_t ev = 0u, od = 0u;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
              const float ce = __builtin_amdgcn_fmed3f(fmaf(x[i][8 * k + 2 * m], inv, z), 0.0f, 15.0f);
              const float co =
                  __builtin_amdgcn_fmed3f(fmaf(x[i][8 * k + 2 * m + 1], inv, z), 0.0f, 15.0f);
              ev = __builtin_amdgcn_cvt_pk_u8_f32(ce, m, ev);
              od = __builtin_amdgcn_cvt_pk_u8_f32(co, m, od);
            }
            wc[i][k] = ev | (od << 4);
          }
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            // v_cvt_pk_u8_f32 rounds to nearest even and saturates to [0, 255]
            uint32_t c = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(x[i][4 * j], inv, z), 0, 0u);
            c = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(x[i][4 * j + 1], inv, z), 1, c);
            c = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(x[i][4 * j + 2], inv, z), 2, c);
            wc[i][j] = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(x[i][4 * j + 3], inv, z), 3, c);
          }
        }
      }
      if (i == 0) {
        if constexpr (kNib) wa0 = __builtin_shufflevector(wc[0], wc[0], 0, 1, -1, -1);
        else wa0 = wc[0];
        wb0 = u32x4{0u, 0u, 0u, 0u};
      }
    }
    // metadata of the wave's rows: the group formats' 16 bytes per row go
    // through the wave's LDS slice (a wave's 8 consecutive rows make a whole
    // 128-byte line); 8-byte metadata into the tile's table, stored after the
    // next barrier (store_prev_meta)
    if constexpr (kP) {
      if ((cg & 1) == 0) {
#pragma unroll
        for (int i = 0; i < RPT; ++i)
          reinterpret_cast<uint32_t*>(&mshp[wave][1][0])[(rgw + 8 * i) * 4 + (cg >> 1)] = wg[i];
      }
    } else if constexpr (FMT == kNvfp4) {  // each lane its block's scale byte
#pragma unroll
      for (int i = 0; i < RPT; ++i)
        reinterpret_cast<uint8_t*>(&mout[pb][0])[(rg + RG * i) * 8 + cg] =
            static_cast<uint8_t>(wg[i]);
    } else if (cg == 0) {
#pragma unroll
      for (int i = 0; i < RPT; ++i) mout[pb][rg + RG * i] = wm[i];
    }
    // the high rows of a wave_hi wave as two whole 1 KB blocks
    if (wave_hi) {
      hsh[wave][2 * lane] = wa0;
      hsh[wave][2 * lane + 1] = wb0;
    }
    wave_sync();
    // every lane issues the same stores; lanes with nothing to write use an
    // offset past the buffer, which the hardware drops
    if (wave_hi) {
      st16(hsh[wave][lane], rs_cur, off_a0);
      st16(hsh[wave][64 + lane], rs_cur, off_b0);
    } else if constexpr (kNib) {  // 8 bytes of codes, or 32 of a 16-bit row
      st8(u32x2{wa0.x, wa0.y}, rs_cur, off_a0);
      if (!wave_lo) {
        st8(u32x2{wa0.z, wa0.w}, rs_cur, hi0 ? off_a0 + 8 : kDrop);
        st16(wb0, rs_cur, st_b0);
      }
    } else {
      st16(wa0, rs_cur, off_a0);
      if (!wave_lo) st16(wb0, rs_cur, st_b0);
    }
#pragma unroll
    for (int i = 1; i < RPT; ++i) {
      if constexpr (kNib) st8(wc[i], rs_cur, off_a1, (i - 1) * kStepA);
      else st16(wc[i], rs_cur, off_a1, (i - 1) * kStepA);
    }
    if constexpr (kP) st16(mshp[wave][1][lane & 31], rs_cur, st_m);
    if (has_next) stage_meta(oth);

    done = !has_next;
    b = b_n;
    buf = buf_n;
    pb ^= 1;
    slot_cur = slot_n1;
    slot_n1 = slot_n2;
    slot_n2 = slot_n3;
    rs_prev = rs_cur;
    rs_cur = rs_n1;
    rs_n1 = rs_n2;
  };

  // ---- prologue: the bytes and operands of tile 0 in flight, and those of
  // tile 1 (its bytes only with DEPTH = 2)
  OpsRegs ops_a = {0u, 0u, 0u, 0u, 0u}, ops_b = {0u, 0u, 0u, 0u, 0u};
  RawSet set_a, set_b;
  issue_ops(ops_a, b);
  issue_raw(set_a, rs_cur);
  if (b + b_step < B) {
    if constexpr (DEPTH == 2) issue_raw(set_b, rs_n1);
    issue_ops(ops_b, b + b_step);
  }
  publish_ops(ops_a, 0);
  stage_meta(set_a);
  lds_barrier();

  // two tiles per trip so the operand (and with DEPTH = 2 the raw) register
  // sets alternate without copies
  RawSet& set_2 = DEPTH == 1 ? set_a : set_b;
  for (;;) {
    tile(ops_b, ops_a, set_a, set_2);
    if (done) break;
    tile(ops_a, ops_b, set_2, set_a);
    if (done) break;
  }
  // the last tile's 8-byte metadata, once every wave has put its rows in mout
  if constexpr (!kP) {
    lds_barrier();
    // the lane index afresh: keeping the loop's copy alive to here costs a spill
    store_prev_meta(pb ^ 1, static_cast<int>(__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u))));
  }
}

// The instantiations that launch_stream128 chooses from, and their
// resident workgroups per CU (queried once per device).
enum StreamKernel {
  kGdnMixed1, kGdnMixed2, kKdaMixed1, kKdaMixed2,
  kGdnPaper2, kKdaPaper2, kGdnInt42, kKdaInt42, kGdnFp82, kKdaFp82,
  kGdnNvfp42, kKdaNvfp42, kNumStream
};

template <bool KDA, int FMT, int DEPTH>
const void* kernel_ptr() {
  return reinterpret_cast<const void*>(update_stream128<KDA, FMT, DEPTH>);
}

const void* stream_kernel(int which) {
  switch (which) {
    case kGdnMixed1: return kernel_ptr<false, kMixed, 1>();
    case kGdnMixed2: return kernel_ptr<false, kMixed, 2>();
    case kKdaMixed1: return kernel_ptr<true, kMixed, 1>();
    case kKdaMixed2: return kernel_ptr<true, kMixed, 2>();
    case kGdnPaper2: return kernel_ptr<false, kPaper, 2>();
    case kKdaPaper2: return kernel_ptr<true, kPaper, 2>();
    case kGdnInt42: return kernel_ptr<false, kInt4, 2>();
    case kKdaInt42: return kernel_ptr<true, kInt4, 2>();
    case kGdnFp82: return kernel_ptr<false, kFp8, 2>();
    case kKdaFp82: return kernel_ptr<true, kFp8, 2>();
    case kGdnNvfp42: return kernel_ptr<false, kNvfp4, 2>();
    default: return kernel_ptr<true, kNvfp4, 2>();
  }
}

struct Occupancy {
  int cus = 0;
  int per_cu[kNumStream] = {};
};

bool occupancy(int which, int& cus, int& per_cu) {
  static Occupancy cache[16];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 16) return false;
  Occupancy& c = cache[dev];
  if (c.cus == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return false;
    int a[kNumStream] = {};
    for (int i = 0; i < kNumStream; ++i)
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&a[i], stream_kernel(i), 256, 0) != hipSuccess)
        return false;
    for (int i = 0; i < kNumStream; ++i) c.per_cu[i] = a[i] > 0 ? a[i] : 1;
    c.cus = n;
  }
  cus = c.cus;
  per_cu = c.per_cu[which];
  return true;
}

}  // namespace

bool launch_stream128(bool kda, int fmt, const UpdateParams& p, int B, hipStream_t stream) {
  const int ntiles = B * p.HV;
  int which;
  switch (fmt) {
    case kPaper: which = kda ? kKdaPaper2 : kGdnPaper2; break;
    case kInt4: which = kda ? kKdaInt42 : kGdnInt42; break;
    case kFp8: which = kda ? kKdaFp82 : kGdnFp82; break;
    case kNvfp4: which = kda ? kKdaNvfp42 : kGdnNvfp42; break;
    default: which = kda ? kKdaMixed2 : kGdnMixed2; break;
  }
  int cus = 0, per_cu = 0;
  if (!occupancy(which, cus, per_cu)) return false;
  // The default tiers prefetch one tile with three workgroups per CU when
  // each of the two-per-CU workgroups would stream at most 16 tiles (the
  // batch of 256 requests x 32 heads), two tiles otherwise. The group
  // formats need more registers and always prefetch two.
  if (fmt == kMixed && static_cast<long>(ntiles) <= 16L * cus * per_cu) {
    which = kda ? kKdaMixed1 : kGdnMixed1;
    if (!occupancy(which, cus, per_cu)) return false;
  }
  // resident workgroups, rounded down to a multiple of HV (at least HV)
  const long capacity = static_cast<long>(cus) * per_cu;
  long per_head = capacity / p.HV;
  if (per_head < 1) per_head = 1;
  if (per_head > B) per_head = B;
  // When the batch takes two rounds of tiles, as few workgroups as give
  // every one of them two tiles: one GPU's share of an 8-way tensor-parallel
  // step (1024 tiles) 0.75-0.9 us faster than 768 workgroups of which a
  // third take a second tile; with three or more rounds the same rule was
  // slower (B = 64: +0.7 us), with one it changes nothing.
  if ((B + per_head - 1) / per_head == 2) per_head = (B + 1) / 2;
  const int grid = static_cast<int>(per_head * p.HV);
  const int lo_rows = 128 - p.k_hi;
  const bool nib = fmt == kInt4 || fmt == kNvfp4, meta8 = fmt == kMixed || fmt == kNvfp4;
  const int tile_bytes = p.k_hi * 128 * 2 + lo_rows * (nib ? 64 : 128) +
                         lo_rows * (meta8 ? 8 : 16) + (fmt == kNvfp4 ? 4 : 0);
  UpdateParams pa = p;
  int nt = ntiles, tb = tile_bytes;
  void* args[] = {&pa, &nt, &tb};
  return hipLaunchKernel(stream_kernel(which), dim3(grid), dim3(256), args, 0, stream) ==
         hipSuccess;
}

}  // namespace damp
