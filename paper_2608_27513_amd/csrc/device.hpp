// Device helpers of libdamp for gfx950 (CDNA4, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include <cfloat>
#include <cstdint>

namespace damp {

constexpr int kFp32 = 0;   // DAMP_STATE_FP32
constexpr int kMixed = 1;  // DAMP_STATE_MIXED with the default tiers
// DAMP_STATE_MIXED with the paper's tiers (App. A.1, Eq. (17)): FP16 high
// rows; low rows in groups of 32 values with FP16 (s, z), optionally after
// the normalized block-32 Hadamard transform.
constexpr int kPaper = 2;
// The other rows of App. A.1's format table, each with an FP16 high tier:
// INT4 (groups of 32, FP16 (s, z), optional block-32 transform), FP8 E4M3
// (one fp32 scale per group of 32, Eq. (16)) and NVFP4 (E2M1 in blocks of
// 16 with an E4M3 block scale and one fp32 global scale per tile).
constexpr int kInt4 = 3;
constexpr int kFp8 = 4;
constexpr int kNvfp4 = 5;

template <int KIND>
constexpr bool is_nibble() {
  return KIND == kInt4 || KIND == kNvfp4;
}
// Bytes of one low-tier row: codes, then metadata.
template <int KIND, int D>
constexpr int code_row_bytes() {
  return is_nibble<KIND>() ? D / 2 : D;
}
template <int KIND, int D>
constexpr int meta_row_bytes() {
  return KIND == kMixed ? 8 : (KIND == kNvfp4 ? D / 16 : (D / 32) * 4);
}

// ------------------------------------------------------------ conversions

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Two fp32 -> packed bf16 pair, round-to-nearest-even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  f2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, b2));
}

__device__ __forceinline__ uint16_t f32_to_bf16(float a) {
  return static_cast<uint16_t>(pack_bf16x2(a, 0.0f) & 0xffffu);
}

// FP16 halves of a word, and two fp32 -> packed FP16 pair (round to nearest
// even, IEEE overflow to infinity).
__device__ __forceinline__ float f16_lo(uint32_t w) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xffffu)));
}
__device__ __forceinline__ float f16_hi(uint32_t w) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w >> 16)));
}
__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  f2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
}
__device__ __forceinline__ float round_f16(float a) {
  return static_cast<float>(static_cast<_Float16>(a));
}

// Byte i of w as a float (v_cvt_f32_ubyte{i}).
template <int I>
__device__ __forceinline__ float ubyte(uint32_t w) {
  return static_cast<float>((w >> (8 * I)) & 0xffu);
}

// ---------------------------------------------------- lane reductions (DPP)

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, true));
}

// Min and max over aligned groups of N consecutive lanes (N in 1..16).
// quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror.
template <int N>
__device__ __forceinline__ void group_minmax(float& mn, float& mx) {
  if constexpr (N >= 2) {
    mn = fminf(mn, dpp_mov<0xb1>(mn));
    mx = fmaxf(mx, dpp_mov<0xb1>(mx));
  }
  if constexpr (N >= 4) {
    mn = fminf(mn, dpp_mov<0x4e>(mn));
    mx = fmaxf(mx, dpp_mov<0x4e>(mx));
  }
  if constexpr (N >= 8) {
    mn = fminf(mn, dpp_mov<0x141>(mn));
    mx = fmaxf(mx, dpp_mov<0x141>(mx));
  }
  if constexpr (N >= 16) {
    mn = fminf(mn, dpp_mov<0x140>(mn));
    mx = fmaxf(mx, dpp_mov<0x140>(mx));
  }
}

// Sum over the 64 lanes of a wave (every lane receives the total).
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// Sum over the 64 lanes of a wave with DPP only (no LDS traffic): butterfly
// within rows of 16 lanes, then row broadcasts; the total ends in lane 63 and
// is returned to every lane as a wave-uniform value.
__device__ __forceinline__ float wave_sum_dpp(float x) {
  x += dpp_mov<0xb1>(x);   // quad_perm [1,0,3,2]
  x += dpp_mov<0x4e>(x);   // quad_perm [2,3,0,1]
  x += dpp_mov<0x141>(x);  // row_half_mirror
  x += dpp_mov<0x140>(x);  // row_mirror: every lane holds its row's sum
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x142, 0xa, 0xf, false));
  x += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x143, 0xc, 0xf, false));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

// ------------------------------------------------------------- vector I/O

template <int NBYTES>
__device__ __forceinline__ void load_words(const uint8_t* p, uint32_t* w) {
  static_assert(NBYTES % 4 == 0, "word-sized loads only");
  if constexpr (NBYTES % 16 == 0) {
#pragma unroll
    for (int k = 0; k < NBYTES / 16; ++k) {
      const uint4 v = reinterpret_cast<const uint4*>(p)[k];
      w[4 * k + 0] = v.x;
      w[4 * k + 1] = v.y;
      w[4 * k + 2] = v.z;
      w[4 * k + 3] = v.w;
    }
  } else if constexpr (NBYTES == 8) {
    const uint2 v = *reinterpret_cast<const uint2*>(p);
    w[0] = v.x;
    w[1] = v.y;
  } else {
    static_assert(NBYTES == 4, "unsupported width");
    w[0] = *reinterpret_cast<const uint32_t*>(p);
  }
}

template <int NBYTES>
__device__ __forceinline__ void store_words(uint8_t* p, const uint32_t* w) {
  static_assert(NBYTES % 4 == 0, "word-sized stores only");
  if constexpr (NBYTES % 16 == 0) {
#pragma unroll
    for (int k = 0; k < NBYTES / 16; ++k)
      reinterpret_cast<uint4*>(p)[k] = make_uint4(w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]);
  } else if constexpr (NBYTES == 8) {
    *reinterpret_cast<uint2*>(p) = make_uint2(w[0], w[1]);
  } else {
    static_assert(NBYTES == 4, "unsupported width");
    *reinterpret_cast<uint32_t*>(p) = w[0];
  }
}

// ------------------------------------------------- Eq. (3) row quantizer

// Scale, zero point and reciprocal scale of a row with extrema (mn, mx):
// s = (mx - mn) / 255 and z = round(-mn / s) (round half to even). A row
// whose s is not a normal fp32 number uses s = |mn| / 255, else s = 1.
// Both quotients come from a hardware reciprocal refined by one
// residual step, which rounds like IEEE division except in rare last-bit
// cases.
__device__ __forceinline__ void row_qparams(float mn, float mx, float& s, float& z,
                                            float& inv) {
  constexpr float k255inv = 1.0f / 255.0f;
  const float r = mx - mn;
  float q = r * k255inv;
  q = fmaf(fmaf(-q, 255.0f, r), k255inv, q);
  // the fallback runs only in a wave that has such a row (a wave-uniform
  // branch) rather than being evaluated and selected on every row
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(!(q >= FLT_MIN)) != 0, 0)) {
    if (!(q >= FLT_MIN)) {
      const float a = fabsf(mn);
      q = a * k255inv;
      q = fmaf(fmaf(-q, 255.0f, a), k255inv, q);
      if (!(q >= FLT_MIN)) q = 1.0f;
    }
  }
  const float rc = __builtin_amdgcn_rcpf(q);
  const float nm = -mn;
  float zq = nm * rc;
  zq = fmaf(fmaf(-zq, q, nm), rc, zq);
  s = q;
  z = rintf(zq);
  inv = rc;
}

// Code of x: clamp(round(x / s) + z, 0, 255), computed as round(x * (1/s) + z).
__device__ __forceinline__ float quant_code(float x, float inv, float z) {
  return __builtin_amdgcn_fmed3f(rintf(fmaf(x, inv, z)), 0.0f, 255.0f);
}

// Four codes (already integral in [0, 255]) packed little-endian into a word.
__device__ __forceinline__ uint32_t pack_codes4(float c0, float c1, float c2, float c3) {
  uint32_t w = __builtin_amdgcn_cvt_pk_u8_f32(c0, 0, 0u);
  w = __builtin_amdgcn_cvt_pk_u8_f32(c1, 1, w);
  w = __builtin_amdgcn_cvt_pk_u8_f32(c2, 2, w);
  return __builtin_amdgcn_cvt_pk_u8_f32(c3, 3, w);
}

// -------------------------------------- paper low tier (App. A.1, Eq. 17)

constexpr float kInvSqrt32 = 0.17677669529663687f;

// Unnormalized Hadamard transform (Sylvester order) of the 32 values of a
// group held as 16 per lane by the lane pair (L, L ^ 1); `upper` is true on
// the lane holding values 16..31. Four butterfly stages in the lane, the
// fifth across the pair.
__device__ __forceinline__ void fwht32_pair(float (&x)[16], bool upper) {
#pragma unroll
  for (int m = 1; m < 16; m <<= 1)
#pragma unroll
    for (int j = 0; j < 16; ++j)
      if (!(j & m)) {
        const float a = x[j], b = x[j | m];
        x[j] = a + b;
        x[j | m] = a - b;
      }
  const float sgn = upper ? -1.0f : 1.0f;
#pragma unroll
  for (int j = 0; j < 16; ++j) x[j] = fmaf(sgn, x[j], dpp_mov<0xb1>(x[j]));
}

// Stored (s, z) of one group of 32 values held by a lane pair, given the
// lane's extrema, and the reciprocal of the stored scale: s from Eq. (3) in
// fp32 (constant groups as for rows), rounded to FP16 and kept positive and
// finite; z = round(-min / s) from the stored s, within FP16's finite range,
// rounded to FP16. Divisions are IEEE (a few per group).
template <int LEVELS = 255>
__device__ __forceinline__ void group_qparams_f16(float mn, float mx, float& s16, float& z16,
                                                  float& inv) {
  mn = fminf(mn, dpp_mov<0xb1>(mn));
  mx = fmaxf(mx, dpp_mov<0xb1>(mx));
  float s = (mx - mn) / static_cast<float>(LEVELS);
  if (!(s >= FLT_MIN)) {
    s = fabsf(mn) / static_cast<float>(LEVELS);
    if (!(s >= FLT_MIN)) s = 1.0f;
  }
  s16 = round_f16(s);
  if (!(s16 > 0.0f)) s16 = 5.9604644775390625e-08f;  // smallest positive FP16
  if (s16 > 65504.0f) s16 = 65504.0f;
  float zf = rintf(-mn / s16);
  zf = fminf(fmaxf(zf, -65504.0f), 65504.0f);
  z16 = round_f16(zf);
  const float rc = __builtin_amdgcn_rcpf(s16);
  inv = fmaf(fmaf(-rc, s16, 1.0f), rc, rc);
}

// group_qparams_f16 with both quotients from a hardware reciprocal refined
// by one residual step (as row_qparams): the same s16, z16 and inv except
// where a quotient's IEEE rounding differs in its last bit and that bit
// moves the FP16 rounding of s or the integer rounding of -min / s (fp32
// values within one ulp of such a boundary). The unrefined z quotient is
// clamped first so that the residual step stays finite.
template <int LEVELS = 255>
__device__ __forceinline__ void group_qparams_f16_rcp(float mn, float mx, float& s16, float& z16,
                                                      float& inv) {
  constexpr float kL = static_cast<float>(LEVELS), kInvL = 1.0f / static_cast<float>(LEVELS);
  mn = fminf(mn, dpp_mov<0xb1>(mn));
  mx = fmaxf(mx, dpp_mov<0xb1>(mx));
  const float r = mx - mn;
  float s = r * kInvL;
  s = fmaf(fmaf(-s, kL, r), kInvL, s);
  if (__builtin_expect(__builtin_amdgcn_ballot_w64(!(s >= FLT_MIN)) != 0, 0)) {
    if (!(s >= FLT_MIN)) {  // as row_qparams: only in a wave that has such a group
      const float a = fabsf(mn);
      s = a * kInvL;
      s = fmaf(fmaf(-s, kL, a), kInvL, s);
      if (!(s >= FLT_MIN)) s = 1.0f;
    }
  }
  s16 = round_f16(s);
  if (!(s16 > 0.0f)) s16 = 5.9604644775390625e-08f;  // smallest positive FP16
  if (s16 > 65504.0f) s16 = 65504.0f;
  const float rc = __builtin_amdgcn_rcpf(s16);
  inv = fmaf(fmaf(-rc, s16, 1.0f), rc, rc);
  const float nm = -mn;
  const float z0 = __builtin_amdgcn_fmed3f(nm * inv, -65536.0f, 65536.0f);
  float zf = rintf(fmaf(fmaf(-z0, s16, nm), inv, z0));
  zf = fminf(fmaxf(zf, -65504.0f), 65504.0f);
  z16 = round_f16(zf);
}

// ------------------------------------------ small floating-point codes

// The gfx950 conversions between fp32 and OCP E4M3 (bias 7, largest finite
// 448) and E2M1 (magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6; sign in bit 3): they
// round to nearest even and saturate at the largest finite value, as the
// formats' definitions (a scale of 1 leaves the E2M1 values unscaled).
// Two fp32 values into bytes 2 HI, 2 HI + 1 of `old`.
template <bool HI>
__device__ __forceinline__ uint32_t cvt_e4m3x2(float a, float b, uint32_t old) {
  return static_cast<uint32_t>(__builtin_amdgcn_cvt_pk_fp8_f32(a, b, static_cast<int>(old), HI));
}
template <int BYTE>
__device__ __forceinline__ float e4m3_byte(uint32_t w) {
  return __builtin_amdgcn_cvt_f32_fp8(static_cast<int>(w), BYTE);
}
// Two fp32 values into the nibbles of byte BYTE of `old` (a in the low one).
template <int BYTE>
__device__ __forceinline__ uint32_t cvt_e2m1x2(float a, float b, uint32_t old) {
  return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, 1.0f, BYTE);
}
template <int BYTE>
__device__ __forceinline__ void e2m1_byte(uint32_t w, float& lo, float& hi) {
  const auto v = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, BYTE);
  lo = v[0];
  hi = v[1];
}

// 1 / s from the hardware reciprocal refined by one residual step.
__device__ __forceinline__ float refined_rcp(float s) {
  const float rc = __builtin_amdgcn_rcpf(s);
  return fmaf(fmaf(-rc, s, 1.0f), rc, rc);
}

// NVFP4 global scale of a tile's low tier from its largest magnitude.
__device__ __forceinline__ float nvfp4_global(float amax) {
  return amax > 0.0f ? amax / 2688.0f : 1.0f;  // 2688 = 6 * 448
}

// Where an E2M1 tile keeps its global scale: after the metadata of its low
// rows (byte-wise, as the offset may be only 2-aligned).
template <int D>
__device__ __forceinline__ float load_global_scale(const uint8_t* meta_bytes, int k_hi) {
  const uint8_t* p = meta_bytes + static_cast<size_t>(D - k_hi) * (D / 16);
  return __uint_as_float(static_cast<uint32_t>(p[0]) | (static_cast<uint32_t>(p[1]) << 8) |
                         (static_cast<uint32_t>(p[2]) << 16) | (static_cast<uint32_t>(p[3]) << 24));
}
template <int D>
__device__ __forceinline__ void store_global_scale(uint8_t* meta_bytes, int k_hi, float s_g) {
  uint8_t* p = meta_bytes + static_cast<size_t>(D - k_hi) * (D / 16);
  const uint32_t w = __float_as_uint(s_g);
  p[0] = static_cast<uint8_t>(w);
  p[1] = static_cast<uint8_t>(w >> 8);
  p[2] = static_cast<uint8_t>(w >> 16);
  p[3] = static_cast<uint8_t>(w >> 24);
}

// Largest value of v over the workgroup (every thread receives it). Called
// by all threads of the workgroup.
template <int NT>
__device__ __forceinline__ float block_max(float v) {
  __shared__ float part[NT / 64];
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = v;
  __syncthreads();
  float r = part[0];
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) r = fmaxf(r, part[i]);
  __syncthreads();
  return r;
}

// One lane's slice (16 values = half a group of 32, or one NVFP4 block) of a
// low row encoded in the table formats. `codes` and `meta_bytes` point at the
// row's codes and metadata.
template <int KIND, int D>
__device__ __forceinline__ void encode_slice_table(const float* x, int cg, int col0, bool had,
                                                   float s_g, uint8_t* codes, uint8_t* meta) {
  if constexpr (KIND == kInt4) {
    float y[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) y[j] = x[j];
    if (had) {
      fwht32_pair(y, (cg & 1) != 0);
#pragma unroll
      for (int j = 0; j < 16; ++j) y[j] *= kInvSqrt32;
    }
    float mn = y[0], mx = y[0];
#pragma unroll
    for (int j = 1; j < 16; ++j) {
      mn = fminf(mn, y[j]);
      mx = fmaxf(mx, y[j]);
    }
    float s16, z16, inv;
    group_qparams_f16<15>(mn, mx, s16, z16, inv);
    uint32_t w[2] = {0u, 0u};
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float c = __builtin_amdgcn_fmed3f(rintf(fmaf(y[j], inv, z16)), 0.0f, 15.0f);
      w[j >> 3] |= static_cast<uint32_t>(c) << (4 * (j & 7));
    }
    store_words<8>(codes + col0 / 2, w);
    if ((cg & 1) == 0) reinterpret_cast<uint32_t*>(meta)[col0 >> 5] = pack_f16x2(s16, z16);
  } else if constexpr (KIND == kFp8) {
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) amax = fmaxf(amax, fabsf(x[j]));
    amax = fmaxf(amax, dpp_mov<0xb1>(amax));  // the lane pair holds the group
    const float s = __fdiv_rn(amax > 1e-10f ? amax : 1e-10f, 448.0f);
    const float inv = refined_rcp(s);
    uint32_t w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t lo = cvt_e4m3x2<false>(x[4 * k] * inv, x[4 * k + 1] * inv, 0u);
      w[k] = cvt_e4m3x2<true>(x[4 * k + 2] * inv, x[4 * k + 3] * inv, lo);
    }
    store_words<16>(codes + col0, w);
    if ((cg & 1) == 0) reinterpret_cast<float*>(meta)[col0 >> 5] = s;
  } else {
    static_assert(KIND == kNvfp4, "table formats only");
    float amax = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) amax = fmaxf(amax, fabsf(x[j]));
    const float t = fminf(__fdiv_rn(amax, 6.0f * s_g), 448.0f);
    const uint32_t sb = cvt_e4m3x2<false>(t, 0.0f, 0u) & 0xffu;
    const float scale = e4m3_byte<0>(sb) * s_g;
    uint32_t w[2] = {0u, 0u};
    if (scale > 0.0f) {
      const float inv = refined_rcp(scale);
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        uint32_t v = cvt_e2m1x2<0>(x[8 * k] * inv, x[8 * k + 1] * inv, 0u);
        v = cvt_e2m1x2<1>(x[8 * k + 2] * inv, x[8 * k + 3] * inv, v);
        v = cvt_e2m1x2<2>(x[8 * k + 4] * inv, x[8 * k + 5] * inv, v);
        w[k] = cvt_e2m1x2<3>(x[8 * k + 6] * inv, x[8 * k + 7] * inv, v);
      }
    }
    store_words<8>(codes + col0 / 2, w);
    meta[cg] = static_cast<uint8_t>(sb);
  }
}

// The inverse: one lane's 16 decoded values of a low row (before the inverse
// transform of INT4 with had, which the caller applies with fwht32_pair).
// For INT4 the values are s (c - z) scaled by `a` (the caller's decay and the
// transform's normalization), as one FMA each.
template <int KIND, int D>
__device__ __forceinline__ void decode_slice_table(const uint8_t* codes, const uint8_t* meta,
                                                   int cg, int col0, float s_g, float a,
                                                   float* x) {
  if constexpr (KIND == kInt4) {
    uint32_t w[2];
    load_words<8>(codes + col0 / 2, w);
    const uint32_t m = reinterpret_cast<const uint32_t*>(meta)[col0 >> 5];
    const float A = a * f16_lo(m);
    const float B0 = -A * f16_hi(m);
#pragma unroll
    for (int j = 0; j < 16; ++j)
      x[j] = fmaf(A, static_cast<float>((w[j >> 3] >> (4 * (j & 7))) & 0xfu), B0);
  } else if constexpr (KIND == kFp8) {
    uint32_t w[4];
    load_words<16>(codes + col0, w);
    const float s = reinterpret_cast<const float*>(meta)[col0 >> 5];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[4 * k + 0] = a * (s * e4m3_byte<0>(w[k]));
      x[4 * k + 1] = a * (s * e4m3_byte<1>(w[k]));
      x[4 * k + 2] = a * (s * e4m3_byte<2>(w[k]));
      x[4 * k + 3] = a * (s * e4m3_byte<3>(w[k]));
    }
  } else {
    static_assert(KIND == kNvfp4, "table formats only");
    uint32_t w[2];
    load_words<8>(codes + col0 / 2, w);
    const float scale = e4m3_byte<0>(meta[cg]) * s_g;
    float q[16];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      e2m1_byte<0>(w[k], q[8 * k + 0], q[8 * k + 1]);
      e2m1_byte<1>(w[k], q[8 * k + 2], q[8 * k + 3]);
      e2m1_byte<2>(w[k], q[8 * k + 4], q[8 * k + 5]);
      e2m1_byte<3>(w[k], q[8 * k + 6], q[8 * k + 7]);
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) x[j] = a * (q[j] * scale);
  }
}

// ------------------------------------------------------------- row encode

// Stores one row slice of CPT values (columns col0..col0+CPT of tile row r)
// in its tier. Lanes cg = 0..TPR-1 of a row group hold the slices of one
// row; the (s, z) pair of a low-tier row is written by lane cg == 0. The
// branch on r is uniform across the TPR lanes of the row.
template <int KIND, int D, int CPT, int TPR>
__device__ __forceinline__ void encode_row(const float* x, int r, int k_hi, int cg, int col0,
                                           uint8_t* tile, uint8_t* codes, uint8_t* meta_bytes,
                                           bool had = false, float s_g = 1.0f) {
  if constexpr (KIND >= kInt4) {
    static_assert(CPT == 16, "a lane holds 16 values of a row");
    if (r < k_hi) {
      uint32_t w[CPT / 2];
#pragma unroll
      for (int j = 0; j < CPT / 2; ++j) w[j] = pack_f16x2(x[2 * j], x[2 * j + 1]);
      store_words<CPT * 2>(tile + (static_cast<size_t>(r) * D + col0) * 2, w);
      return;
    }
    const size_t l = static_cast<size_t>(r - k_hi);
    encode_slice_table<KIND, D>(x, cg, col0, had, s_g, codes + l * code_row_bytes<KIND, D>(),
                                meta_bytes + l * meta_row_bytes<KIND, D>());
    return;
  } else if constexpr (KIND == kPaper) {
    static_assert(CPT == 16, "a lane pair holds one group of 32");
    if (r < k_hi) {
      uint32_t w[CPT / 2];
#pragma unroll
      for (int j = 0; j < CPT / 2; ++j) w[j] = pack_f16x2(x[2 * j], x[2 * j + 1]);
      store_words<CPT * 2>(tile + (static_cast<size_t>(r) * D + col0) * 2, w);
      return;
    }
    float y[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) y[j] = x[j];
    if (had) {
      fwht32_pair(y, (cg & 1) != 0);
#pragma unroll
      for (int j = 0; j < 16; ++j) y[j] *= kInvSqrt32;
    }
    float mn = y[0], mx = y[0];
#pragma unroll
    for (int j = 1; j < 16; ++j) {
      mn = fminf(mn, y[j]);
      mx = fmaxf(mx, y[j]);
    }
    float s16, z16, inv;
    group_qparams_f16(mn, mx, s16, z16, inv);
    uint32_t w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint32_t c = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(y[4 * j], inv, z16), 0, 0u);
      c = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(y[4 * j + 1], inv, z16), 1, c);
      c = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(y[4 * j + 2], inv, z16), 2, c);
      w[j] = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(y[4 * j + 3], inv, z16), 3, c);
    }
    const int l = r - k_hi;
    store_words<16>(codes + static_cast<size_t>(l) * D + col0, w);
    if ((cg & 1) == 0)
      reinterpret_cast<uint32_t*>(meta_bytes)[static_cast<size_t>(l) * (D / 32) + (col0 >> 5)] =
          pack_f16x2(s16, z16);
    return;
  }
  float2* meta = reinterpret_cast<float2*>(meta_bytes);
  if (KIND == kFp32) {
    uint32_t w[CPT];
#pragma unroll
    for (int j = 0; j < CPT; ++j) w[j] = __float_as_uint(x[j]);
    store_words<CPT * 4>(tile + (static_cast<size_t>(r) * D + col0) * 4, w);
  } else if (r < k_hi) {
    uint32_t w[CPT / 2];
#pragma unroll
    for (int j = 0; j < CPT / 2; ++j) w[j] = pack_bf16x2(x[2 * j], x[2 * j + 1]);
    store_words<CPT * 2>(tile + (static_cast<size_t>(r) * D + col0) * 2, w);
  } else {
    float mn = x[0], mx = x[0];
#pragma unroll
    for (int j = 1; j < CPT; ++j) {
      mn = fminf(mn, x[j]);
      mx = fmaxf(mx, x[j]);
    }
    group_minmax<TPR>(mn, mx);
    float s, z, inv;
    row_qparams(mn, mx, s, z, inv);
    uint32_t w[CPT / 4];
#pragma unroll
    for (int j = 0; j < CPT / 4; ++j)
      w[j] = pack_codes4(quant_code(x[4 * j], inv, z), quant_code(x[4 * j + 1], inv, z),
                         quant_code(x[4 * j + 2], inv, z), quant_code(x[4 * j + 3], inv, z));
    const int l = r - k_hi;
    store_words<CPT>(codes + static_cast<size_t>(l) * D + col0, w);
    if (cg == 0) meta[l] = make_float2(s, z);
  }
}

// ------------------------------------------------------------- row decode

// Loads and decodes one row slice (columns col0 .. col0 + CPT of tile row r)
// into fp32: the high tier widened, the low tier as s * (c - z) (then the
// inverse transform for the paper tiers with had). Lanes of a row take the
// same branch (r is uniform across them).
template <int KIND, int D, int CPT>
__device__ __forceinline__ void decode_row(const uint8_t* tile, const uint8_t* codes,
                                           const uint8_t* meta_bytes, int r, int k_hi, int cg,
                                           int col0, bool had, float* x) {
  if (KIND == kFp32) {
    uint32_t w[CPT];
    load_words<CPT * 4>(tile + (static_cast<size_t>(r) * D + col0) * 4, w);
#pragma unroll
    for (int j = 0; j < CPT; ++j) x[j] = __uint_as_float(w[j]);
    return;
  }
  if (r < k_hi) {
    uint32_t w[CPT / 2];
    load_words<CPT * 2>(tile + (static_cast<size_t>(r) * D + col0) * 2, w);
#pragma unroll
    for (int j = 0; j < CPT / 2; ++j) {
      x[2 * j] = KIND >= kPaper ? f16_lo(w[j]) : bf16_lo(w[j]);
      x[2 * j + 1] = KIND >= kPaper ? f16_hi(w[j]) : bf16_hi(w[j]);
    }
    return;
  }
  if constexpr (KIND >= kInt4) {
    const size_t lr = static_cast<size_t>(r - k_hi);
    const float s_g = KIND == kNvfp4 ? load_global_scale<D>(meta_bytes, k_hi) : 1.0f;
    decode_slice_table<KIND, D>(codes + lr * code_row_bytes<KIND, D>(),
                                meta_bytes + lr * meta_row_bytes<KIND, D>(), cg, col0, s_g,
                                (KIND == kInt4 && had) ? kInvSqrt32 : 1.0f, x);
    if constexpr (KIND == kInt4) {
      if (had) fwht32_pair(reinterpret_cast<float(&)[16]>(*x), (cg & 1) != 0);
    }
    return;
  } else {
  const int l = r - k_hi;
  uint32_t w[CPT / 4];
  load_words<CPT>(codes + static_cast<size_t>(l) * D + col0, w);
  float s, z;
  if constexpr (KIND == kPaper) {
    const uint32_t m =
        reinterpret_cast<const uint32_t*>(meta_bytes)[static_cast<size_t>(l) * (D / 32) + (col0 >> 5)];
    s = f16_lo(m);
    z = f16_hi(m);
  } else {
    const float2 sz = reinterpret_cast<const float2*>(meta_bytes)[l];
    s = sz.x;
    z = sz.y;
  }
  // s * (c - z) as one FMA per value, with the transform's normalization
  // folded into the factor
  const float A = s * ((KIND == kPaper && had) ? kInvSqrt32 : 1.0f);
  const float B0 = -A * z;
#pragma unroll
  for (int j = 0; j < CPT / 4; ++j) {
    x[4 * j + 0] = fmaf(A, ubyte<0>(w[j]), B0);
    x[4 * j + 1] = fmaf(A, ubyte<1>(w[j]), B0);
    x[4 * j + 2] = fmaf(A, ubyte<2>(w[j]), B0);
    x[4 * j + 3] = fmaf(A, ubyte<3>(w[j]), B0);
  }
  if constexpr (KIND == kPaper && CPT == 16) {
    if (had) fwht32_pair(reinterpret_cast<float(&)[16]>(*x), (cg & 1) != 0);
  }
  }
}

}  // namespace damp
