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
  if (!(q >= FLT_MIN)) {
    const float a = fabsf(mn);
    q = a * k255inv;
    q = fmaf(fmaf(-q, 255.0f, a), k255inv, q);
    if (!(q >= FLT_MIN)) q = 1.0f;
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
__device__ __forceinline__ void group_qparams_f16(float mn, float mx, float& s16, float& z16,
                                                  float& inv) {
  mn = fminf(mn, dpp_mov<0xb1>(mn));
  mx = fmaxf(mx, dpp_mov<0xb1>(mx));
  float s = (mx - mn) / 255.0f;
  if (!(s >= FLT_MIN)) {
    s = fabsf(mn) / 255.0f;
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

// ------------------------------------------------------------- row encode

// Stores one row slice of CPT values (columns col0..col0+CPT of tile row r)
// in its tier. Lanes cg = 0..TPR-1 of a row group hold the slices of one
// row; the (s, z) pair of a low-tier row is written by lane cg == 0. The
// branch on r is uniform across the TPR lanes of the row.
template <int KIND, int D, int CPT, int TPR>
__device__ __forceinline__ void encode_row(const float* x, int r, int k_hi, int cg, int col0,
                                           uint8_t* tile, uint8_t* codes, uint8_t* meta_bytes,
                                           bool had = false) {
  if constexpr (KIND == kPaper) {
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
      x[2 * j] = KIND == kPaper ? f16_lo(w[j]) : bf16_lo(w[j]);
      x[2 * j + 1] = KIND == kPaper ? f16_hi(w[j]) : bf16_hi(w[j]);
    }
    return;
  }
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

}  // namespace damp
