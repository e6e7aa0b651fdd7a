/*
 * damp_oracle.c - plain, slow CPU oracle of DAMP's decode-step state update
 * (arXiv 2608.27513). TEST INFRASTRUCTURE ONLY: it exists so that tests, the
 * smoke check and the benchmark's CPU baseline can check and time the HIP
 * library. It shares no code, header, table or helper with the HIP library
 * and the product path never calls it.
 *
 * Arithmetic precision. The paper's fused executor evaluates the recurrence
 * in FP32 and quantizes the FP32 result before it is stored (section 3.2;
 * App. A.5, "Fused decode executor"), so this oracle computes in fp32, with
 * every sum taken in ascending index order, no contraction into FMA
 * (built with -ffp-contract=off) and libm's expf. Channel selection follows
 * App. A.2 in double on the host. An independent fp64 brute force of the
 * recurrence lives in brute.py and pins this file.
 *
 * Readings taken where the paper is silent:
 *  - round() in Eq. (3) is round-half-to-even (rintf), for z and for codes;
 *    codes saturate to [0, 255] (App. A.1); z is not clamped.
 *  - A row whose scale s is not a normal fp32 number (a constant row) uses
 *    s = |min| / 255, or s = 1 if that is not normal either.
 *  - o is read from the updated FP32 state before it is re-quantized.
 *  - One (s, z) pair per low-tier row (the quantizer group is the whole row),
 *    stored as fp32; the high tier is bf16 with round-to-nearest-even.
 *  - GDN's per-head decay is applied as the same a for every row, so KDA with
 *    a channel-constant g reproduces GDN exactly.
 *  - The paper's own low tier (App. A.1 format table; Eq. (17)) is available
 *    as a storage format: groups of 32 values along d_v with FP16 (s, z),
 *    an optional normalized block-32 Hadamard transform applied before
 *    quantization and again after reconstruction (it is its own inverse),
 *    and an FP16 high tier. s follows Eq. (3) in fp32 and is stored in FP16
 *    (round to nearest even, kept within the positive finite FP16 range);
 *    z = round(-min / s) uses the stored s and is stored in FP16 (within the
 *    finite range); codes use the stored (s, z), so the encoder and the
 *    reconstruction agree.
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_KIND_FP32 0
#define ORC_KIND_MIXED 1

/* Threads the OpenMP loops below use (1 without OpenMP). */
int orc_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ---------------------------------------------------------------- formats */

static float orc_from_bf16(uint16_t h) {
  uint32_t bits = ((uint32_t)h) << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return f;
}

/* fp32 -> bf16 with round-to-nearest, ties to even (finite inputs). */
static uint16_t orc_to_bf16(float f) {
  uint32_t bits;
  memcpy(&bits, &f, sizeof bits);
  if ((bits & 0x7f800000u) == 0x7f800000u) /* inf / nan: truncate, keep quiet */
    return (uint16_t)((bits >> 16) | ((bits & 0xffffu) ? 0x40u : 0u));
  uint32_t lsb = (bits >> 16) & 1u;
  bits += 0x7fffu + lsb;
  return (uint16_t)(bits >> 16);
}

void orc_bf16_round(const float* x, uint16_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_to_bf16(x[i]);
}

void orc_bf16_widen(const uint16_t* x, float* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_from_bf16(x[i]);
}

/* fp32 -> IEEE binary16 bits, round to nearest even (overflow -> inf). The
 * rounding is done on exact double quotients: subnormals count in units of
 * 2^-24, normals carry 11 significant bits. */
static uint16_t orc_to_fp16(float f) {
  uint32_t bits;
  memcpy(&bits, &f, 4);
  uint16_t sign = (uint16_t)((bits >> 16) & 0x8000u);
  double a = fabs((double)f);
  if (a != a) return (uint16_t)(sign | 0x7E00u);           /* NaN */
  if (a >= 65520.0) return (uint16_t)(sign | 0x7C00u);     /* rounds past the largest */
  if (a < 6.103515625e-05) {                               /* below 2^-14: subnormal */
    double m = rint(a * 16777216.0);                        /* units of 2^-24 */
    return (uint16_t)(sign | (uint16_t)m);                  /* 1024 is the first normal */
  }
  int e2;
  frexp(a, &e2);                                            /* a = f 2^e2, f in [0.5, 1) */
  int e = e2 - 1;                                           /* a in [2^e, 2^(e+1)) */
  double m = rint(ldexp(a, 10 - e));                        /* in [1024, 2048] */
  if (m == 2048.0) {
    m = 1024.0;
    e += 1;
  }
  if (e > 15) return (uint16_t)(sign | 0x7C00u);
  return (uint16_t)(sign | (uint16_t)((e + 15) << 10) | (uint16_t)(m - 1024.0));
}

static float orc_from_fp16(uint16_t h) {
  int e = (h >> 10) & 0x1F, m = h & 0x3FF;
  double v;
  if (e == 0) v = ldexp((double)m, -24);
  else if (e == 31) v = m ? NAN : INFINITY;
  else v = ldexp((double)(1024 + m), e - 25);
  return (float)((h & 0x8000u) ? -v : v);
}

void orc_fp16_round(const float* x, uint16_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_to_fp16(x[i]);
}
void orc_fp16_widen(const uint16_t* x, float* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_from_fp16(x[i]);
}

/* Normalized block-32 Hadamard transform (App. A.1): y_i = 32^(-1/2)
 * sum_j (-1)^popcount(i & j) x_j, summed in fp32 in ascending j. The matrix
 * is symmetric and orthogonal, so the same call inverts it. */
void orc_hadamard32(const float* x, float* y) {
  const float norm = 0.17677669529663687f; /* 1 / sqrt(32) */
  for (int i = 0; i < 32; ++i) {
    float acc = 0.0f;
    for (int j = 0; j < 32; ++j) {
      if (__builtin_popcount((unsigned)(i & j)) & 1) acc = acc - x[j];
      else acc = acc + x[j];
    }
    y[i] = acc * norm;
  }
}

/* ------------------------------------------------- Eq. (3): one-row INT8 */

/* Scale and zero point of n values with 2^b - 1 = `levels` steps (Eq. (3)). */
static void orc_quant_params_levels(const float* x, int n, float levels, float* s_out,
                                    float* z_out) {
  float lo = x[0], hi = x[0];
  for (int j = 1; j < n; ++j) {
    if (x[j] < lo) lo = x[j];
    if (x[j] > hi) hi = x[j];
  }
  float s = (hi - lo) / levels;
  if (!(s >= FLT_MIN)) {           /* constant row */
    s = fabsf(lo) / levels;
    if (!(s >= FLT_MIN)) s = 1.0f; /* zero row */
  }
  *s_out = s;
  *z_out = rintf(-lo / s);
}

/* Scale and zero point of a row (Eq. (3) with b = 8). */
void orc_quant_params(const float* x, int n, float* s_out, float* z_out) {
  orc_quant_params_levels(x, n, 255.0f, s_out, z_out);
}

/* One code: round(x / s) + z, saturated to [0, levels]. */
static uint8_t orc_code_levels(float x, float s, float z, float levels) {
  float c = rintf(x / s) + z;
  if (c < 0.0f) c = 0.0f;
  if (c > levels) c = levels;
  return (uint8_t)c;
}

/* One code: round(x / s) + z, saturated to the unsigned 8-bit range. */
static uint8_t orc_code(float x, float s, float z) { return orc_code_levels(x, s, z, 255.0f); }

/* Reconstruction Q(x) = s * (c - z). */
static float orc_decode(uint8_t c, float s, float z) { return s * ((float)c - z); }

void orc_quant_row(const float* x, int n, uint8_t* codes, float* s, float* z) {
  orc_quant_params(x, n, s, z);
  for (int j = 0; j < n; ++j) codes[j] = orc_code(x[j], *s, *z);
}

void orc_dequant_row(const uint8_t* codes, int n, float s, float z, float* out) {
  for (int j = 0; j < n; ++j) out[j] = orc_decode(codes[j], s, z);
}

/* One group with FP16 metadata (App. A.1, integer formats): s from Eq. (3) in
 * fp32, stored in FP16; z from the stored s, stored in FP16; codes from the
 * stored pair. s and z are returned widened to fp32. */
static void orc_quant_group_fp16_levels(const float* x, int n, float levels, uint8_t* codes,
                                        float* s_out, float* z_out) {
  float s, z;
  orc_quant_params_levels(x, n, levels, &s, &z);
  float lo = x[0];
  for (int j = 1; j < n; ++j)
    if (x[j] < lo) lo = x[j];
  float s16 = orc_from_fp16(orc_to_fp16(s));
  if (!(s16 > 0.0f)) s16 = orc_from_fp16(0x0001u);   /* smallest positive FP16 */
  if (s16 > 65504.0f) s16 = 65504.0f;
  float zf = rintf(-lo / s16);
  if (zf > 65504.0f) zf = 65504.0f;
  if (zf < -65504.0f) zf = -65504.0f;
  float z16 = orc_from_fp16(orc_to_fp16(zf));
  for (int j = 0; j < n; ++j) codes[j] = orc_code_levels(x[j], s16, z16, levels);
  *s_out = s16;
  *z_out = z16;
}

void orc_quant_group_fp16(const float* x, int n, uint8_t* codes, float* s_out, float* z_out) {
  orc_quant_group_fp16_levels(x, n, 255.0f, codes, s_out, z_out);
}

/* INT4 of App. A.1: as above with 15 steps, codes in [0, 15]. */
void orc_quant_group_fp16_u4(const float* x, int n, uint8_t* codes, float* s_out, float* z_out) {
  orc_quant_group_fp16_levels(x, n, 15.0f, codes, s_out, z_out);
}

/* ------------------------------------------- small floating-point codes */

/* OCP E4M3 (FN variant: bias 7, no infinities, largest finite 448), round to
 * nearest even, saturating at +-448. Exact arithmetic in double. */
uint8_t orc_to_e4m3(float f) {
  uint8_t sign = signbit(f) ? 0x80 : 0x00;
  double a = fabs((double)f);
  if (a != a) return 0x7F;                         /* NaN */
  if (a < 0.015625) {                              /* below 2^-6: steps of 2^-9 */
    double m = rint(a * 512.0);                    /* 8 is the first normal */
    return (uint8_t)(sign | (uint8_t)m);
  }
  int e2;
  frexp(a, &e2);
  int e = e2 - 1;                                  /* a in [2^e, 2^(e+1)) */
  double m = rint(ldexp(a, 3 - e));                /* in [8, 16] */
  if (m == 16.0) {
    m = 8.0;
    e += 1;
  }
  if (e > 8 || (e == 8 && m > 14.0)) return (uint8_t)(sign | 0x7E);  /* saturate at 448 */
  return (uint8_t)(sign | (uint8_t)((e + 7) << 3) | (uint8_t)(m - 8.0));
}

float orc_from_e4m3(uint8_t c) {
  int e = (c >> 3) & 15, m = c & 7;
  double v = e == 0 ? ldexp((double)m, -9) : ldexp((double)(8 + m), e - 10);
  if ((c & 0x7F) == 0x7F) v = NAN;
  return (float)((c & 0x80) ? -v : v);
}

/* E2M1 (bias 1; magnitudes 0, 0.5, 1, 1.5, 2, 3, 4, 6), round to nearest
 * even, saturating at +-6; bit 3 is the sign. */
uint8_t orc_to_e2m1(float f) {
  uint8_t sign = signbit(f) ? 0x8 : 0x0;
  double a = fabs((double)f);
  if (a >= 6.0) return (uint8_t)(sign | 0x7);
  if (a < 1.0) return (uint8_t)(sign | (uint8_t)rint(a * 2.0));  /* 2 is the first normal */
  int e2;
  frexp(a, &e2);
  int e = e2 - 1;                                  /* a in [2^e, 2^(e+1)), e in 0..2 */
  double m = rint(ldexp(a, 1 - e));                /* in [2, 4] */
  if (m == 4.0) {
    m = 2.0;
    e += 1;
  }
  if (e > 2) return (uint8_t)(sign | 0x7);
  return (uint8_t)(sign | (uint8_t)((e + 1) << 1) | (uint8_t)(m - 2.0));
}

float orc_from_e2m1(uint8_t c) {
  int e = (c >> 1) & 3, m = c & 1;
  double v = e == 0 ? 0.5 * m : ldexp(1.0 + 0.5 * m, e - 1);
  return (float)((c & 0x8) ? -v : v);
}

void orc_e4m3_round(const float* x, uint8_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_to_e4m3(x[i]);
}
void orc_e4m3_widen(const uint8_t* c, float* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_from_e4m3(c[i]);
}
void orc_e2m1_round(const float* x, uint8_t* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_to_e2m1(x[i]);
}
void orc_e2m1_widen(const uint8_t* c, float* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_from_e2m1(c[i]);
}

/* FP8 of App. A.1 (Eq. (16)): one fp32 scale per group, no zero point:
 * s = max(max|x|, 1e-10) / 448, q = E4M3(clip(x / s, -448, 448)). */
void orc_quant_group_e4m3(const float* x, int n, uint8_t* codes, float* s_out) {
  float amax = 0.0f;
  for (int j = 0; j < n; ++j)
    if (fabsf(x[j]) > amax) amax = fabsf(x[j]);
  float s = (amax > 1e-10f ? amax : 1e-10f) / 448.0f;
  for (int j = 0; j < n; ++j) {
    float y = x[j] / s;
    if (y > 448.0f) y = 448.0f;
    if (y < -448.0f) y = -448.0f;
    codes[j] = orc_to_e4m3(y);
  }
  *s_out = s;
}

/* NVFP4 of App. A.1: the global scale of a tile's low tier from its largest
 * magnitude, s_g = amax / (6 * 448) (1 if amax is 0). */
float orc_nvfp4_global(float amax) {
  return amax > 0.0f ? amax / 2688.0f : 1.0f;
}

/* One NVFP4 block: E4M3 block scale s_b = E4M3(max|x| / (6 s_g)); codes
 * E2M1(x / (s_b s_g)) (all 0 if s_b is 0). Returns the block-scale code. */
uint8_t orc_quant_block_e2m1(const float* x, int n, float s_g, uint8_t* codes) {
  float amax = 0.0f;
  for (int j = 0; j < n; ++j)
    if (fabsf(x[j]) > amax) amax = fabsf(x[j]);
  float t = amax / (6.0f * s_g);
  if (t > 448.0f) t = 448.0f;
  uint8_t sb = orc_to_e4m3(t);
  float scale = orc_from_e4m3(sb) * s_g;
  for (int j = 0; j < n; ++j) codes[j] = scale > 0.0f ? orc_to_e2m1(x[j] / scale) : 0;
  return sb;
}

/* ------------------------------------------------------- layout (Eq. 17) */

/* Storage format: fmt[0] high-tier type (1 BF16, 2 FP16), fmt[1] values per
 * metadata group along d_v, fmt[2] metadata type (0 FP32, 2 FP16), fmt[3] 1
 * for the block-32 Hadamard transform of the low tier, fmt[4] code type (3
 * UINT8, 4 UINT4, 5 E4M3, 6 E2M1; the App. A.1 format table). NULL: BF16,
 * one UINT8 (s, z) pair per row in FP32, no transform. */
enum { ORC_CODE_U8 = 3, ORC_CODE_U4 = 4, ORC_CODE_E4M3 = 5, ORC_CODE_E2M1 = 6 };
typedef struct {
  int hi_fp16, group, meta_fp16, hadamard, code;
} orc_fmt_t;

static orc_fmt_t orc_fmt(const int32_t* f, int dv) {
  orc_fmt_t r = {0, dv, 0, 0, ORC_CODE_U8};
  if (f) {
    r.hi_fp16 = f[0] == 2;
    r.group = f[1];
    r.meta_fp16 = f[2] == 2;
    r.hadamard = f[3] != 0;
    r.code = f[4];
  }
  return r;
}

static int orc_code_is_nibble(orc_fmt_t f) {
  return f.code == ORC_CODE_U4 || f.code == ORC_CODE_E2M1;
}

/* Bytes per low row: codes (two per byte for 4-bit codes, the even column in
 * the low nibble) and metadata: (s, z) per group for the integer codes, an
 * fp32 s per group for E4M3, an E4M3 block scale per group for E2M1. */
static int64_t orc_code_row_bytes(orc_fmt_t f, int dv) {
  return orc_code_is_nibble(f) ? dv / 2 : dv;
}
static int64_t orc_meta_row_bytes(orc_fmt_t f, int dv) {
  const int64_t groups = dv / f.group;
  if (f.code == ORC_CODE_E4M3) return groups * 4;
  if (f.code == ORC_CODE_E2M1) return groups;
  return groups * 2 * (f.meta_fp16 ? 2 : 4);
}
/* E2M1 tiles end with the fp32 global scale of their low tier. */
static int64_t orc_tile_tail_bytes(orc_fmt_t f) { return f.code == ORC_CODE_E2M1 ? 4 : 0; }

/* Bytes of one tile: high tier, codes, the metadata of each low row group by
 * group, then (E2M1) the global scale. */
int64_t orc_tile_bytes(int kind, const int32_t* fmt, int dk, int dv, int k_hi) {
  if (kind == ORC_KIND_FP32) return (int64_t)dk * dv * 4;
  orc_fmt_t f = orc_fmt(fmt, dv);
  return (int64_t)k_hi * dv * 2 + (int64_t)(dk - k_hi) * orc_code_row_bytes(f, dv) +
         (int64_t)(dk - k_hi) * orc_meta_row_bytes(f, dv) + orc_tile_tail_bytes(f);
}

/* Storage bits per value of a mixed layout, general form of Eq. (7): the low
 * tier costs its code bits plus two metadata words per `group` values. */
double orc_bits_per_value(int dk, int k_hi, int hi_bits, int code_bits, int group,
                          int meta_bits) {
  double b_lo = (double)code_bits + 2.0 * (double)meta_bits / (double)group;
  double b_hi = (double)hi_bits;
  return b_lo + ((double)k_hi / (double)dk) * (b_hi - b_lo);
}

/* Codes of one low row as one byte per value. */
static void orc_codes_unpack(orc_fmt_t f, const uint8_t* row, int dv, uint8_t* c) {
  if (!orc_code_is_nibble(f)) {
    memcpy(c, row, (size_t)dv);
    return;
  }
  for (int j = 0; j < dv; j += 2) {
    c[j] = row[j / 2] & 0xF;
    c[j + 1] = row[j / 2] >> 4;
  }
}
static void orc_codes_pack(orc_fmt_t f, const uint8_t* c, int dv, uint8_t* row) {
  if (!orc_code_is_nibble(f)) {
    memcpy(row, c, (size_t)dv);
    return;
  }
  for (int j = 0; j < dv; j += 2) row[j / 2] = (uint8_t)((c[j] & 0xF) | (c[j + 1] << 4));
}

/* Decode tile rows (in tile order) into S[dk][dv]. */
static void orc_tile_decode(int kind, orc_fmt_t f, int dk, int dv, int k_hi,
                            const uint8_t* tile, float* S) {
  if (kind == ORC_KIND_FP32) {
    memcpy(S, tile, (size_t)dk * dv * sizeof(float));
    return;
  }
  const uint8_t* hi = tile;
  const uint8_t* codes = tile + (size_t)k_hi * dv * 2;
  const uint8_t* meta = codes + (size_t)(dk - k_hi) * orc_code_row_bytes(f, dv);
  const int64_t mrow = orc_meta_row_bytes(f, dv);
  float s_g = 1.0f;
  if (f.code == ORC_CODE_E2M1) memcpy(&s_g, meta + (size_t)(dk - k_hi) * mrow, 4);
  uint8_t crow[4096];
  for (int r = 0; r < dk; ++r) {
    float* x = S + (size_t)r * dv;
    if (r < k_hi) {
      for (int j = 0; j < dv; ++j) {
        uint16_t h;
        memcpy(&h, hi + ((size_t)r * dv + j) * 2, 2);
        x[j] = f.hi_fp16 ? orc_from_fp16(h) : orc_from_bf16(h);
      }
      continue;
    }
    int l = r - k_hi;
    orc_codes_unpack(f, codes + (size_t)l * orc_code_row_bytes(f, dv), dv, crow);
    for (int g = 0; g < dv / f.group; ++g) {
      float sz[2];
      const uint8_t* m = meta + (size_t)l * mrow;
      float* xg = x + (size_t)g * f.group;
      const uint8_t* cg = crow + (size_t)g * f.group;
      if (f.code == ORC_CODE_E4M3) {            /* x = s q */
        float sc;
        memcpy(&sc, m + (size_t)g * 4, 4);
        for (int j = 0; j < f.group; ++j) xg[j] = sc * orc_from_e4m3(cg[j]);
        continue;
      }
      if (f.code == ORC_CODE_E2M1) {            /* x = q (s_b s_g) */
        const float scale = orc_from_e4m3(m[g]) * s_g;
        for (int j = 0; j < f.group; ++j) xg[j] = orc_from_e2m1(cg[j]) * scale;
        continue;
      }
      if (f.meta_fp16) {
        uint16_t h[2];
        memcpy(h, m + (size_t)g * 4, 4);
        sz[0] = orc_from_fp16(h[0]);
        sz[1] = orc_from_fp16(h[1]);
      } else {
        memcpy(sz, m + (size_t)g * 8, 8);
      }
      orc_dequant_row(cg, f.group, sz[0], sz[1], xg);
      if (f.hadamard) {
        float y[32];
        orc_hadamard32(xg, y);
        memcpy(xg, y, sizeof y);
      }
    }
  }
}

/* Encode S[dk][dv] (tile order) into the tile. */
static void orc_tile_encode(int kind, orc_fmt_t f, int dk, int dv, int k_hi, const float* S,
                            uint8_t* tile) {
  if (kind == ORC_KIND_FP32) {
    memcpy(tile, S, (size_t)dk * dv * sizeof(float));
    return;
  }
  uint8_t* hi = tile;
  uint8_t* codes = tile + (size_t)k_hi * dv * 2;
  uint8_t* meta = codes + (size_t)(dk - k_hi) * orc_code_row_bytes(f, dv);
  const int64_t mrow = orc_meta_row_bytes(f, dv);
  float s_g = 1.0f;
  if (f.code == ORC_CODE_E2M1) {  /* the global scale of the low tier */
    float amax = 0.0f;
    for (int64_t i = (int64_t)k_hi * dv; i < (int64_t)dk * dv; ++i)
      if (fabsf(S[i]) > amax) amax = fabsf(S[i]);
    s_g = orc_nvfp4_global(amax);
    memcpy(meta + (size_t)(dk - k_hi) * mrow, &s_g, 4);
  }
  uint8_t crow[4096];
  for (int r = 0; r < dk; ++r) {
    const float* x = S + (size_t)r * dv;
    if (r < k_hi) {
      for (int j = 0; j < dv; ++j) {
        uint16_t h = f.hi_fp16 ? orc_to_fp16(x[j]) : orc_to_bf16(x[j]);
        memcpy(hi + ((size_t)r * dv + j) * 2, &h, 2);
      }
      continue;
    }
    int l = r - k_hi;
    for (int g = 0; g < dv / f.group; ++g) {
      const float* xg = x + (size_t)g * f.group;
      float y[32];
      if (f.hadamard) {
        orc_hadamard32(xg, y);
        xg = y;
      }
      uint8_t* c = crow + (size_t)g * f.group;
      uint8_t* m = meta + (size_t)l * mrow;
      float sz[2];
      if (f.code == ORC_CODE_E4M3) {
        orc_quant_group_e4m3(xg, f.group, c, &sz[0]);
        memcpy(m + (size_t)g * 4, &sz[0], 4);
      } else if (f.code == ORC_CODE_E2M1) {
        m[g] = orc_quant_block_e2m1(xg, f.group, s_g, c);
      } else if (f.code == ORC_CODE_U4) {
        orc_quant_group_fp16_u4(xg, f.group, c, &sz[0], &sz[1]);
        uint16_t h[2] = {orc_to_fp16(sz[0]), orc_to_fp16(sz[1])};
        memcpy(m + (size_t)g * 4, h, 4);
      } else if (f.meta_fp16) {
        orc_quant_group_fp16(xg, f.group, c, &sz[0], &sz[1]);
        uint16_t h[2] = {orc_to_fp16(sz[0]), orc_to_fp16(sz[1])};
        memcpy(m + (size_t)g * 4, h, 4);
      } else {
        orc_quant_row(xg, f.group, c, &sz[0], &sz[1]);
        memcpy(m + (size_t)g * 8, sz, 8);
      }
    }
    orc_codes_pack(f, crow, dv, codes + (size_t)l * orc_code_row_bytes(f, dv));
  }
}

static int orc_perm_at(const uint8_t* perm, int h, int dk, int r) {
  return perm ? (int)perm[(size_t)h * dk + r] : r;
}

/* ---------------------------------------------------------- pack / unpack */

/* Pool addressing: tile of (slot, head) at pool + slot*slot_stride +
 * head*tile_stride (pool already offset to the layer). */
void orc_pack(int kind, const int32_t* fmt, int dk, int dv, int k_hi, uint8_t* pool,
              int64_t slot_stride, int64_t tile_stride, int num_slots, const int32_t* slot_idx,
              int B, int HV, const float* S, const uint8_t* perm) {
  const orc_fmt_t f = orc_fmt(fmt, dv);
  int64_t ntiles = (int64_t)B * HV;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < ntiles; ++t) {
    int b = (int)(t / HV), h = (int)(t % HV);
    int slot = slot_idx[b];
    if (slot < 0 || slot >= num_slots) continue;
    float* W = (float*)malloc((size_t)dk * dv * sizeof(float));
    const float* src = S + (size_t)t * dk * dv;
    for (int r = 0; r < dk; ++r)
      memcpy(W + (size_t)r * dv, src + (size_t)orc_perm_at(perm, h, dk, r) * dv,
             (size_t)dv * sizeof(float));
    orc_tile_encode(kind, f, dk, dv, k_hi, W,
                    pool + (size_t)slot * slot_stride + (size_t)h * tile_stride);
    free(W);
  }
}

void orc_unpack(int kind, const int32_t* fmt, int dk, int dv, int k_hi, const uint8_t* pool,
                int64_t slot_stride, int64_t tile_stride, int num_slots,
                const int32_t* slot_idx, int B, int HV, const uint8_t* perm, float* S) {
  const orc_fmt_t f = orc_fmt(fmt, dv);
  int64_t ntiles = (int64_t)B * HV;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < ntiles; ++t) {
    int b = (int)(t / HV), h = (int)(t % HV);
    int slot = slot_idx[b];
    float* dst = S + (size_t)t * dk * dv;
    if (slot < 0 || slot >= num_slots) {
      memset(dst, 0, (size_t)dk * dv * sizeof(float));
      continue;
    }
    float* W = (float*)malloc((size_t)dk * dv * sizeof(float));
    orc_tile_decode(kind, f, dk, dv, k_hi,
                    pool + (size_t)slot * slot_stride + (size_t)h * tile_stride, W);
    for (int r = 0; r < dk; ++r)
      memcpy(dst + (size_t)orc_perm_at(perm, h, dk, r) * dv, W + (size_t)r * dv,
             (size_t)dv * sizeof(float));
    free(W);
  }
}

/* ------------------------------------------------- decode-step update */

/*
 * One token of Eq. (1) on an fp32 state S[dk][dv] in tile-row order (row r
 * holds key channel perm[h][r]):
 *   S_bar = Lambda S;  delta = v - S_bar^T k;  S = S_bar + beta k delta^T;
 *   o = scale * S^T q.
 * GDN (is_kda = 0): Lambda = exp(g) I with one g. KDA: Lambda = diag(exp(g)).
 * kb, qb, gb (KDA) are the d_k bf16 operands in natural channel order, so they
 * are read through the permutation (section 5.2); vb has d_v values.
 */
static void orc_step(int is_kda, int dk, int dv, const uint8_t* perm, int h, float* S,
                     const uint16_t* kb, const uint16_t* qb, const uint16_t* gb,
                     uint16_t beta_bits, const uint16_t* vb, float scale, float* ob) {
  float* kp = (float*)malloc((size_t)dk * sizeof(float));
  float* qp = (float*)malloc((size_t)dk * sizeof(float));
  float* a = (float*)malloc((size_t)dk * sizeof(float));
  float* delta = (float*)malloc((size_t)dv * sizeof(float));
  for (int r = 0; r < dk; ++r) {
    int u = orc_perm_at(perm, h, dk, r);
    kp[r] = orc_from_bf16(kb[u]);
    qp[r] = orc_from_bf16(qb[u]);
    a[r] = expf(orc_from_bf16(is_kda ? gb[u] : gb[0]));
  }
  float bt = orc_from_bf16(beta_bits);

  /* decay: S_bar = Lambda S */
  for (int r = 0; r < dk; ++r)
    for (int j = 0; j < dv; ++j) S[(size_t)r * dv + j] = a[r] * S[(size_t)r * dv + j];

  /* key read-out and residual: delta = v - S_bar^T k */
  for (int j = 0; j < dv; ++j) {
    float acc = 0.0f;
    for (int r = 0; r < dk; ++r) acc = acc + kp[r] * S[(size_t)r * dv + j];
    delta[j] = orc_from_bf16(vb[j]) - acc;
  }

  /* rank-1 delta update: S = S_bar + beta k delta^T */
  for (int r = 0; r < dk; ++r) {
    float bk = bt * kp[r];
    for (int j = 0; j < dv; ++j) S[(size_t)r * dv + j] = S[(size_t)r * dv + j] + bk * delta[j];
  }

  /* read-out of the updated state: o = scale * S^T q */
  for (int j = 0; j < dv; ++j) {
    float acc = 0.0f;
    for (int r = 0; r < dk; ++r) acc = acc + qp[r] * S[(size_t)r * dv + j];
    ob[j] = scale * acc;
  }
  free(kp); free(qp); free(a); free(delta);
}

/*
 * One decode step of one layer for B requests (section 3.1, Eq. (1)): the
 * tile is decoded, updated by one token (orc_step) and stored per its tier
 * (section 3.2). q, k: bf16 [B, HK, dk]; v: [B, HV, dv]; g: [B, HV] (GDN) or
 * [B, HV, dk] (KDA); beta: [B, HV]; o fp32 [B, HV, dv]. If pre_out is not
 * NULL it receives the updated state before re-encoding, [B, HV, dk, dv] in
 * tile-row order (used for the error analysis of Eq. (5)).
 */
void orc_update(int is_kda, int kind, const int32_t* fmt, int dk, int dv, int k_hi,
                uint8_t* pool, int64_t slot_stride, int64_t tile_stride, int num_slots,
                const int32_t* slot_idx, int B, int HK, int HV, const uint16_t* q,
                const uint16_t* k, const uint16_t* v, const uint16_t* g,
                const uint16_t* beta, const uint8_t* perm, float scale, float* o,
                float* pre_out) {
  const orc_fmt_t f = orc_fmt(fmt, dv);
  int64_t ntiles = (int64_t)B * HV;
  int group = HV / HK;
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t t = 0; t < ntiles; ++t) {
    int b = (int)(t / HV), h = (int)(t % HV);
    int hk = h / group;
    float* ob = o + (size_t)t * dv;
    int slot = slot_idx[b];
    if (slot < 0 || slot >= num_slots) {
      for (int j = 0; j < dv; ++j) ob[j] = 0.0f;
      continue;
    }
    uint8_t* tile = pool + (size_t)slot * slot_stride + (size_t)h * tile_stride;
    float* S = (float*)malloc((size_t)dk * dv * sizeof(float));
    orc_tile_decode(kind, f, dk, dv, k_hi, tile, S);
    const uint16_t* gb = is_kda ? g + ((size_t)b * HV + h) * dk : g + (size_t)b * HV + h;
    orc_step(is_kda, dk, dv, perm, h, S, k + ((size_t)b * HK + hk) * dk,
             q + ((size_t)b * HK + hk) * dk, gb, beta[(size_t)b * HV + h],
             v + ((size_t)b * HV + h) * dv, scale, ob);
    if (pre_out) memcpy(pre_out + (size_t)t * dk * dv, S, (size_t)dk * dv * sizeof(float));
    /* store: the high tier rounded, Eq. (3) per low-tier group */
    orc_tile_encode(kind, f, dk, dv, k_hi, S, tile);
    free(S);
  }
}

/*
 * Prefill of one chunk of T tokens per request (App. A.5, prefill path): the
 * tile is decoded once, the recurrence runs in fp32 for t = 0 .. T-1
 * (orc_step, o_t from the state updated by token t), and only the state after
 * the last token is stored per its tier. Inputs carry a token axis after the
 * request axis: q, k [B, T, HK, dk]; v [B, T, HV, dv]; g [B, T, HV] (GDN) or
 * [B, T, HV, dk] (KDA); beta [B, T, HV]; o fp32 [B, T, HV, dv].
 */
void orc_prefill(int is_kda, int kind, const int32_t* fmt, int dk, int dv, int k_hi,
                 uint8_t* pool, int64_t slot_stride, int64_t tile_stride, int num_slots,
                 const int32_t* slot_idx, int B, int T, int HK, int HV, const uint16_t* q,
                 const uint16_t* k, const uint16_t* v, const uint16_t* g,
                 const uint16_t* beta, const uint8_t* perm, float scale, float* o) {
  const orc_fmt_t f = orc_fmt(fmt, dv);
  int64_t ntiles = (int64_t)B * HV;
  int group = HV / HK;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t ti = 0; ti < ntiles; ++ti) {
    int b = (int)(ti / HV), h = (int)(ti % HV);
    int hk = h / group;
    int slot = slot_idx[b];
    if (slot < 0 || slot >= num_slots) {
      for (int t = 0; t < T; ++t)
        memset(o + (((size_t)b * T + t) * HV + h) * dv, 0, (size_t)dv * sizeof(float));
      continue;
    }
    uint8_t* tile = pool + (size_t)slot * slot_stride + (size_t)h * tile_stride;
    float* S = (float*)malloc((size_t)dk * dv * sizeof(float));
    orc_tile_decode(kind, f, dk, dv, k_hi, tile, S);
    for (int t = 0; t < T; ++t) {
      size_t bt = (size_t)b * T + t;
      const uint16_t* gb = is_kda ? g + (bt * HV + h) * dk : g + bt * HV + h;
      orc_step(is_kda, dk, dv, perm, h, S, k + (bt * HK + hk) * dk, q + (bt * HK + hk) * dk, gb,
               beta[bt * HV + h], v + (bt * HV + h) * dv, scale, o + (bt * HV + h) * dv);
    }
    orc_tile_encode(kind, f, dk, dv, k_hi, S, tile);
    free(S);
  }
}

/* Packed zero state for every head of the listed slots. */
void orc_reset(int kind, const int32_t* fmt, int dk, int dv, int k_hi, uint8_t* pool,
               int64_t slot_stride, int64_t tile_stride, int num_slots, const int32_t* slots,
               int n, int HV) {
  const orc_fmt_t f = orc_fmt(fmt, dv);
  float* Z = (float*)calloc((size_t)dk * dv, sizeof(float));
  for (int i = 0; i < n; ++i) {
    if (slots[i] < 0 || slots[i] >= num_slots) continue;
    for (int h = 0; h < HV; ++h)
      orc_tile_encode(kind, f, dk, dv, k_hi, Z,
                      pool + (size_t)slots[i] * slot_stride + (size_t)h * tile_stride);
  }
  free(Z);
}

/* -------------------------------------------- offline channel selection */

/* Squared reconstruction error of one row under the low-tier quantizer,
 * summed in double in ascending column order (one term of Eq. (8)). */
static double orc_row_error(const float* x, int n) {
  float s, z;
  orc_quant_params(x, n, &s, &z);
  double acc = 0.0;
  for (int j = 0; j < n; ++j) {
    float xh = orc_decode(orc_code(x[j], s, z), s, z);
    double e = (double)xh - (double)x[j];
    acc = acc + e * e;
  }
  return acc;
}

typedef struct {
  double c;
  int u;
} orc_ranked;

static int orc_rank_cmp(const void* pa, const void* pb) {
  const orc_ranked* a = (const orc_ranked*)pa;
  const orc_ranked* b = (const orc_ranked*)pb;
  if (a->c > b->c) return -1; /* larger score first */
  if (a->c < b->c) return 1;
  return a->u - b->u;         /* ties: lower channel first */
}

/*
 * Alg. 1 (App. A.4) with the estimates of App. A.2, Eq. (14)-(15), on one
 * calibration domain (so the domain-balanced mean of Eq. (13) is a plain
 * mean over the N samples):
 *   E_u = (1/N) sum_n ||Q_lo(S_n[u,:]) - S_n[u,:]||^2
 *   a_eff = exp((1/N) sum_n log a_n[u]),  P_u = 1 / max(1 - a_eff^2, tau)
 *   C_u = E_u P_u;  keep TopK_{k_hi}(C);  perm = kept ascending ++ rest ascending.
 * states: fp32 [N, H, dk, dv]; log_decay: [N, H] (GDN) or [N, H, dk] (KDA).
 * Outputs: sel [H, k_hi], perm [H, dk], and optionally E, P, C [H, dk].
 */
int orc_select(int is_kda, int N, int H, int dk, int dv, const float* states,
               const float* log_decay, int k_hi, double tau, int32_t* sel,
               uint8_t* perm, double* E_out, double* P_out, double* C_out) {
  if (N <= 0 || H <= 0 || dk <= 0 || dk > 256 || dv <= 0 || k_hi < 0 || k_hi > dk)
    return 1;
  double* err = (double*)malloc((size_t)N * H * dk * sizeof(double));
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)N * H * dk; ++i)
    err[i] = orc_row_error(states + (size_t)i * dv, dv);

  orc_ranked* rk = (orc_ranked*)malloc((size_t)dk * sizeof(orc_ranked));
  unsigned char* keep = (unsigned char*)malloc((size_t)dk);
  for (int h = 0; h < H; ++h) {
    for (int u = 0; u < dk; ++u) {
      double e = 0.0, l = 0.0;
      for (int n = 0; n < N; ++n) {
        e = e + err[((size_t)n * H + h) * dk + u];
        l = l + (double)(is_kda ? log_decay[((size_t)n * H + h) * dk + u]
                                : log_decay[(size_t)n * H + h]);
      }
      double E = e / (double)N;
      double a_eff = exp(l / (double)N);
      double one_minus = 1.0 - a_eff * a_eff;
      double P = 1.0 / (one_minus > tau ? one_minus : tau);
      double C = E * P;
      if (E_out) E_out[(size_t)h * dk + u] = E;
      if (P_out) P_out[(size_t)h * dk + u] = P;
      if (C_out) C_out[(size_t)h * dk + u] = C;
      rk[u].c = C;
      rk[u].u = u;
    }
    qsort(rk, (size_t)dk, sizeof(orc_ranked), orc_rank_cmp);
    memset(keep, 0, (size_t)dk);
    for (int i = 0; i < k_hi; ++i) keep[rk[i].u] = 1;
    int p = 0, s = 0;
    for (int u = 0; u < dk; ++u)
      if (keep[u]) {
        perm[(size_t)h * dk + p++] = (uint8_t)u;
        sel[(size_t)h * k_hi + s++] = u;
      }
    for (int u = 0; u < dk; ++u)
      if (!keep[u]) perm[(size_t)h * dk + p++] = (uint8_t)u;
  }
  free(rk);
  free(keep);
  free(err);
  return 0;
}

/* ------------------------------------------- calibration over a trajectory */

/* ||Q_lo(x) - x||^2 of one row of n values, for the low tier of format f: one
 * (s, z) per row (Eq. (3)), or groups of f.group values with FP16 (s, z), in
 * the block-32 transformed domain when f.hadamard (App. A.1). The
 * reconstruction is taken back to the state's domain before the difference;
 * squared differences are summed in double over ascending columns. */
static double orc_row_error_fmt(const float* x, int n, orc_fmt_t f) {
  if (f.code != ORC_CODE_U8) return NAN;  /* calibration takes the UINT8 tiers */
  if (!f.meta_fp16) return orc_row_error(x, n);
  double acc = 0.0;
  for (int g0 = 0; g0 < n; g0 += f.group) {
    const float* xg = x + g0;
    float y[256], yq[256], xr[256];
    uint8_t c[256];
    if (f.hadamard) orc_hadamard32(xg, y);
    else memcpy(y, xg, (size_t)f.group * sizeof(float));
    float s, z;
    orc_quant_group_fp16(y, f.group, c, &s, &z);
    orc_dequant_row(c, f.group, s, z, yq);
    if (f.hadamard) orc_hadamard32(yq, xr);
    else memcpy(xr, yq, (size_t)f.group * sizeof(float));
    for (int j = 0; j < f.group; ++j) {
      double e = (double)xr[j] - (double)xg[j];
      acc = acc + e * e;
    }
  }
  return acc;
}

/*
 * One sampled state write (App. A.2): for each of the B requests in turn and
 * each head h and key channel u, adds to the running sums
 *   err[h,u]  += ||Q_lo(S_b[h,u,:]) - S_b[h,u,:]||^2        (Eq. (14))
 *   en[h,u]   += ||S_b[h,u,:]||^2                            (state energy)
 *   loga[h,u] += log a_b[h,u] (the bf16 log-decay g widened) (Eq. (15))
 * and 1 to *count. states: fp32 [B, H, dk, dv] in natural channel order;
 * g: bf16 [B, H] (GDN) or [B, H, dk] (KDA). fmt as for orc_pack (NULL: one
 * fp32 (s, z) per row).
 */
void orc_calib_accumulate(int is_kda, const int32_t* fmt, int B, int H, int dk, int dv,
                          const float* states, const uint16_t* g, double* err, double* en,
                          double* loga, double* count) {
  orc_fmt_t f = orc_fmt(fmt, dv);
  for (int b = 0; b < B; ++b) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < (int64_t)H * dk; ++i) {
      const int h = (int)(i / dk), u = (int)(i % dk);
      const float* x = states + (((size_t)b * H + h) * dk + u) * dv;
      double e2 = 0.0;
      for (int j = 0; j < dv; ++j) e2 = e2 + (double)x[j] * (double)x[j];
      const uint16_t gb = is_kda ? g[((size_t)b * H + h) * dk + u] : g[(size_t)b * H + h];
      err[i] = err[i] + orc_row_error_fmt(x, dv, f);
      en[i] = en[i] + e2;
      loga[i] = loga[i] + (double)orc_from_bf16(gb);
    }
    *count = *count + 1.0;
  }
}

/*
 * Selection from accumulated statistics (Alg. 1 with App. A.2's estimates and
 * the domain-balanced mean of Eq. (13)): for each head and key channel the
 * mean over domains (ascending) of each domain's mean, then
 *   a_eff = exp(mean log a),  P = 1 / max(1 - a_eff^2, tau)   (Eq. (15))
 * and the score of the selector: 0 C = E P, 1 E, 2 P, 3 the mean squared
 * row norm, 4 the caller's rand [H, dk]. The k_hi largest scores are kept
 * (ties to the lower channel); perm is the stable partition.
 * sums: [D][3][H][dk] (err, en, loga); counts: [D]. stats (nullable):
 * [4][H][dk] = E, P, mean squared norm, mean log a. Returns nonzero if a
 * domain has no samples or an argument is out of range.
 */
int orc_calib_finalize(int D, int H, int dk, const double* sums, const double* counts,
                       int selector, int k_hi, double tau, const double* rand, int32_t* sel,
                       uint8_t* perm, double* score, double* stats) {
  if (D <= 0 || H <= 0 || dk <= 0 || dk > 256 || k_hi < 0 || k_hi > dk || selector < 0 ||
      selector > 4 || (selector == 4 && !rand))
    return 1;
  for (int d = 0; d < D; ++d)
    if (!(counts[d] > 0.0)) return 1;
  const size_t hk = (size_t)H * dk;
  orc_ranked* rk = (orc_ranked*)malloc((size_t)dk * sizeof(orc_ranked));
  unsigned char* keep = (unsigned char*)malloc((size_t)dk);
  for (int h = 0; h < H; ++h) {
    for (int u = 0; u < dk; ++u) {
      const size_t i = (size_t)h * dk + u;
      double E = 0.0, En = 0.0, L = 0.0;
      for (int d = 0; d < D; ++d) {
        const double* s = sums + (size_t)d * 3 * hk;
        E = E + s[i] / counts[d];
        En = En + s[hk + i] / counts[d];
        L = L + s[2 * hk + i] / counts[d];
      }
      E = E / (double)D;
      En = En / (double)D;
      L = L / (double)D;
      double a_eff = exp(L);
      double one_minus = 1.0 - a_eff * a_eff;
      double P = 1.0 / (one_minus > tau ? one_minus : tau);
      double c;
      if (selector == 0) c = E * P;
      else if (selector == 1) c = E;
      else if (selector == 2) c = P;
      else if (selector == 3) c = En;
      else c = rand[i];
      if (score) score[i] = c;
      if (stats) {
        stats[i] = E;
        stats[hk + i] = P;
        stats[2 * hk + i] = En;
        stats[3 * hk + i] = L;
      }
      rk[u].c = c;
      rk[u].u = u;
    }
    qsort(rk, (size_t)dk, sizeof(orc_ranked), orc_rank_cmp);
    memset(keep, 0, (size_t)dk);
    for (int i = 0; i < k_hi; ++i) keep[rk[i].u] = 1;
    int p = 0, s = 0;
    for (int u = 0; u < dk; ++u)
      if (keep[u]) {
        perm[(size_t)h * dk + p++] = (uint8_t)u;
        sel[(size_t)h * k_hi + s++] = u;
      }
    for (int u = 0; u < dk; ++u)
      if (!keep[u]) perm[(size_t)h * dk + p++] = (uint8_t)u;
  }
  free(rk);
  free(keep);
  return 0;
}
