// Calibration of the protected key channels on the device (App. A.2 Eq. (13)
// to (15), Alg. 1 of App. A.4; the selector ablation of section 6; the split
// agreement of App. B).
//
// The reference (FP32) trajectory runs in an FP32 pool, a stride of tokens at
// a time, through the prefill kernel; after each stride the sampled state
// write is folded into per-domain double accumulators:
//   err[h][u]  += || Q_lo(S[h,u,:]) - S[h,u,:] ||^2   (Eq. (14))
//   en[h][u]   += || S[h,u,:] ||^2                    (state-energy selector)
//   loga[h][u] += log a[h,u] of the sampled token     (Eq. (15))
// so no tensor of sampled states is ever formed. Every sum follows the order
// of the definitions (columns ascending within a row, samples in the order
// they arrive) with IEEE operations only, so equal states give equal
// accumulators bit for bit. The estimates, the score of each selector, the
// top-k partition and the split-agreement measures are computed on the host
// in double.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

#pragma clang fp contract(off)

namespace damp {
namespace {

constexpr int kCalibThreads = 256;

struct CalibParams {
  const uint8_t* layer_base;
  uint64_t slot_stride;
  uint64_t tile_stride;
  const int32_t* slot_idx;
  const uint8_t* perm;   // [H, d_k] or NULL
  const uint16_t* g;     // bf16 log-decay: [B, H] (GDN) or [B, H, d_k] (KDA), request stride g_bstride
  int64_t g_bstride;     // elements between consecutive requests of g
  double* err;           // [H, d_k] of this domain
  double* en;
  double* loga;
  double* count;         // this domain's sample count
  int32_t B;
  int32_t num_slots;
  int32_t H;
  int32_t dk;
  int32_t dv;
  int32_t is_kda;
  int32_t paper;         // groups of 32 with FP16 (s, z)
  int32_t had;           // block-32 transform of each group
};

// s of Eq. (3) from a row's or group's extrema, IEEE division; constant and
// zero groups as for the stored tiers.
__device__ __forceinline__ float qscale_exact(float lo, float hi) {
  float s = __fdiv_rn(__fsub_rn(hi, lo), 255.0f);
  if (!(s >= FLT_MIN)) {
    s = __fdiv_rn(fabsf(lo), 255.0f);
    if (!(s >= FLT_MIN)) s = 1.0f;
  }
  return s;
}

__device__ __forceinline__ float decode_exact(float x, float s, float z) {
  float c = __fadd_rn(rintf(__fdiv_rn(x, s)), z);
  c = c < 0.0f ? 0.0f : (c > 255.0f ? 255.0f : c);
  return __fmul_rn(s, __fsub_rn(c, z));
}

// (xh - x)^2 in double, the term of || Q_lo(x) - x ||^2
__device__ __forceinline__ double sq_term(float xh, float x) {
  const double e = __dsub_rn(static_cast<double>(xh), static_cast<double>(x));
  return __dmul_rn(e, e);
}

// Extrema over the lanes whose bit `span` and above agree (span = 64: the
// wave, 32: each half).
template <int SPAN>
__device__ __forceinline__ void lane_minmax(float& lo, float& hi) {
#pragma unroll
  for (int m = 1; m < SPAN; m <<= 1) {
    lo = fminf(lo, __shfl_xor(lo, m, 64));
    hi = fmaxf(hi, __shfl_xor(hi, m, 64));
  }
}

// Per-wave scratch for the statistics of one row sample (d_v <= 128).
struct RowScratch {
  float x[128];   // the row
  float yh[128];  // paper tiers with the transform: the reconstruction, transformed domain
  double te[128];  // per column: (Q_lo(x) - x)^2
  double tn[128];  // per column: x^2
};

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

// || Q_lo(x) - x ||^2 and || x ||^2 of one row by one wave, a lane per column
// (columns lane, lane + 64). Every per-column operation is written out as
// the definition: the row's (or, for the paper's tiers, each group of 32's)
// s and z of Eq. (3) with IEEE division, the FP16 rounding of the stored
// group (s, z), the normalized block-32 transform as its direct sum over
// ascending j, and the reconstruction s (c - z). The extrema are order-free;
// the two sums over the columns run in ascending column order in one lane
// each (lanes 0 and 32). Returns the sums in those two lanes.
__device__ void row_stats_wave(const float* xrow, int dv, bool paper, bool had, RowScratch& sc,
                               int lane, double& err, double& en) {
  for (int j = lane; j < dv; j += 64) sc.x[j] = xrow[j];
  wave_sync();
  if (!paper) {
    float lo = INFINITY, hi = -INFINITY;
    for (int j = lane; j < dv; j += 64) {
      lo = fminf(lo, sc.x[j]);
      hi = fmaxf(hi, sc.x[j]);
    }
    lane_minmax<64>(lo, hi);
    const float s = qscale_exact(lo, hi);
    const float z = rintf(__fdiv_rn(-lo, s));
    for (int j = lane; j < dv; j += 64) {
      const float xv = sc.x[j];
      sc.te[j] = sq_term(decode_exact(xv, s, z), xv);
      sc.tn[j] = __dmul_rn(static_cast<double>(xv), static_cast<double>(xv));
    }
  } else {
    // lane holds output i = j % 32 of group j / 32, for j = lane + 64 m; the
    // 32 lanes of a half-wave hold one group
    float y[2], yh[2];
    const int nm = (dv + 63) / 64;
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const int j = lane + 64 * m;
      if (m >= nm || j >= dv) {
        y[m] = 0.0f;
        continue;
      }
      const int base = j & ~31, i = j & 31;
      if (had) {
        float acc = 0.0f;
        for (int jj = 0; jj < 32; ++jj)
          acc = (__builtin_popcount(static_cast<unsigned>(i & jj)) & 1) ? __fsub_rn(acc, sc.x[base + jj])
                                                                        : __fadd_rn(acc, sc.x[base + jj]);
        y[m] = __fmul_rn(acc, kInvSqrt32);
      } else {
        y[m] = sc.x[j];
      }
    }
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const int j = lane + 64 * m;
      const bool on = m < nm && j < dv;
      float lo = on ? y[m] : INFINITY, hi = on ? y[m] : -INFINITY;
      lane_minmax<32>(lo, hi);
      if (!on) {
        yh[m] = 0.0f;
        continue;
      }
      const float s = qscale_exact(lo, hi);
      float s16 = round_f16(s);
      if (!(s16 > 0.0f)) s16 = 5.9604644775390625e-08f;  // smallest positive FP16
      if (s16 > 65504.0f) s16 = 65504.0f;
      float zf = rintf(__fdiv_rn(-lo, s16));
      if (zf > 65504.0f) zf = 65504.0f;
      if (zf < -65504.0f) zf = -65504.0f;
      const float z16 = round_f16(zf);
      yh[m] = decode_exact(y[m], s16, z16);
    }
    if (had) {
      for (int m = 0; m < nm; ++m) {
        const int j = lane + 64 * m;
        if (j < dv) sc.yh[j] = yh[m];
      }
      wave_sync();
    }
    for (int m = 0; m < nm; ++m) {
      const int j = lane + 64 * m;
      if (j >= dv) continue;
      float xh = yh[m];
      if (had) {  // back from the transformed domain, the same direct sum
        const int base = j & ~31, i = j & 31;
        float acc = 0.0f;
        for (int jj = 0; jj < 32; ++jj)
          acc = (__builtin_popcount(static_cast<unsigned>(i & jj)) & 1) ? __fsub_rn(acc, sc.yh[base + jj])
                                                                        : __fadd_rn(acc, sc.yh[base + jj]);
        xh = __fmul_rn(acc, kInvSqrt32);
      }
      const float xv = sc.x[j];
      sc.te[j] = sq_term(xh, xv);
      sc.tn[j] = __dmul_rn(static_cast<double>(xv), static_cast<double>(xv));
    }
  }
  wave_sync();
  // ascending sums: lane 0 the error terms, lane 32 the energies
  double acc = 0.0;
  if (lane == 0 || lane == 32) {
    const double* src = lane == 0 ? sc.te : sc.tn;
    for (int j = 0; j < dv; ++j) acc = __dadd_rn(acc, src[j]);
  }
  err = acc;
  en = acc;
  wave_sync();  // the scratch is reused by the wave's next sample
}

// One workgroup per (head, tile row). Its four waves evaluate up to 256
// samples at a time, one sample per wave at a time, into LDS; thread 0 then
// adds them to the accumulators in sample order, continuing from the values
// already stored.
__global__ __launch_bounds__(kCalibThreads) void calib_accumulate_kernel(const CalibParams p) {
  __shared__ double se[kCalibThreads], sn[kCalibThreads], sl[kCalibThreads];
  __shared__ int sv[kCalibThreads];
  __shared__ RowScratch scr[kCalibThreads / 64];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int h = blockIdx.x / p.dk;
  const int r = blockIdx.x % p.dk;
  const int u = p.perm ? static_cast<int>(p.perm[static_cast<size_t>(h) * p.dk + r]) : r;
  const size_t hu = static_cast<size_t>(h) * p.dk + u;
  double acc_e = 0.0, acc_n = 0.0, acc_l = 0.0, nvalid = 0.0;
  if (t == 0) {
    acc_e = p.err[hu];
    acc_n = p.en[hu];
    acc_l = p.loga[hu];
  }
  for (int b0 = 0; b0 < p.B; b0 += kCalibThreads) {
    const int n = min(kCalibThreads, p.B - b0);
    for (int i = wave; i < n; i += kCalibThreads / 64) {
      const int b = b0 + i;
      const int slot = p.slot_idx[b];
      const bool valid = slot >= 0 && slot < p.num_slots;
      if (valid) {
        const float* x = reinterpret_cast<const float*>(
            p.layer_base + static_cast<size_t>(slot) * p.slot_stride +
            static_cast<size_t>(h) * p.tile_stride) + static_cast<size_t>(r) * p.dv;
        double e = 0.0, e2 = 0.0;
        row_stats_wave(x, p.dv, p.paper != 0, p.had != 0, scr[wave], lane, e, e2);
        if (lane == 0) {
          se[i] = e;
          const uint16_t gb = p.is_kda ? p.g[b * p.g_bstride + static_cast<int64_t>(h) * p.dk + u]
                                       : p.g[b * p.g_bstride + h];
          sl[i] = static_cast<double>(bf16_to_f32(gb));
        }
        if (lane == 32) sn[i] = e2;
      }
      if (lane == 0) sv[i] = valid ? 1 : 0;
    }
    __syncthreads();
    if (t == 0) {
      for (int i = 0; i < n; ++i) {
        if (!sv[i]) continue;
        acc_e = __dadd_rn(acc_e, se[i]);
        acc_n = __dadd_rn(acc_n, sn[i]);
        acc_l = __dadd_rn(acc_l, sl[i]);
        nvalid += 1.0;
      }
    }
    __syncthreads();
  }
  if (t == 0) {
    p.err[hu] = acc_e;
    p.en[hu] = acc_n;
    p.loga[hu] = acc_l;
    if (blockIdx.x == 0) *p.count = __dadd_rn(*p.count, nvalid);
  }
}

__global__ __launch_bounds__(256) void fill_zero_kernel(double* p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.0;
}

int64_t sums_per_domain(const damp_calib* c) {
  return 3 * static_cast<int64_t>(c->num_heads) * c->lo.d_k;
}

damp_status check_calib(const damp_calib* c, const char* name) {
  if (!c) return fail(DAMP_ERR_INVALID_ARG, "%s: calib is NULL", name);
  if (!c->sums) return fail(DAMP_ERR_INVALID_ARG, "%s: calib has no accumulators", name);
  if (c->num_domains <= 0 || c->num_domains > DAMP_CALIB_MAX_DOMAINS || c->num_heads <= 0)
    return fail(DAMP_ERR_INVALID_ARG, "%s: calib is not initialized", name);
  if (c->bytes < damp_calib_required_bytes(c->num_domains, c->num_heads, c->lo.d_k))
    return fail(DAMP_ERR_INVALID_ARG, "%s: calib accumulators are too small", name);
  return DAMP_OK;
}

damp_status accumulate(const damp_calib* c, int32_t domain, const damp_pool* pool, int32_t layer,
                       const int32_t* slot_idx, int32_t B, const uint8_t* perm,
                       const uint16_t* g, int64_t g_bstride, hipStream_t stream) {
  CalibParams p;
  p.layer_base = layer_base(pool, layer);
  p.tile_stride = pool->tile_stride;
  p.slot_stride = pool->tile_stride * static_cast<uint64_t>(pool->num_v_heads);
  p.slot_idx = slot_idx;
  p.perm = perm;
  p.g = g;
  p.g_bstride = g_bstride;
  const int64_t per = sums_per_domain(c);
  const int64_t hk = static_cast<int64_t>(c->num_heads) * c->lo.d_k;
  double* base = c->sums + domain * per;
  p.err = base;
  p.en = base + hk;
  p.loga = base + 2 * hk;
  p.count = c->sums + c->num_domains * per + domain;
  p.B = B;
  p.num_slots = pool->num_slots;
  p.H = c->num_heads;
  p.dk = c->lo.d_k;
  p.dv = c->lo.d_v;
  p.is_kda = c->is_kda;
  p.paper = layout_is_paper(&c->lo) ? 1 : 0;
  p.had = c->lo.hadamard;
  hipLaunchKernelGGL(calib_accumulate_kernel, dim3(static_cast<unsigned>(hk)),
                     dim3(kCalibThreads), 0, stream, p);
  return check_launch("damp_calib_accumulate");
}

damp_status check_fp32_pool(const damp_calib* c, const damp_pool* pool, int32_t layer,
                            const char* name) {
  damp_status st = check_pool(pool);
  if (st != DAMP_OK) return st;
  if (pool->layout.kind != DAMP_STATE_FP32)
    return fail(DAMP_ERR_INVALID_ARG, "%s: the calibration pool must hold FP32 states", name);
  if (pool->layout.d_k != c->lo.d_k || pool->layout.d_v != c->lo.d_v ||
      pool->num_v_heads != c->num_heads)
    return fail(DAMP_ERR_INVALID_ARG, "%s: pool shape (%d x %d, %d heads) differs from calib "
                "(%d x %d, %d heads)", name, pool->layout.d_k, pool->layout.d_v,
                pool->num_v_heads, c->lo.d_k, c->lo.d_v, c->num_heads);
  if (layer < 0 || layer >= pool->num_layers)
    return fail(DAMP_ERR_INVALID_ARG, "%s: layer %d outside [0, %d)", name, layer,
                pool->num_layers);
  return DAMP_OK;
}

// || Q_lo(x) - x ||^2 of independent rows (row i at states + i * dv) under
// the paper's UINT8 group tier, one row per wave, the same per-row
// evaluation as the accumulation above.
__global__ __launch_bounds__(256) void row_error_group_kernel(const float* __restrict__ states,
                                                              int64_t rows, int dv, int had,
                                                              double* __restrict__ err) {
  __shared__ RowScratch scr[4];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int64_t row = static_cast<int64_t>(blockIdx.x) * 4 + wave;
  if (row >= rows) return;  // whole waves leave: the evaluation synchronises within a wave only
  double e = 0.0, e2 = 0.0;
  row_stats_wave(states + row * dv, dv, true, had != 0, scr[wave], lane, e, e2);
  if (lane == 0) err[row] = e;
}

// Average ranks (ties share the mean of their positions), 1-based.
std::vector<double> ranks_of(const double* x, int n) {
  std::vector<int> idx(n);
  for (int i = 0; i < n; ++i) idx[i] = i;
  std::sort(idx.begin(), idx.end(), [&](int a, int b) { return x[a] < x[b]; });
  std::vector<double> rk(n);
  for (int i = 0; i < n;) {
    int j = i;
    while (j + 1 < n && x[idx[j + 1]] == x[idx[i]]) ++j;
    const double r = 0.5 * (static_cast<double>(i) + static_cast<double>(j)) + 1.0;
    for (int m = i; m <= j; ++m) rk[idx[m]] = r;
    i = j + 1;
  }
  return rk;
}

}  // namespace

void launch_row_errors_group(const float* states, int64_t rows, int dv, bool had, double* err,
                             hipStream_t stream) {
  const int64_t blocks = (rows + 3) / 4;
  hipLaunchKernelGGL(row_error_group_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     stream, states, rows, dv, had ? 1 : 0, err);
}

}  // namespace damp

extern "C" {

size_t damp_calib_required_bytes(int32_t num_domains, int32_t num_heads, int32_t d_k) {
  if (num_domains <= 0 || num_heads <= 0 || d_k <= 0) return 0;
  return sizeof(double) * static_cast<size_t>(num_domains) *
         (3 * static_cast<size_t>(num_heads) * static_cast<size_t>(d_k) + 1);
}

damp_status damp_calib_init(damp_calib* calib, const damp_layout* lo, int32_t is_kda,
                            int32_t num_heads, int32_t num_domains, void* sums, size_t bytes,
                            void* stream) {
  using namespace damp;
  clear_error();
  if (!calib || !lo || !sums)
    return fail(DAMP_ERR_INVALID_ARG, "damp_calib_init: a required pointer is NULL");
  if (reinterpret_cast<uintptr_t>(sums) % alignof(double) != 0)
    return fail(DAMP_ERR_INVALID_ARG, "damp_calib_init: accumulators must be 8-byte aligned");
  if (num_heads <= 0 || num_domains <= 0 || num_domains > DAMP_CALIB_MAX_DOMAINS)
    return fail(DAMP_ERR_INVALID_ARG, "damp_calib_init: num_heads = %d, num_domains = %d "
                "(at most %d)", num_heads, num_domains, DAMP_CALIB_MAX_DOMAINS);
  if (lo->kind != DAMP_STATE_MIXED || lo->d_k != lo->d_v || lo->d_k > 256)
    return fail(DAMP_ERR_INVALID_ARG, "damp_calib_init: Q_lo must be the low tier of a mixed "
                "layout with d_k == d_v <= 256");
  if (!layout_has_kernels(lo))
    return fail(DAMP_ERR_UNSUPPORTED, "damp_calib_init: no kernel for this low tier");
  const size_t need = damp_calib_required_bytes(num_domains, num_heads, lo->d_k);
  if (bytes < need)
    return fail(DAMP_ERR_INVALID_ARG, "damp_calib_init: accumulators need %zu bytes, got %zu",
                need, bytes);
  damp_calib c;
  c.lo = *lo;
  c.is_kda = is_kda ? 1 : 0;
  c.num_heads = num_heads;
  c.num_domains = num_domains;
  c.sums = static_cast<double*>(sums);
  c.bytes = bytes;
  const int64_t n = static_cast<int64_t>(need / sizeof(double));
  hipLaunchKernelGGL(fill_zero_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256),
                     0, as_stream(stream), c.sums, n);
  damp_status st = check_launch("damp_calib_init");
  if (st == DAMP_OK) *calib = c;
  return st;
}

damp_status damp_calib_accumulate(const damp_calib* calib, int32_t domain, const damp_pool* pool,
                                  int32_t layer, const int32_t* slot_idx, int32_t B,
                                  const uint8_t* perm, const uint16_t* g, void* stream) {
  using namespace damp;
  clear_error();
  const char* name = "damp_calib_accumulate";
  damp_status st = check_calib(calib, name);
  if (st != DAMP_OK) return st;
  st = check_fp32_pool(calib, pool, layer, name);
  if (st != DAMP_OK) return st;
  if (domain < 0 || domain >= calib->num_domains)
    return fail(DAMP_ERR_INVALID_ARG, "%s: domain %d outside [0, %d)", name, domain,
                calib->num_domains);
  if (B < 0 || B > 65535) return fail(DAMP_ERR_INVALID_ARG, "%s: B = %d outside [0, 65535]", name, B);
  if (B == 0) return DAMP_OK;
  if (!slot_idx || !g) return fail(DAMP_ERR_INVALID_ARG, "%s: a required pointer is NULL", name);
  const int64_t gb = calib->is_kda ? static_cast<int64_t>(calib->num_heads) * calib->lo.d_k
                                   : calib->num_heads;
  return accumulate(calib, domain, pool, layer, slot_idx, B, perm, g, gb, as_stream(stream));
}

damp_status damp_calibrate_sequence(const damp_calib* calib, int32_t domain,
                                    const damp_pool* pool, int32_t layer,
                                    const int32_t* slot_idx, int32_t B, int32_t T,
                                    int32_t stride, int32_t num_k_heads, const uint16_t* q,
                                    const uint16_t* k, const uint16_t* v, const uint16_t* g,
                                    const uint16_t* beta, void* stream) {
  using namespace damp;
  clear_error();
  const char* name = "damp_calibrate_sequence";
  damp_status st = check_calib(calib, name);
  if (st != DAMP_OK) return st;
  st = check_fp32_pool(calib, pool, layer, name);
  if (st != DAMP_OK) return st;
  if (domain < 0 || domain >= calib->num_domains)
    return fail(DAMP_ERR_INVALID_ARG, "%s: domain %d outside [0, %d)", name, domain,
                calib->num_domains);
  if (B < 0 || B > 65535) return fail(DAMP_ERR_INVALID_ARG, "%s: B = %d outside [0, 65535]", name, B);
  if (T < 0 || stride <= 0)
    return fail(DAMP_ERR_INVALID_ARG, "%s: T = %d, stride = %d", name, T, stride);
  if (num_k_heads <= 0 || calib->num_heads % num_k_heads != 0 ||
      (calib->is_kda && num_k_heads != calib->num_heads))
    return fail(DAMP_ERR_INVALID_ARG, "%s: num_k_heads %d does not divide %d heads%s", name,
                num_k_heads, calib->num_heads, calib->is_kda ? " (KDA needs equal counts)" : "");
  if (B == 0 || T == 0) return DAMP_OK;
  if (!slot_idx || !q || !k || !v || !g || !beta)
    return fail(DAMP_ERR_INVALID_ARG, "%s: a required pointer is NULL", name);
  st = debug_check_slots(pool, slot_idx, B, as_stream(stream), name);
  if (st != DAMP_OK) return st;
  const bool kda = calib->is_kda != 0;
  const int64_t per_tok = kda ? static_cast<int64_t>(calib->num_heads) * calib->lo.d_k
                              : calib->num_heads;
  hipStream_t s = as_stream(stream);
  for (int32_t t0 = 0; t0 < T; t0 += stride) {
    const int32_t n = std::min(stride, T - t0);
    prefill_window(kda, pool, layer, slot_idx, B, t0, n, T, num_k_heads, q, k, v, g, beta,
                   nullptr, 1.0f, nullptr, false, s);
    st = check_launch(name);
    if (st != DAMP_OK) return st;
    if (n < stride) break;  // a trailing partial stride is run but not sampled
    st = accumulate(calib, domain, pool, layer, slot_idx, B, nullptr,
                    g + (t0 + stride - 1) * per_tok, per_tok * T, s);
    if (st != DAMP_OK) return st;
  }
  return DAMP_OK;
}

damp_status damp_calib_finalize(const damp_calib* calib, int32_t selector, int32_t k_hi,
                                double tau, const double* rand_scores, int32_t* sel_out,
                                uint8_t* perm_out, double* score_out, double* stats_out,
                                void* stream) {
  using namespace damp;
  clear_error();
  const char* name = "damp_calib_finalize";
  damp_status st = check_calib(calib, name);
  if (st != DAMP_OK) return st;
  const int H = calib->num_heads, dk = calib->lo.d_k, D = calib->num_domains;
  if (selector < DAMP_SEL_DAMP || selector > DAMP_SEL_RANDOM)
    return fail(DAMP_ERR_INVALID_ARG, "%s: unknown selector %d", name, selector);
  if (k_hi < 0 || k_hi > dk)
    return fail(DAMP_ERR_INVALID_ARG, "%s: k_hi = %d outside [0, %d]", name, k_hi, dk);
  if (!(tau > 0.0)) return fail(DAMP_ERR_INVALID_ARG, "%s: tau must be > 0", name);
  if (!perm_out || (k_hi > 0 && !sel_out) || (selector == DAMP_SEL_RANDOM && !rand_scores))
    return fail(DAMP_ERR_INVALID_ARG, "%s: a required pointer is NULL", name);

  const int64_t per = sums_per_domain(calib);
  const size_t n = static_cast<size_t>(D * per + D);
  std::vector<double> h(n);
  hipStream_t s = as_stream(stream);
  hipError_t e = hipMemcpyAsync(h.data(), calib->sums, n * sizeof(double), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return fail(DAMP_ERR_HIP, "%s: %s", name, hipGetErrorString(e));
  const double* count = h.data() + D * per;
  for (int d = 0; d < D; ++d)
    if (!(count[d] > 0.0)) return fail(DAMP_ERR_INVALID_ARG, "%s: domain %d has no samples", name, d);

  const size_t hk = static_cast<size_t>(H) * dk;
  std::vector<double> score(dk);
  std::vector<int> order(dk);
  std::vector<char> keep(dk);
  for (int hh = 0; hh < H; ++hh) {
    for (int u = 0; u < dk; ++u) {
      const size_t i = static_cast<size_t>(hh) * dk + u;
      // Eq. (13): the mean over domains of the per-domain means
      double E = 0.0, En = 0.0, L = 0.0;
      for (int d = 0; d < D; ++d) {
        const double* b = h.data() + d * per;
        E = E + b[i] / count[d];
        En = En + b[hk + i] / count[d];
        L = L + b[2 * hk + i] / count[d];
      }
      E = E / static_cast<double>(D);
      En = En / static_cast<double>(D);
      L = L / static_cast<double>(D);
      const double a_eff = std::exp(L);                       // Eq. (15)
      const double gap = 1.0 - a_eff * a_eff;
      const double P = 1.0 / (gap > tau ? gap : tau);
      double sc = 0.0;
      switch (selector) {
        case DAMP_SEL_DAMP: sc = E * P; break;                 // C = E P
        case DAMP_SEL_ERROR: sc = E; break;
        case DAMP_SEL_PERSISTENCE: sc = P; break;
        case DAMP_SEL_STATE_ENERGY: sc = En; break;
        default: sc = rand_scores[i]; break;
      }
      score[u] = sc;
      if (score_out) score_out[i] = sc;
      if (stats_out) {
        stats_out[i] = E;
        stats_out[hk + i] = P;
        stats_out[2 * hk + i] = En;
        stats_out[3 * hk + i] = L;
      }
      order[u] = u;
    }
    std::sort(order.begin(), order.end(), [&](int a, int b) {
      if (score[a] != score[b]) return score[a] > score[b];
      return a < b;
    });
    std::fill(keep.begin(), keep.end(), 0);
    for (int i = 0; i < k_hi; ++i) keep[order[i]] = 1;
    int p = 0, q = 0;
    for (int u = 0; u < dk; ++u)
      if (keep[u]) {
        perm_out[static_cast<size_t>(hh) * dk + p++] = static_cast<uint8_t>(u);
        sel_out[static_cast<size_t>(hh) * k_hi + q++] = u;
      }
    for (int u = 0; u < dk; ++u)
      if (!keep[u]) perm_out[static_cast<size_t>(hh) * dk + p++] = static_cast<uint8_t>(u);
  }
  return DAMP_OK;
}

double damp_topk_overlap(const int32_t* sel_a, const int32_t* sel_b, int32_t k) {
  if (!sel_a || !sel_b || k <= 0) return NAN;
  int common = 0;
  for (int i = 0; i < k; ++i)
    for (int j = 0; j < k; ++j)
      if (sel_a[i] == sel_b[j]) {
        ++common;
        break;
      }
  return static_cast<double>(common) / static_cast<double>(k);
}

double damp_spearman(const double* a, const double* b, int32_t n) {
  if (!a || !b || n < 2) return NAN;
  const std::vector<double> ra = damp::ranks_of(a, n), rb = damp::ranks_of(b, n);
  double ma = 0.0, mb = 0.0;
  for (int i = 0; i < n; ++i) {
    ma += ra[i];
    mb += rb[i];
  }
  ma /= n;
  mb /= n;
  double sab = 0.0, saa = 0.0, sbb = 0.0;
  for (int i = 0; i < n; ++i) {
    const double da = ra[i] - ma, db = rb[i] - mb;
    sab += da * db;
    saa += da * da;
    sbb += db * db;
  }
  if (!(saa > 0.0) || !(sbb > 0.0)) return NAN;
  return sab / std::sqrt(saa * sbb);
}

}  // extern "C"
