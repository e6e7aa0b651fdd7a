// Offline selection of the protected key channels (section 5.1 Eq. (8)-(10),
// App. A.2 Eq. (14)-(15), Alg. 1 of App. A.4).
//
// The device computes, for every calibration row S_n[h, u, :], the squared
// reconstruction error under the low-tier quantizer Q_lo: the per-row
// quantizer of Eq. (3) (one thread per row, ascending columns) or the paper's
// group tier (one wave per row, the calibration kernel's evaluation). Both
// use IEEE operations only (correctly rounded fp32 division, no contraction,
// double accumulation in ascending column order), so the per-row sums are
// reproducible bit for bit. A second pass sums each (head, channel) over the
// samples in ascending n, and the log-decays likewise, in double. The host
// then forms E, the geometric-mean decay, the persistence of Eq. (9),
// C = E P and the top-k_hi partition.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <mutex>

#include "internal.hpp"

#pragma clang fp contract(off)

namespace damp {
namespace {

__global__ __launch_bounds__(256) void row_error_kernel(const float* __restrict__ states,
                                                        int64_t rows, int dv,
                                                        double* __restrict__ err) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i >= rows) return;
  const float* x = states + i * dv;
  float lo = x[0], hi = x[0];
  for (int j = 1; j < dv; ++j) {
    const float xj = x[j];
    if (xj < lo) lo = xj;
    if (xj > hi) hi = xj;
  }
  float s = __fdiv_rn(__fsub_rn(hi, lo), 255.0f);
  if (!(s >= FLT_MIN)) {
    s = __fdiv_rn(fabsf(lo), 255.0f);
    if (!(s >= FLT_MIN)) s = 1.0f;
  }
  const float z = rintf(__fdiv_rn(-lo, s));
  double acc = 0.0;
  for (int j = 0; j < dv; ++j) {
    const float xj = x[j];
    float c = __fadd_rn(rintf(__fdiv_rn(xj, s)), z);
    c = c < 0.0f ? 0.0f : (c > 255.0f ? 255.0f : c);
    const float xh = __fmul_rn(s, __fsub_rn(c, z));
    const double e = __dsub_rn(static_cast<double>(xh), static_cast<double>(xj));
    acc = __dadd_rn(acc, __dmul_rn(e, e));
  }
  err[i] = acc;
}

// esum[h, u] = sum_n err[n, h, u] and lsum[h, u] = sum_n log a[n, h(, u)],
// both in double, n ascending: one thread per (head, channel).
__global__ __launch_bounds__(256) void sum_samples_kernel(const double* __restrict__ err,
                                                          const float* __restrict__ logs, int N,
                                                          int H, int dk, int is_kda,
                                                          double* __restrict__ esum,
                                                          double* __restrict__ lsum) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= H * dk) return;
  const int h = i / dk, u = i % dk;
  double e = 0.0, l = 0.0;
  for (int n = 0; n < N; ++n) {
    const size_t nh = static_cast<size_t>(n) * H + h;
    e = __dadd_rn(e, err[nh * dk + u]);
    l = __dadd_rn(l, static_cast<double>(is_kda ? logs[nh * dk + u] : logs[nh]));
  }
  esum[i] = e;
  lsum[i] = l;
}

// Low tier the selection measures E under: 0 the per-row quantizer, 1 the
// paper's groups of 32 with FP16 (s, z), 2 the same after the block-32
// transform; -1 if `lo` is not a low tier with a kernel here.
int select_tier(const damp_layout* lo, int d_k, int d_v) {
  if (!lo) return 0;
  if (lo->kind != DAMP_STATE_MIXED || lo->d_k != d_k || lo->d_v != d_v) return -1;
  if (layout_is_default(lo)) return 0;
  if (layout_is_paper(lo) && d_v <= 128 && d_v % 32 == 0) return lo->hadamard ? 2 : 1;
  return -1;
}

}  // namespace

int64_t select_scratch_doubles(int32_t N, int32_t H, int32_t d_k) {
  const int64_t hk = static_cast<int64_t>(H) * d_k;
  return static_cast<int64_t>(N) * hk + 2 * hk;
}

damp_status select_validate(const char* name, int32_t is_kda, int32_t N, int32_t H, int32_t d_k,
                            int32_t d_v, const float* states, const float* log_decay,
                            const damp_layout* lo, int32_t k_hi, double tau,
                            const int32_t* sel_out, const uint8_t* perm_out) {
  (void)is_kda;
  if (N <= 0 || H <= 0 || d_k <= 0 || d_k > 256 || d_v <= 0)
    return fail(DAMP_ERR_INVALID_ARG, "%s: bad sizes N=%d H=%d d_k=%d d_v=%d", name, N, H, d_k,
                d_v);
  if (k_hi < 0 || k_hi > d_k)
    return fail(DAMP_ERR_INVALID_ARG, "%s: k_hi = %d outside [0, %d]", name, k_hi, d_k);
  if (!(tau > 0.0)) return fail(DAMP_ERR_INVALID_ARG, "%s: tau must be > 0", name);
  if (!states || !log_decay || !perm_out || (k_hi > 0 && !sel_out))
    return fail(DAMP_ERR_INVALID_ARG, "%s: a required pointer is NULL", name);
  if (static_cast<int64_t>(H) * d_k > INT32_MAX)
    return fail(DAMP_ERR_INVALID_ARG, "%s: H * d_k too large", name);
  if (select_tier(lo, d_k, d_v) < 0)
    return fail(DAMP_ERR_UNSUPPORTED, "%s: Q_lo must be the per-row tier or the paper's UINT8 "
                "group tier (d_v <= 128, a multiple of 32) with d_k, d_v as given", name);
  return DAMP_OK;
}

damp_status select_run(const char* name, int32_t is_kda, int32_t N, int32_t H, int32_t d_k,
                       int32_t d_v, const float* states, const float* log_decay,
                       const damp_layout* lo, int32_t k_hi, double tau, int32_t* sel_out,
                       uint8_t* perm_out, double* score_out, double* scratch,
                       hipStream_t s) {
  const int64_t rows = static_cast<int64_t>(N) * H * d_k;
  const int64_t hk = static_cast<int64_t>(H) * d_k;
  double* d_err = scratch;
  double* d_esum = scratch + rows;
  double* d_lsum = d_esum + hk;
  const int tier = select_tier(lo, d_k, d_v);
  if (tier == 0) {
    hipLaunchKernelGGL(row_error_kernel, dim3(static_cast<unsigned>((rows + 255) / 256)),
                       dim3(256), 0, s, states, rows, d_v, d_err);
  } else {
    launch_row_errors_group(states, rows, d_v, tier == 2, d_err, s);
  }
  hipLaunchKernelGGL(sum_samples_kernel, dim3(static_cast<unsigned>((hk + 255) / 256)),
                     dim3(256), 0, s, d_err, log_decay, N, H, d_k, is_kda ? 1 : 0, d_esum,
                     d_lsum);
  damp_status st = check_launch(name);
  if (st != DAMP_OK) return st;
  // The per-channel sums reach the host a few heads at a time through a
  // fixed staging buffer, and the ranking works in fixed arrays (d_k <= 256),
  // so the host side allocates nothing either.
  constexpr int kStage = 4096;
  double stage[kStage];
  double score[256];
  int order[256];
  bool keep[256];
  const int per_copy = kStage / (2 * d_k);
  for (int h0 = 0; h0 < H; h0 += per_copy) {
    const int nh = std::min(per_copy, H - h0);
    const size_t n = static_cast<size_t>(nh) * d_k;
    const size_t off = static_cast<size_t>(h0) * d_k;
    hipError_t e = hipMemcpyAsync(stage, d_esum + off, n * sizeof(double),
                                  hipMemcpyDeviceToHost, s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(stage + n, d_lsum + off, n * sizeof(double), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail(DAMP_ERR_HIP, "%s: %s", name, hipGetErrorString(e));
    for (int h = h0; h < h0 + nh; ++h) {
      const double* esum = stage + static_cast<size_t>(h - h0) * d_k;
      const double* lsum = esum + n;
      for (int u = 0; u < d_k; ++u) {
        const double E = esum[u] / static_cast<double>(N);           // Eq. (8)
        const double a_eff = std::exp(lsum[u] / static_cast<double>(N));
        const double gap = 1.0 - a_eff * a_eff;
        const double P = 1.0 / (gap > tau ? gap : tau);              // Eq. (9)
        score[u] = E * P;                                              // C = E P
        if (score_out) score_out[static_cast<size_t>(h) * d_k + u] = score[u];
        order[u] = u;
        keep[u] = false;
      }
      std::sort(order, order + d_k, [&](int a, int b) {
        if (score[a] != score[b]) return score[a] > score[b];
        return a < b;
      });
      for (int i = 0; i < k_hi; ++i) keep[order[i]] = true;
      int p = 0, q = 0;
      for (int u = 0; u < d_k; ++u)
        if (keep[u]) {
          perm_out[static_cast<size_t>(h) * d_k + p++] = static_cast<uint8_t>(u);
          sel_out[static_cast<size_t>(h) * k_hi + q++] = u;
        }
      for (int u = 0; u < d_k; ++u)
        if (!keep[u]) perm_out[static_cast<size_t>(h) * d_k + p++] = static_cast<uint8_t>(u);
    }
  }
  return DAMP_OK;
}

}  // namespace damp

extern "C" damp_status damp_select_channels(int32_t is_kda, int32_t N, int32_t H, int32_t d_k,
                                            int32_t d_v, const float* states,
                                            const float* log_decay, const damp_layout* lo,
                                            int32_t k_hi, double tau, int32_t* sel_out,
                                            uint8_t* perm_out, double* score_out,
                                            void* stream) {
  using namespace damp;
  clear_error();
  const char* name = "damp_select_channels";
  damp_status st = select_validate(name, is_kda, N, H, d_k, d_v, states, log_decay, lo, k_hi,
                                   tau, sel_out, perm_out);
  if (st != DAMP_OK) return st;
  const size_t bytes = static_cast<size_t>(select_scratch_doubles(N, H, d_k)) * sizeof(double);
  double* scratch = nullptr;
  if (hipMalloc(&scratch, bytes) != hipSuccess)
    return fail(DAMP_ERR_HIP, "%s: hipMalloc of %zu bytes failed", name, bytes);
  st = select_run(name, is_kda, N, H, d_k, d_v, states, log_decay, lo, k_hi, tau, sel_out,
                  perm_out, score_out, scratch, as_stream(stream));
  // the stream was synchronised unless a launch failed; the free waits for the device
  (void)hipFree(scratch);
  return st;
}

// ---- damp_select_channels_noalloc: the same selection with its device
// scratch in a fixed array of the library, one copy per GPU (held until the
// process ends), instead of a hipMalloc per call.

static __device__ __align__(256) double
    scratch[DAMP_SELECT_NOALLOC_SCRATCH_BYTES / sizeof(double)];

namespace damp {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
double* g_scratch[kMaxDevices] = {};

// The device address of `scratch` on the GPU that runs stream s, looked up
// once per GPU with that GPU current. In host code the array's name stands
// for a host-side shadow, never for device memory, so kernels only ever get
// this address.
damp_status scratch_for(hipStream_t s, double** out, const char* name) {
  int dev = 0;
  hipError_t e = s ? hipStreamGetDevice(s, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return fail(DAMP_ERR_HIP, "%s: %s", name, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(DAMP_ERR_INVALID_ARG, "%s: device %d beyond the %d supported", name, dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    int cur = 0;
    e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    void* p = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p)
      return fail(DAMP_ERR_HIP, "%s: device address of the scratch array: %s", name,
                  e != hipSuccess ? hipGetErrorString(e) : "null");
    g_scratch[dev] = static_cast<double*>(p);
  }
  *out = g_scratch[dev];
  return DAMP_OK;
}

}  // namespace
}  // namespace damp

extern "C" damp_status damp_select_channels_noalloc(int32_t is_kda, int32_t N, int32_t H,
                                                    int32_t d_k, int32_t d_v,
                                                    const float* states,
                                                    const float* log_decay,
                                                    const damp_layout* lo, int32_t k_hi,
                                                    double tau, int32_t* sel_out,
                                                    uint8_t* perm_out, double* score_out,
                                                    void* stream) {
  using namespace damp;
  clear_error();
  const char* name = "damp_select_channels_noalloc";
  damp_status st = select_validate(name, is_kda, N, H, d_k, d_v, states, log_decay, lo, k_hi,
                                   tau, sel_out, perm_out);
  if (st != DAMP_OK) return st;
  const int64_t need = select_scratch_doubles(N, H, d_k);
  constexpr int64_t kMax = DAMP_SELECT_NOALLOC_SCRATCH_BYTES / sizeof(double);
  if (need > kMax)
    return fail(DAMP_ERR_INVALID_ARG, "%s: (N + 2) * H * d_k = %lld doubles exceed the %lld of "
                "the fixed scratch (%d bytes)", name, static_cast<long long>(need),
                static_cast<long long>(kMax), DAMP_SELECT_NOALLOC_SCRATCH_BYTES);
  hipStream_t s = as_stream(stream);
  double* buf = nullptr;
  st = scratch_for(s, &buf, name);
  if (st != DAMP_OK) return st;
  return select_run(name, is_kda, N, H, d_k, d_v, states, log_decay, lo, k_hi, tau, sel_out,
                    perm_out, score_out, buf, s);
}
