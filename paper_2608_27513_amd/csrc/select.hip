// Offline selection of the protected key channels (section 5.1 Eq. (8)-(10),
// App. A.2 Eq. (14)-(15), Alg. 1 of App. A.4).
//
// The device pass computes, for every calibration row S_n[h, u, :], the
// squared reconstruction error under the low-tier quantizer of Eq. (3). Each
// row is handled by one thread in ascending column order with IEEE
// operations only (correctly rounded fp32 division, no contraction, double
// accumulation), so the per-row sums are reproducible bit for bit. The host
// then averages over samples in ascending order, forms the geometric-mean
// decay, the persistence of Eq. (9), C = E P, and the top-k_hi partition.
#include <algorithm>
#include <cfloat>
#include <cmath>
#include <vector>

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

}  // namespace
}  // namespace damp

extern "C" damp_status damp_select_channels(int32_t is_kda, int32_t N, int32_t H, int32_t d_k,
                                            int32_t d_v, const float* states,
                                            const float* log_decay, int32_t k_hi, double tau,
                                            int32_t* sel_out, uint8_t* perm_out,
                                            double* score_out, void* stream) {
  using namespace damp;
  clear_error();
  if (N <= 0 || H <= 0 || d_k <= 0 || d_k > 256 || d_v <= 0)
    return fail(DAMP_ERR_INVALID_ARG, "damp_select_channels: bad sizes N=%d H=%d d_k=%d d_v=%d",
                N, H, d_k, d_v);
  if (k_hi < 0 || k_hi > d_k)
    return fail(DAMP_ERR_INVALID_ARG, "damp_select_channels: k_hi = %d outside [0, %d]", k_hi,
                d_k);
  if (!(tau > 0.0)) return fail(DAMP_ERR_INVALID_ARG, "damp_select_channels: tau must be > 0");
  if (!states || !log_decay || !perm_out || (k_hi > 0 && !sel_out))
    return fail(DAMP_ERR_INVALID_ARG, "damp_select_channels: a required pointer is NULL");

  const int64_t rows = static_cast<int64_t>(N) * H * d_k;
  const int64_t nlog = static_cast<int64_t>(N) * H * (is_kda ? d_k : 1);
  hipStream_t s = as_stream(stream);
  double* d_err = nullptr;
  if (hipMalloc(&d_err, rows * sizeof(double)) != hipSuccess)
    return fail(DAMP_ERR_HIP, "damp_select_channels: hipMalloc of %lld bytes failed",
                static_cast<long long>(rows * sizeof(double)));
  const int64_t blocks = (rows + 255) / 256;
  hipLaunchKernelGGL(row_error_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s,
                     states, rows, d_v, d_err);
  std::vector<double> err(rows);
  std::vector<float> logs(nlog);
  damp_status st = check_launch("damp_select_channels");
  if (st == DAMP_OK) {
    hipError_t e = hipMemcpyAsync(err.data(), d_err, rows * sizeof(double),
                                  hipMemcpyDeviceToHost, s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(logs.data(), log_decay, nlog * sizeof(float), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess)
      st = fail(DAMP_ERR_HIP, "damp_select_channels: %s", hipGetErrorString(e));
  }
  (void)hipFree(d_err);
  if (st != DAMP_OK) return st;

  std::vector<double> score(d_k);
  std::vector<int> order(d_k);
  std::vector<char> keep(d_k);
  for (int h = 0; h < H; ++h) {
    for (int u = 0; u < d_k; ++u) {
      double esum = 0.0, lsum = 0.0;
      for (int n = 0; n < N; ++n) {
        esum = esum + err[(static_cast<size_t>(n) * H + h) * d_k + u];
        lsum = lsum + static_cast<double>(
                          is_kda ? logs[(static_cast<size_t>(n) * H + h) * d_k + u]
                                 : logs[static_cast<size_t>(n) * H + h]);
      }
      const double E = esum / static_cast<double>(N);           // Eq. (8)
      const double a_eff = std::exp(lsum / static_cast<double>(N));
      const double gap = 1.0 - a_eff * a_eff;
      const double P = 1.0 / (gap > tau ? gap : tau);           // Eq. (9)
      score[u] = E * P;                                          // C = E P
      if (score_out) score_out[static_cast<size_t>(h) * d_k + u] = score[u];
      order[u] = u;
    }
    std::sort(order.begin(), order.end(), [&](int a, int b) {
      if (score[a] != score[b]) return score[a] > score[b];
      return a < b;
    });
    std::fill(keep.begin(), keep.end(), 0);
    for (int i = 0; i < k_hi; ++i) keep[order[i]] = 1;
    int p = 0, q = 0;
    for (int u = 0; u < d_k; ++u)
      if (keep[u]) {
        perm_out[static_cast<size_t>(h) * d_k + p++] = static_cast<uint8_t>(u);
        sel_out[static_cast<size_t>(h) * k_hi + q++] = u;
      }
    for (int u = 0; u < d_k; ++u)
      if (!keep[u]) perm_out[static_cast<size_t>(h) * d_k + p++] = static_cast<uint8_t>(u);
  }
  return DAMP_OK;
}
