// Host-only part of libzo: the per-probe coefficient function of 1.5-SPSA and status text.
//
// Curvature along probe k (section 4.1, Eq. 3), its alpha-saturated weight (Eq. 4) and the
// coefficient that zo_update multiplies by lr (section 4.2, Eq. 5/6; Algorithm 1's gamma_k
// when lr = eps). Compiled with -ffp-contract=off and without fast-math so that every
// operation below is one IEEE float64 operation in the order written.

#include <cmath>
#include <cstdint>

#include "zo.h"

extern "C" {

int zo_probe_coeffs_ex(const double* L_plus, const double* L_minus, uint32_t K, double L_clean, double eps,
                       double alpha, double lambda_reg, float* c_out, double* c64_out, double* curv_out,
                       double* w_out) {
  if (L_plus == nullptr || L_minus == nullptr) return ZO_ERR_NULL;
  if (K == 0) return ZO_ERR_ARG;
  if (!std::isfinite(L_clean) || !std::isfinite(eps) || !std::isfinite(alpha) || !std::isfinite(lambda_reg))
    return ZO_ERR_NONFINITE;
  for (uint32_t k = 0; k < K; ++k)
    if (!std::isfinite(L_plus[k]) || !std::isfinite(L_minus[k])) return ZO_ERR_NONFINITE;
  if (!(eps > 0.0) || !(alpha >= 0.0 && alpha <= 1.0) || !(lambda_reg > 0.0)) return ZO_ERR_ARG;

  const double two_k_eps = (2.0 * static_cast<double>(K)) * eps;
  for (uint32_t k = 0; k < K; ++k) {
    const double d2 = (L_plus[k] - 2.0 * L_clean) + L_minus[k];
    const double chat = d2 / (eps * eps);
    const double a = std::pow(std::fabs(chat), alpha);
    const double den = a > lambda_reg ? a : lambda_reg;
    const double w = 1.0 / den;
    const double c64 = ((L_plus[k] - L_minus[k]) * w) / two_k_eps;
    if (c_out) c_out[k] = static_cast<float>(c64);
    if (c64_out) c64_out[k] = c64;
    if (curv_out) curv_out[k] = chat;
    if (w_out) w_out[k] = w;
  }
  return ZO_OK;
}

int zo_probe_coeffs(const double* L_plus, const double* L_minus, uint32_t K, double L_clean, double eps,
                    float* c_out) {
  if (c_out == nullptr) return ZO_ERR_NULL;
  return zo_probe_coeffs_ex(L_plus, L_minus, K, L_clean, eps, 0.1, 1.0, c_out, nullptr, nullptr, nullptr);
}

const char* zo_strerror(int status) {
  switch (status) {
    case ZO_OK: return "success";
    case ZO_ERR_NULL: return "a required pointer is NULL";
    case ZO_ERR_ARG: return "invalid argument (dtype, alignment, probe count or index range)";
    case ZO_ERR_NONFINITE: return "non-finite eps, lr, loss or coefficient";
    case ZO_ERR_HIP: return "the HIP runtime refused the launch";
    default: return "unknown status";
  }
}

const char* zo_version(void) { return "libzo 0.1.0 (gfx950, Philox4x32-10 probes)"; }

}  // extern "C"
