// Host-side CKKS slot encoder (offline plaintext preparation; not on the
// device hot path).  Slot j is the evaluation at zeta^(5^j mod 2N),
// zeta = exp(i pi / N); the real plaintext polynomial m with
// m(zeta^(5^j)) = Delta z_j and m(zeta^(-5^j)) = Delta conj(z_j) is
//     m_k = (1/N) zeta^-k sum_u Z[2u+1] w^(-u k),   w = zeta^2,
// one length-N complex FFT over the odd exponents, rounded half away from
// zero.
#include <cmath>
#include <complex>
#include <cstdint>
#include <vector>

#include "fesc_internal.hpp"

namespace fesc {

namespace {

using cd = std::complex<double>;

// in-place forward DFT, X[k] = sum_u x[u] exp(-2 pi i u k / N)
void fft(std::vector<cd>& x, uint32_t log_n) {
  const uint32_t n = 1u << log_n;
  for (uint32_t i = 0; i < n; ++i) {
    const uint32_t r = __builtin_bitreverse32(i) >> (32 - log_n);
    if (i < r) std::swap(x[i], x[r]);
  }
  std::vector<cd> root(n / 2);
  for (uint32_t k = 0; k < n / 2; ++k) {
    const double ang = -2.0 * M_PI * (double)k / (double)n;
    root[k] = cd(std::cos(ang), std::sin(ang));
  }
  for (uint32_t len = 2; len <= n; len <<= 1) {
    const uint32_t step = n / len;
    for (uint32_t s = 0; s < n; s += len)
      for (uint32_t j = 0; j < len / 2; ++j) {
        const cd u = x[s + j], v = x[s + j + len / 2] * root[j * step];
        x[s + j] = u + v;
        x[s + j + len / 2] = u - v;
      }
  }
}

}  // namespace

int encode(uint32_t log_n, const double* re, const double* im, double scale, int64_t* out) {
  if (!re || !out || log_n < 2 || log_n > 20) return fail(FESC_ERR_ARG, "bad encode arguments");
  const uint32_t n = 1u << log_n, two_n = 2 * n;
  std::vector<cd> y(n, cd(0.0, 0.0));
  uint64_t e = 1;
  for (uint32_t j = 0; j < n / 2; ++j) {
    const cd z(re[j], im ? im[j] : 0.0);
    y[(e - 1) / 2] = z;
    y[(two_n - e - 1) / 2] = std::conj(z);
    e = e * 5 % two_n;
  }
  fft(y, log_n);
  for (uint32_t k = 0; k < n; ++k) {
    const double ang = -M_PI * (double)k / (double)n;
    const double v = (y[k] * cd(std::cos(ang), std::sin(ang))).real() / (double)n * scale;
    const double r = std::round(v);  // half away from zero
    if (!(std::fabs(r) < 9.2233720368547758e18))
      return fail(FESC_ERR_ARG, "encoded coefficient does not fit in int64");
    out[k] = (int64_t)r;
  }
  return FESC_OK;
}

}  // namespace fesc
