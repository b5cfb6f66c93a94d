// CKKS decoding on the device: evaluation-form plaintexts -> slot vectors, the
// inverse of the device encoder (encode_gpu.hip).
//
// Slot j of a plaintext with integer coefficients m is z_j = m(zeta^(e_j)) /
// Delta, zeta = exp(i pi / N), e_j = 5^j mod 2N.  With e_j = 2 p_j + 1,
//     m(zeta^(e_j)) = sum_k (m_k zeta^k) exp(2 pi i k p_j / N),
// i.e. the unnormalised inverse DFT of the twisted coefficients m_k zeta^k read
// at p_j.  Per plaintext:
//   1. inverse NTT of a copy of the limbs (canonical residues, coefficient
//      form);
//   2. k_dec_crt: the centred integer m_k from its residues by a mixed-radix
//      CRT with balanced digits (Garner's method: v_0 = [y_0], v_i =
//      [(...((y_i - v_0) q_0^-1 - v_1) q_1^-1 ...) q_(i-1)^-1]_(q_i), each in
//      (-q_i/2, q_i/2]), so m_k = v_0 + q_0 (v_1 + q_1 (v_2 + ...)) exactly; the
//      Horner evaluation in fp64 rounds once per level; then the twist;
//   3. log2 N radix-2 Stockham stages (out of place, natural order in and
//      out), the inverse transform's sign;
//   4. k_dec_gather: z_j = v[p_j] / Delta through the encoder's inverse slot
//      table.
// Every twiddle is an entry of the encoder's table T[k] = exp(-i pi k / N):
// the twist zeta^k = conj(T[k]), the stage twiddle exp(i pi t / Ns) =
// conj(T[t N / Ns]).
#include <algorithm>

#include "fesc_internal.hpp"
#include "ops.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ double2 cmul(double2 a, double2 b) {
  return double2{a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x};
}

// Coefficient k = blockIdx.x * 256 + t of plaintext blockIdx.y: residues
// y_i = res[b][i][k] (canonical, i < level) -> centred m_k (fp64) * zeta^k.
__global__ __launch_bounds__(kThreads) void k_dec_crt(const uint64_t* __restrict__ res,
                                                      uint32_t level, uint32_t L, uint32_t n,
                                                      const PrimeK* __restrict__ pk,
                                                      const double2* __restrict__ garner,
                                                      const double2* __restrict__ T,
                                                      double2* __restrict__ out) {
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x, b = blockIdx.y;
  if (k >= n) return;
  const uint64_t* r = res + (size_t)b * level * n + k;
  double v[FESC_MAX_PRIMES];
  for (uint32_t i = 0; i < level; ++i) {
    const PrimeK P = pk[i];
    double t = u2d(r[(size_t)i * n]);
    const double2* gi = garner + (size_t)i * L;
    for (uint32_t j = 0; j < i; ++j) {  // t = (t - v_j) q_j^-1 mod q_i
      const double2 w = gi[j];
      t = red_bal(mm_shoup(red_bal(t - v[j], P.q, P.qinv), w.x, w.y, P.q), P.q, P.qinv);
    }
    v[i] = center(red_full(t, P.q, P.qinv), P.q);
  }
  double m = v[level - 1];
  for (uint32_t i = level - 1; i-- > 0;) m = v[i] + pk[i].q * m;
  const double2 tw = T[k];  // zeta^-k
  out[(size_t)b * n + k] = double2{m * tw.x, -m * tw.y};
}

// One radix-2 Stockham stage of the inverse transform (half size ns).
__global__ __launch_bounds__(kThreads) void k_dec_fft_stage(const double2* __restrict__ in,
                                                            double2* __restrict__ out, uint32_t n,
                                                            uint32_t ns, uint32_t log_ns,
                                                            uint32_t log_n,
                                                            const double2* __restrict__ T) {
  const uint32_t j = blockIdx.x * kThreads + threadIdx.x, b = blockIdx.y;
  if (j >= n / 2) return;
  const double2* x = in + (size_t)b * n;
  double2* y = out + (size_t)b * n;
  const uint32_t t = j & (ns - 1);
  const double2 c = T[(size_t)t << (log_n - log_ns)];  // exp(-i pi t / ns)
  const double2 w{c.x, -c.y};
  const double2 u = x[j], v = cmul(x[j + n / 2], w);
  const uint32_t d = ((j - t) << 1) + t;
  y[d] = double2{u.x + v.x, u.y + v.y};
  y[d + ns] = double2{u.x - v.x, u.y - v.y};
}

// z[b][j] = v[b][p] / Delta for the transform position p of slot j.
__global__ __launch_bounds__(kThreads) void k_dec_gather(const double2* __restrict__ v,
                                                         const int32_t* __restrict__ inv,
                                                         double2* __restrict__ z, uint32_t n,
                                                         double rdelta) {
  const uint32_t p = blockIdx.x * kThreads + threadIdx.x, b = blockIdx.y;
  if (p >= n) return;
  const int32_t j = inv[p];
  if (j < 0) return;
  const double2 x = v[(size_t)b * n + p];
  z[(size_t)b * (n / 2) + (uint32_t)j] = double2{x.x * rdelta, x.y * rdelta};
}

}  // namespace

// Decodes `count` plaintexts pt[count][level][N] into z[count][N/2], as many
// per round as fit in the scratch ciphertext slots (limbs, then two complex
// buffers of N per plaintext).
int op_decode_plain(Context* c, const uint64_t* pt, uint32_t count, uint32_t level, double scale,
                    double2* z, uint64_t* slots, uint32_t nslots, hipStream_t s) {
  const uint32_t n = c->n;
  const size_t per = (size_t)(level + 4) * n, room = (size_t)2 * c->L * n * nslots;
  const uint32_t cap = (uint32_t)std::min<size_t>(room / per, 65535);  // grid y limit
  if (cap == 0) return fail(FESC_ERR_ARG, "decode scratch too small");
  const double rdelta = 1.0 / scale;
  for (uint32_t b0 = 0; b0 < count; b0 += cap) {
    const uint32_t m = std::min(cap, count - b0);
    uint64_t* limbs = slots;                                              // [m][level][N]
    double2* A = reinterpret_cast<double2*>(slots + (size_t)m * level * n);  // [m][N]
    double2* B = A + (size_t)m * n;                                        // [m][N]
    if (int rc = hip_check(hipMemcpyAsync(limbs, pt + (size_t)b0 * level * n,
                                          (size_t)m * level * n * 8, hipMemcpyDeviceToDevice, s),
                           "decode copy"))
      return rc;
    if (int rc = hip_check(launch_ntt(c, limbs, m, (size_t)level * n, level, n, 0, true, s),
                           "decode iNTT"))
      return rc;
    const dim3 g(n / kThreads, m);
    k_dec_crt<<<g, kThreads, 0, s>>>(limbs, level, c->L, n, c->d_pk, c->d_garner, c->d_enc_tw,
                                     A);
    if (int rc = hip_check(hipGetLastError(), "k_dec_crt")) return rc;
    double2 *src = A, *dst = B;
    for (uint32_t log_ns = 0; log_ns < c->log_n; ++log_ns) {
      k_dec_fft_stage<<<dim3(n / 2 / kThreads, m), kThreads, 0, s>>>(src, dst, n, 1u << log_ns,
                                                                      log_ns, c->log_n,
                                                                      c->d_enc_tw);
      if (int rc = hip_check(hipGetLastError(), "k_dec_fft_stage")) return rc;
      std::swap(src, dst);
    }
    k_dec_gather<<<g, kThreads, 0, s>>>(src, c->d_enc_inv, z + (size_t)b0 * (n / 2), n, rdelta);
    if (int rc = hip_check(hipGetLastError(), "k_dec_gather")) return rc;
  }
  return FESC_OK;
}

}  // namespace fesc
