// Ciphertext-level elementwise kernels (evaluation form): add / sub, plaintext
// product and addition, monomial product, Galois permutation (key
// generation), lifting of signed integer coefficients, the HEConv
// accumulation, and the combine steps of key generation and encryption.  (The
// tensor of a relinearised product is formed inside the key switch; the
// rescale runs in the transforms' passes.)
//
// Ciphertext layout [l][2][N]: row r = 2*i + t holds component t of limb i,
// so the prime of row r is r >> 1.
#include "fesc_internal.hpp"
#include "ops.hpp"
#include "seedkey.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ double ld(const uint64_t* p) { return u2d(*p); }
__device__ __forceinline__ void st(uint64_t* p, double v, double q, double qinv) {
  *p = to_res(v, q, qinv);
}

// ---------------------------------------------------------------- binary

// op 0: a + b, op 1: a - b, op 2: a * b (all rows), prime of row r = r >> shift
__global__ __launch_bounds__(kThreads) void k_binary(const uint64_t* __restrict__ a,
                                                     const uint64_t* __restrict__ b,
                                                     uint64_t* out, uint32_t n, uint32_t shift,
                                                     int op, const PrimeK* __restrict__ pk) {
  const uint32_t r = blockIdx.y;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const PrimeK P = pk[r >> shift];
  const size_t o = (size_t)r * n + k;
  const double x = ld(a + o), y = ld(b + o);
  double v = op == 0 ? x + y : op == 1 ? x - y : mm_var(x, y, P.q, P.qinv);
  st(out + o, v, P.q, P.qinv);
}

// out[i][t] = ct[i][t] * pt[i]
__global__ __launch_bounds__(kThreads) void k_mul_plain(const uint64_t* ct,
                                                        const uint64_t* __restrict__ pt,
                                                        uint64_t* out, uint32_t n,
                                                        const PrimeK* __restrict__ pk) {
  const uint32_t i = blockIdx.y;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const PrimeK P = pk[i];
  const double w = ld(pt + (size_t)i * n + k);
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const size_t o = ((size_t)2 * i + t) * n + k;
    st(out + o, mm_var(ld(ct + o), w, P.q, P.qinv), P.q, P.qinv);
  }
}

// out = (c0 + pt, c1); out may alias ct.
__global__ __launch_bounds__(kThreads) void k_add_plain(const uint64_t* ct,
                                                        const uint64_t* __restrict__ pt,
                                                        uint64_t* out, uint32_t n,
                                                        const PrimeK* __restrict__ pk) {
  const uint32_t i = blockIdx.y;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const PrimeK P = pk[i];
  const size_t o = (size_t)2 * i * n + k;
  st(out + o, ld(ct + o) + ld(pt + (size_t)i * n + k), P.q, P.qinv);
  out[o + n] = ct[o + n];
}

// HEConv accumulation: acc[i][t] = sum_r mask_r[i] rot_r[i][t] (+ for t = 0:
// (q_{l-1} mod q_i) bias[i], so that the following rescale adds the bias
// exactly).  Partial sums are reduced every four terms.
__global__ __launch_bounds__(kThreads) void k_conv_acc(ConvTable tab, const uint64_t* bias,
                                                       uint64_t* acc, uint32_t n, uint32_t level,
                                                       const PrimeK* __restrict__ pk) {
  const uint32_t i = blockIdx.y;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const PrimeK P = pk[i];
  const size_t o0 = (size_t)2 * i * n + k, o1 = o0 + n, op = (size_t)i * n + k;
  double a0 = 0.0, a1 = 0.0;
  for (uint32_t r = 0; r < tab.taps; ++r) {
    const double w = ld(tab.mask[r] + op);
    a0 += mm_var(ld(tab.rot[r] + o0), w, P.q, P.qinv);
    a1 += mm_var(ld(tab.rot[r] + o1), w, P.q, P.qinv);
    if ((r & 3) == 3) {
      a0 = red_bal(a0, P.q, P.qinv);
      a1 = red_bal(a1, P.q, P.qinv);
    }
  }
  if (bias) {
    const double ql = pk[level - 1].q;
    const double qlm = ql >= P.q ? ql - P.q : ql;  // all primes within a factor 2
    a0 += mm_var(ld(bias + op), qlm, P.q, P.qinv);
  }
  st(acc + o0, a0, P.q, P.qinv);
  st(acc + o1, a1, P.q, P.qinv);
}

// multiplication by X^m: the evaluation at psi^(2 brv(j) + 1) scales by
// psi^e, e = (2 brv(j) + 1) m mod 2N; psi^e = tw[brv(e)] for e < N and
// -tw[brv(e - N)] otherwise (tw = forward twiddle table).
// Evaluation of X^m at the point of index k (prime i): the value psi^e,
// e = (2 brv(k) + 1) m mod 2N, as a table twiddle and a sign (psi^N = -1).
__device__ __forceinline__ double2 monomial_w(uint32_t k, uint32_t m, uint32_t log_n, uint32_t i,
                                              const double2* __restrict__ twf, bool* neg) {
  const uint32_t n = 1u << log_n;
  const uint32_t b = __builtin_bitreverse32(k) >> (32 - log_n);
  const uint32_t e = ((2u * b + 1u) * m) & (2u * n - 1u);
  *neg = e >= n;
  const uint32_t eb = __builtin_bitreverse32(*neg ? e - n : e) >> (32 - log_n);
  return twf[(size_t)i * n + eb];
}

__global__ __launch_bounds__(kThreads) void k_monomial(const uint64_t* in, uint64_t* out,
                                                       uint32_t log_n, uint32_t m,
                                                       const PrimeK* __restrict__ pk,
                                                       const double2* __restrict__ twf) {
  const uint32_t n = 1u << log_n;
  const uint32_t r = blockIdx.y, i = r >> 1;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const PrimeK P = pk[i];
  bool neg;
  const double2 w = monomial_w(k, m, log_n, i, twf, &neg);
  const size_t o = (size_t)r * n + k;
  double v = mm_shoup(ld(in + o), w.x, w.y, P.q);
  st(out + o, neg ? -v : v, P.q, P.qinv);
}

// Pair blockIdx.z of the table, row blockIdx.y (limb r / 2, component r % 2).
// X^(N/2) and X^(3N/2) evaluate to -+ psi^(N/2) at every point, so the
// monomial is one Shoup product and a sign.
__global__ __launch_bounds__(kThreads) void k_pair(PairTable tab, bool split, uint32_t log_n,
                                                   const PrimeK* __restrict__ pk,
                                                   const double2* __restrict__ twf) {
  const uint32_t n = 1u << log_n;
  const uint32_t r = blockIdx.y, i = r >> 1, j = blockIdx.z;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const PrimeK P = pk[i];
  const size_t o = (size_t)r * n + k;
  bool neg;
  if (!split) {
    const double2 w = monomial_w(k, n / 2, log_n, i, twf, &neg);
    const double v = mm_shoup(ld(tab.y[j] + o), w.x, w.y, P.q);
    st(tab.x[j] + o, ld(tab.x[j] + o) + (neg ? -v : v), P.q, P.qinv);
  } else {
    const double a = ld(tab.x[j] + o), b = ld(tab.y[j] + o);
    const double2 w = monomial_w(k, 3 * n / 2, log_n, i, twf, &neg);
    const double v = mm_shoup(a - b, w.x, w.y, P.q);
    st(tab.first[j] + o, a + b, P.q, P.qinv);
    st(tab.second[j] + o, neg ? -v : v, P.q, P.qinv);
  }
}

// out[row][k] = in[row][galois_src(k)]; rows share one prime list (prime of
// row r = prime0 + r).  out must not alias in.
__global__ __launch_bounds__(kThreads) void k_galois(const uint64_t* __restrict__ in,
                                                     uint64_t* __restrict__ out,
                                                     uint32_t log_n, uint32_t g) {
  const uint32_t n = 1u << log_n;
  const uint32_t r = blockIdx.y;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  out[(size_t)r * n + k] = in[(size_t)r * n + galois_src(k, g, log_n)];
}

// out[r][k] = x[k] mod prime(r) for signed coefficients; x is int64 (or int8
// when x8 != null).  Row r uses prime prime0 + r for r < split, else
// prime1 + (r - split).
__global__ __launch_bounds__(kThreads) void k_lift(const int64_t* __restrict__ x,
                                                   const int8_t* __restrict__ x8,
                                                   uint64_t* __restrict__ out, uint32_t n,
                                                   uint32_t prime0, uint32_t split,
                                                   uint32_t prime1,
                                                   const PrimeK* __restrict__ pk) {
  const uint32_t r = blockIdx.y;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const PrimeK P = pk[r < split ? prime0 + r : prime1 + (r - split)];
  const int64_t v = x8 ? (int64_t)x8[k] : x[k];
  // exact: |v| < 2^63 -> split into hi * 2^32 + lo, reduce each part
  const double hi = (double)(int32_t)(v >> 32);
  const double lo = (double)(uint32_t)(v & 0xffffffffu);
  const double two32 = red_full(4294967296.0, P.q, P.qinv);
  const double t = mm_var(red_full(hi, P.q, P.qinv), two32, P.q, P.qinv);
  st(out + (size_t)r * n + k, t + lo, P.q, P.qinv);
}

// key[j][i][0] = -a*s + e + (i in digit j ? [P]_{q_i} s_from : 0), key[j][i][1] = a.
// a: [dnum][E][N], e_ntt: [dnum][E][N], s, s_from: [E][N]; E = L + alpha rows.
__global__ __launch_bounds__(kThreads) void k_keygen(const uint64_t* __restrict__ a,
                                                     const uint64_t* __restrict__ e_ntt,
                                                     const uint64_t* __restrict__ s,
                                                     const uint64_t* __restrict__ s_from,
                                                     uint64_t* __restrict__ key, uint32_t n,
                                                     uint32_t L, uint32_t alpha,
                                                     const double2* __restrict__ pmod,
                                                     const PrimeK* __restrict__ pk, KeySeed sd) {
  const uint32_t i = blockIdx.y, j = blockIdx.z, E = L + alpha;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (sd.seeded && blockIdx.x == 0 && i == 0 && j == 0 && threadIdx.x < kSeedHeaderWords)
    key[threadIdx.x] = threadIdx.x == 0 ? sd.s0 : threadIdx.x == 1 ? sd.s1
                     : threadIdx.x == 2 ? sd.elt : 0;
  if (k >= n) return;
  const PrimeK P = pk[i];
  const size_t oj = ((size_t)j * E + i) * n + k;
  double av;
  uint64_t au;
  if (sd.seeded) {  // the uniform half regenerated from the seed
    uint64_t blk[3] = {0, 0, 0};
    seeded_key_block(blk, k, i, j / 3, sd.elt, sd.s0, sd.s1, sd.dnum, P);
    au = blk[j % 3];
  } else {
    au = a[oj];
  }
  av = u2d(au);
  double b = ld(e_ntt + oj) - mm_var(av, ld(s + (size_t)i * n + k), P.q, P.qinv);
  if (i < L && i >= j * alpha && i < (j + 1) * alpha) {
    const double2 pm = pmod[i];
    b += mm_shoup(ld(s_from + (size_t)i * n + k), pm.x, pm.y, P.q);
  }
  if (sd.seeded) {  // compact layout: header, then b only
    st(key + kSeedHeaderWords + oj, b, P.q, P.qinv);
    return;
  }
  const size_t ok = (((size_t)j * E + i) * 2) * n + k;
  st(key + ok, b, P.q, P.qinv);
  key[ok + n] = au;
}

// Full layout [dnum][L+alpha][2][N] of a compact seed-expanded key: b copied,
// a regenerated (one generator block per thread: digits 3*blockIdx.z ..).
__global__ __launch_bounds__(kThreads) void k_key_expand(const uint64_t* __restrict__ compact,
                                                         uint64_t* __restrict__ full, uint32_t n,
                                                         uint32_t E, uint32_t dnum,
                                                         const PrimeK* __restrict__ pk) {
  const uint32_t i = blockIdx.y, c = blockIdx.z;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const PrimeK P = pk[i];
  uint64_t blk[3] = {0, 0, 0};
  seeded_key_block(blk, k, i, c, compact[2], compact[0], compact[1], dnum, P);
  for (uint32_t t = 0; t < 3 && 3 * c + t < dnum; ++t) {
    const uint32_t j = 3 * c + t;
    const size_t ok = (((size_t)j * E + i) * 2) * n + k;
    full[ok] = compact[kSeedHeaderWords + ((size_t)j * E + i) * n + k];
    full[ok + n] = blk[t];
  }
}

// ct[i][0] = -a*s + me, ct[i][1] = a
__global__ __launch_bounds__(kThreads) void k_encrypt(const uint64_t* __restrict__ a,
                                                      const uint64_t* __restrict__ s,
                                                      const uint64_t* __restrict__ me,
                                                      uint64_t* __restrict__ ct, uint32_t n,
                                                      const PrimeK* __restrict__ pk) {
  const uint32_t i = blockIdx.y;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const PrimeK P = pk[i];
  const size_t o = (size_t)i * n + k;
  const double av = ld(a + o);
  st(ct + 2 * (size_t)i * n + k, ld(me + o) - mm_var(av, ld(s + o), P.q, P.qinv), P.q, P.qinv);
  ct[(2 * (size_t)i + 1) * n + k] = a[o];
}

inline dim3 grid_rows(uint32_t n, uint32_t rows, uint32_t z = 1) {
  return dim3((n + kThreads - 1) / kThreads, rows, z);
}

}  // namespace

hipError_t k_binary_launch(const Context* c, const uint64_t* a, const uint64_t* b, uint64_t* out,
                           uint32_t rows, uint32_t shift, int op, hipStream_t s) {
  hipLaunchKernelGGL(k_binary, grid_rows(c->n, rows), dim3(kThreads), 0, s, a, b, out, c->n,
                     shift, op, c->d_pk);
  return hipGetLastError();
}

hipError_t k_mul_plain_launch(const Context* c, const uint64_t* ct, const uint64_t* pt,
                              uint64_t* out, uint32_t level, hipStream_t s) {
  hipLaunchKernelGGL(k_mul_plain, grid_rows(c->n, level), dim3(kThreads), 0, s, ct, pt, out,
                     c->n, c->d_pk);
  return hipGetLastError();
}

hipError_t k_add_plain_launch(const Context* c, const uint64_t* ct, const uint64_t* pt,
                              uint64_t* out, uint32_t level, hipStream_t s) {
  hipLaunchKernelGGL(k_add_plain, grid_rows(c->n, level), dim3(kThreads), 0, s, ct, pt, out,
                     c->n, c->d_pk);
  return hipGetLastError();
}

hipError_t k_conv_acc_launch(const Context* c, const ConvTable& tab, const uint64_t* bias,
                             uint64_t* acc, uint32_t level, hipStream_t s) {
  hipLaunchKernelGGL(k_conv_acc, grid_rows(c->n, level), dim3(kThreads), 0, s, tab, bias, acc,
                     c->n, level, c->d_pk);
  return hipGetLastError();
}

hipError_t k_monomial_launch(const Context* c, const uint64_t* in, uint64_t* out,
                             uint32_t level, uint32_t m, hipStream_t s) {
  hipLaunchKernelGGL(k_monomial, grid_rows(c->n, 2 * level), dim3(kThreads), 0, s, in, out,
                     c->log_n, m, c->d_pk, c->d_tw_fwd);
  return hipGetLastError();
}

hipError_t k_pair_launch(const Context* c, const PairTable& tab, uint32_t count, bool split,
                         uint32_t level, hipStream_t s) {
  if (count == 0) return hipSuccess;
  if (count > kPairBatch) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_pair, grid_rows(c->n, 2 * level, count), dim3(kThreads), 0, s, tab, split,
                     c->log_n, c->d_pk, c->d_tw_fwd);
  return hipGetLastError();
}

hipError_t k_galois_launch(const Context* c, const uint64_t* in, uint64_t* out, uint32_t rows,
                           uint32_t g, hipStream_t s) {
  hipLaunchKernelGGL(k_galois, grid_rows(c->n, rows), dim3(kThreads), 0, s, in, out, c->log_n,
                     g);
  return hipGetLastError();
}

hipError_t k_lift_launch(const Context* c, const int64_t* x, const int8_t* x8, uint64_t* out,
                         uint32_t rows, uint32_t prime0, uint32_t split, uint32_t prime1,
                         hipStream_t s) {
  hipLaunchKernelGGL(k_lift, grid_rows(c->n, rows), dim3(kThreads), 0, s, x, x8, out, c->n,
                     prime0, split, prime1, c->d_pk);
  return hipGetLastError();
}

hipError_t k_keygen_launch(const Context* c, const uint64_t* a, const uint64_t* e_ntt,
                           const uint64_t* s, const uint64_t* s_from, uint64_t* key,
                           const double2* pmod, const KeySeed& sd, hipStream_t st) {
  hipLaunchKernelGGL(k_keygen, grid_rows(c->n, c->L + c->alpha, c->dnum), dim3(kThreads), 0, st,
                     a, e_ntt, s, s_from, key, c->n, c->L, c->alpha, pmod, c->d_pk, sd);
  return hipGetLastError();
}

hipError_t k_key_expand_launch(const Context* c, const uint64_t* compact, uint64_t* full,
                               hipStream_t st) {
  hipLaunchKernelGGL(k_key_expand, grid_rows(c->n, c->L + c->alpha, (c->dnum + 2) / 3),
                     dim3(kThreads), 0, st, compact, full, c->n, c->L + c->alpha, c->dnum,
                     c->d_pk);
  return hipGetLastError();
}

hipError_t k_encrypt_launch(const Context* c, const uint64_t* a, const uint64_t* s,
                            const uint64_t* me, uint64_t* ct, uint32_t level, hipStream_t st) {
  hipLaunchKernelGGL(k_encrypt, grid_rows(c->n, level), dim3(kThreads), 0, st, a, s, me, ct,
                     c->n, c->d_pk);
  return hipGetLastError();
}

}  // namespace fesc
