// Host-side parts of the library: error reporting, number theory for the
// parameter set, twiddle tables and scratch memory.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "fesc_internal.hpp"
#include "ops.hpp"

namespace fesc {

static thread_local std::string g_last_error;

int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

int hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return FESC_OK;
  return fail(FESC_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

const char* last_error() { return g_last_error.c_str(); }

// ------------------------------------------------------------ number theory

uint64_t h_mulmod(uint64_t a, uint64_t b, uint64_t m) {
  return (uint64_t)((unsigned __int128)a * b % m);
}

uint64_t h_powmod(uint64_t a, uint64_t e, uint64_t m) {
  uint64_t acc = 1 % m, base = a % m;
  for (; e; e >>= 1, base = h_mulmod(base, base, m))
    if (e & 1) acc = h_mulmod(acc, base, m);
  return acc;
}

uint64_t h_inv(uint64_t a, uint64_t p) {  // p prime
  return h_powmod(a, p - 2, p);
}

// Deterministic Miller-Rabin for 64-bit inputs (witness set of Jim Sinclair).
bool h_is_prime(uint64_t n) {
  if (n < 2) return false;
  for (uint64_t sp : {2ull, 3ull, 5ull, 7ull, 11ull, 13ull, 17ull, 19ull, 23ull, 29ull, 31ull, 37ull})
    if (n % sp == 0) return n == sp;
  uint64_t d = n - 1;
  int s = __builtin_ctzll(d);
  d >>= s;
  for (uint64_t a : {2ull, 325ull, 9375ull, 28178ull, 450775ull, 9780504ull, 1795265022ull}) {
    uint64_t x = h_powmod(a % n, d, n);
    if (a % n == 0 || x == 1 || x == n - 1) continue;
    bool witness = true;
    for (int i = 1; i < s && witness; ++i) {
      x = h_mulmod(x, x, n);
      if (x == n - 1) witness = false;
    }
    if (witness) return false;
  }
  return true;
}

// Smallest primitive 2N-th root of unity modulo q: any root g (g^N = -1)
// generates all of them as g^(2i+1); take the least.
uint64_t h_min_root(uint64_t q, uint32_t log_n) {
  const uint64_t two_n = 2ull << log_n;
  uint64_t g = 0;
  for (uint64_t cand = 3; cand < q && !g; ++cand) {
    uint64_t r = h_powmod(cand, (q - 1) / two_n, q);
    if (h_powmod(r, two_n >> 1, q) == q - 1) g = r;
  }
  const uint64_t g2 = h_mulmod(g, g, q);
  uint64_t best = g, cur = g;
  for (uint64_t i = 1; i < (two_n >> 1); ++i) {
    cur = h_mulmod(cur, g2, q);
    if (cur < best) best = cur;
  }
  return best;
}

static uint32_t bitrev(uint32_t x, uint32_t bits) {
  return __builtin_bitreverse32(x) >> (32 - bits);
}

// ------------------------------------------------- modulus trimming (host)

namespace {

using Big = std::vector<uint32_t>;  // little-endian 32-bit limbs, no leading zeros

void big_mul(Big& a, uint64_t m) {
  unsigned __int128 carry = 0;
  for (uint32_t& w : a) {
    const unsigned __int128 cur = (unsigned __int128)w * m + carry;
    w = (uint32_t)cur;
    carry = cur >> 32;
  }
  while (carry) {
    a.push_back((uint32_t)carry);
    carry >>= 32;
  }
}

uint32_t big_bits(const Big& a) {
  return a.empty() ? 0 : 32 * (uint32_t)(a.size() - 1) + (32 - __builtin_clz(a.back()));
}

// a > floor(d) for a finite d >= 1 (equivalently a > d, a being an integer)
bool big_gt(const Big& a, double d) {
  int e;
  const double m = std::frexp(d, &e);  // d = m 2^e, 0.5 <= m < 1
  uint64_t mant = (uint64_t)std::ldexp(m, 53);
  int sh = e - 53;
  if (sh < 0) {
    mant >>= -sh;
    sh = 0;
  }
  Big b;
  for (uint64_t x = mant; x; x >>= 32) b.push_back((uint32_t)x);
  if (sh) {  // b <<= sh
    const uint32_t words = sh / 32, bits = sh % 32;
    Big t(words, 0);
    uint32_t carry = 0;
    for (uint32_t w : b) {
      t.push_back(bits ? (w << bits) | carry : w);
      carry = bits ? w >> (32 - bits) : 0;
    }
    if (carry) t.push_back(carry);
    b.swap(t);
  }
  while (!b.empty() && !b.back()) b.pop_back();
  if (a.size() != b.size()) return a.size() > b.size();
  for (size_t i = a.size(); i-- > 0;)
    if (a[i] != b[i]) return a[i] > b[i];
  return false;
}

}  // namespace

int c2m_level(const uint64_t* q, uint32_t level, uint32_t ell, uint32_t sigma, double delta,
              double bmax, uint32_t* out) {
  if (!q || !out || level == 0) return fail(FESC_ERR_ARG, "bad modulus-trimming arguments");
  const double bound = 2.0 * delta * bmax;
  if (!(bound >= 0.0)) return fail(FESC_ERR_ARG, "delta * bmax must be a non-negative number");
  Big Q{1};
  *out = 0;
  for (uint32_t lp = 1; lp <= level; ++lp) {
    big_mul(Q, q[lp - 1]);
    const bool enough_bits = big_bits(Q) >= ell + sigma + 2;  // Q >= 2^(ell + sigma + 1)
    const bool no_wrap = std::isinf(bound) ? false : bound < 1.0 || big_gt(Q, bound);
    if (enough_bits && no_wrap) {
      *out = lp;
      return FESC_OK;
    }
  }
  return FESC_OK;
}

// ------------------------------------------------------------------ scratch

void* scratch_get(Context* c, size_t bytes, int* err) {
  *err = FESC_OK;
  if (bytes <= c->scratch_bytes) return c->scratch;
  if (c->scratch) {
    // previous users on the context's stream may still read it
    if ((*err = hip_check(hipDeviceSynchronize(), "hipDeviceSynchronize"))) return nullptr;
    (void)hipFree(c->scratch);
    c->scratch = nullptr;
    c->scratch_bytes = 0;
  }
  if (hipMalloc(&c->scratch, bytes) != hipSuccess) {
    c->scratch = nullptr;
    *err = fail(FESC_ERR_OOM, "scratch allocation of " + std::to_string(bytes) + " bytes failed");
    return nullptr;
  }
  c->scratch_bytes = bytes;
  return c->scratch;
}

// ------------------------------------------------------------------ context

static int build_tables(Context* c) {
  const uint32_t n = c->n, np = (uint32_t)c->ext_count();
  std::vector<PrimeK> pk(np);
  std::vector<double2> fwd((size_t)np * n), inv((size_t)np * n);
  const uint32_t nblk = n / 4096;
  std::vector<double> fwd3((size_t)np * nblk * 256), inv3(fwd3.size());
  std::vector<uint64_t> pw(n);
  for (uint32_t i = 0; i < np; ++i) {
    const uint64_t q = c->primes[i];
    const double qd = (double)q;
    const uint64_t ninv = h_inv(n % q, q);
    pk[i] = PrimeK{qd, 1.0 / qd, (double)ninv, (double)ninv / qd, q, {0, 0, 0}};
    for (int dir = 0; dir < 2; ++dir) {
      const uint64_t root = dir == 0 ? c->psi[i] : h_inv(c->psi[i], q);
      pw[0] = 1;
      for (uint32_t e = 1; e < n; ++e) pw[e] = h_mulmod(pw[e - 1], root, q);
      double2* t = (dir == 0 ? fwd.data() : inv.data()) + (size_t)i * n;
      // balanced representative, |w| <= q/2 (halves the error term of the
      // Shoup products, which the lazy butterflies rely on)
      for (uint32_t k = 0; k < n; ++k) {
        const uint64_t e = pw[bitrev(k, c->log_n)];
        const double w = e > q / 2 ? -(double)(q - e) : (double)e;
        t[k] = double2{w, w / qd};
      }
      // Block blk, thread e: psi_rev[(N + 4096 blk) / 2 + 8 e], the power from
      // which an inner pass generates the twiddles of index bits 3..0 of its
      // 16 consecutive values.
      double* t3 = (dir == 0 ? fwd3.data() : inv3.data()) + (size_t)i * nblk * 256;
      for (uint32_t blk = 0; blk < nblk; ++blk)
        for (uint32_t e = 0; e < 256; ++e)
          t3[(size_t)blk * 256 + e] = t[((n + 4096 * blk) >> 1) + 8 * e].x;
    }
  }
  // device encoding tables
  std::vector<double2> enc_tw(2 * (size_t)n);
  for (uint32_t k = 0; k < 2 * n; ++k) {
    const double ang = -M_PI * (double)k / (double)n;
    enc_tw[k] = double2{std::cos(ang), std::sin(ang)};
  }
  std::vector<int32_t> enc_inv(n);
  {
    uint64_t e = 1;
    for (uint32_t j = 0; j < n / 2; ++j) {
      enc_inv[(e - 1) / 2] = (int32_t)j;
      enc_inv[n - 1 - (e - 1) / 2] = ~(int32_t)j;
      e = e * 5 % (2ull * n);
    }
  }
  std::vector<double2> garner((size_t)c->L * c->L, double2{0.0, 0.0});
  for (uint32_t i = 0; i < c->L; ++i)
    for (uint32_t j = 0; j < i; ++j) {
      const uint64_t qi = c->primes[i];
      const uint64_t v = h_inv(c->primes[j] % qi, qi);
      const double w = v > qi / 2 ? -(double)(qi - v) : (double)v;
      garner[(size_t)i * c->L + j] = double2{w, w / (double)qi};
    }
  int rc;
  if ((rc = hip_check(hipMalloc(&c->d_garner, sizeof(double2) * garner.size()), "hipMalloc")) ||
      (rc = hip_check(hipMemcpy(c->d_garner, garner.data(), sizeof(double2) * garner.size(),
                                hipMemcpyHostToDevice), "hipMemcpy")))
    return rc == FESC_ERR_HIP ? fail(FESC_ERR_OOM, "decoding table allocation failed") : rc;
  if ((rc = hip_check(hipMalloc(&c->d_enc_tw, sizeof(double2) * enc_tw.size()), "hipMalloc")) ||
      (rc = hip_check(hipMalloc(&c->d_enc_inv, sizeof(int32_t) * enc_inv.size()), "hipMalloc")) ||
      (rc = hip_check(hipMemcpy(c->d_enc_tw, enc_tw.data(), sizeof(double2) * enc_tw.size(),
                                hipMemcpyHostToDevice), "hipMemcpy")) ||
      (rc = hip_check(hipMemcpy(c->d_enc_inv, enc_inv.data(), sizeof(int32_t) * enc_inv.size(),
                                hipMemcpyHostToDevice), "hipMemcpy")))
    return rc == FESC_ERR_HIP ? fail(FESC_ERR_OOM, "encoding table allocation failed") : rc;
  if ((rc = hip_check(hipMalloc(&c->d_pk, sizeof(PrimeK) * np), "hipMalloc")) ||
      (rc = hip_check(hipMalloc(&c->d_tw_fwd, sizeof(double2) * fwd.size()), "hipMalloc")) ||
      (rc = hip_check(hipMalloc(&c->d_tw_inv, sizeof(double2) * inv.size()), "hipMalloc")) ||
      (rc = hip_check(hipMalloc(&c->d_tw3_fwd, sizeof(double) * fwd3.size()), "hipMalloc")) ||
      (rc = hip_check(hipMalloc(&c->d_tw3_inv, sizeof(double) * inv3.size()), "hipMalloc")))
    return rc == FESC_ERR_HIP ? fail(FESC_ERR_OOM, "table allocation failed") : rc;
  if ((rc = hip_check(hipMemcpy(c->d_pk, pk.data(), sizeof(PrimeK) * np, hipMemcpyHostToDevice),
                      "hipMemcpy")) ||
      (rc = hip_check(hipMemcpy(c->d_tw_fwd, fwd.data(), sizeof(double2) * fwd.size(),
                                hipMemcpyHostToDevice), "hipMemcpy")) ||
      (rc = hip_check(hipMemcpy(c->d_tw_inv, inv.data(), sizeof(double2) * inv.size(),
                                hipMemcpyHostToDevice), "hipMemcpy")) ||
      (rc = hip_check(hipMemcpy(c->d_tw3_fwd, fwd3.data(), sizeof(double) * fwd3.size(),
                                hipMemcpyHostToDevice), "hipMemcpy")) ||
      (rc = hip_check(hipMemcpy(c->d_tw3_inv, inv3.data(), sizeof(double) * inv3.size(),
                                hipMemcpyHostToDevice), "hipMemcpy")))
    return rc;
  return FESC_OK;
}

void destroy(Context* c) {
  if (!c) return;
  (void)hipDeviceSynchronize();
  for (auto& kv : c->keys) (void)hipFree(kv.second);
  for (auto& kv : c->level_tabs) (void)hipFree(kv.second.base);
  (void)hipFree(c->d_pk);
  (void)hipFree(c->d_tw_fwd);
  (void)hipFree(c->d_tw_inv);
  (void)hipFree(c->d_tw3_fwd);
  (void)hipFree(c->d_tw3_inv);
  (void)hipFree(c->d_enc_tw);
  (void)hipFree(c->d_enc_inv);
  (void)hipFree(c->d_garner);
  (void)hipFree(c->scratch);
  delete static_cast<fesc_ctx*>(c);
}

int create(const fesc_params* p, fesc_ctx** out) {
  if (!p || !out) return fail(FESC_ERR_ARG, "null argument");
  *out = nullptr;
  if (p->log_n < 12 || p->log_n > 16)
    return fail(FESC_ERR_ARG, "log_n must lie in [12, 16]");
  if (p->num_q < 1 || p->num_p < 1 || p->num_p > FESC_MAX_ALPHA ||
      p->num_q + p->num_p > FESC_MAX_PRIMES || !p->q || !p->p)
    return fail(FESC_ERR_ARG, "need 1 <= num_q, 1 <= num_p <= 16, num_q + num_p <= 64");
  const uint32_t dnum = (p->num_q + p->num_p - 1) / p->num_p;
  if (p->dnum != dnum)
    return fail(FESC_ERR_ARG, "dnum must equal ceil(num_q / num_p) = " + std::to_string(dnum));
  if (dnum > 16) return fail(FESC_ERR_ARG, "at most 16 digits (dnum <= 16)");
  const uint64_t two_n = 2ull << p->log_n;
  std::vector<uint64_t> primes(p->q, p->q + p->num_q);
  primes.insert(primes.end(), p->p, p->p + p->num_p);
  for (size_t i = 0; i < primes.size(); ++i) {
    const uint64_t q = primes[i];
    if (q >= (1ull << 50) || q % two_n != 1 || !h_is_prime(q))
      return fail(FESC_ERR_ARG, "prime " + std::to_string(i) +
                                    " is not a prime below 2^50 congruent to 1 mod 2N");
    for (size_t j = 0; j < i; ++j)
      if (primes[j] == q) return fail(FESC_ERR_ARG, "primes must be distinct");
  }
  fesc_ctx* c = new fesc_ctx();
  if (int rc = hip_check(hipGetDevice(&c->device), "hipGetDevice")) {
    delete c;
    return rc;
  }
  c->log_n = p->log_n;
  c->n = 1u << p->log_n;
  c->L = p->num_q;
  c->alpha = p->num_p;
  c->dnum = dnum;
  c->primes = primes;
  for (uint64_t q : primes) c->psi.push_back(h_min_root(q, p->log_n));
  int rc = build_tables(c);
  // the per-level constants of every level up front, so that operations
  // (the rotation batch that allocates nothing among them) find them built
  for (uint32_t l = 1; l <= c->L && !rc; ++l)
    if (!level_tables(c, l, &rc)) break;
  if (!rc) rc = static_scratch_init(c);
  if (rc) {
    destroy(c);
    return rc;
  }
  *out = c;
  return FESC_OK;
}

}  // namespace fesc
