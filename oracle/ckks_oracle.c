/*
 * CPU reference ("the oracle") for the RNS-CKKS linear computations used by
 * FESC's encrypted scan-contract (arXiv 2608.17442, Sec. 2.1 "Fully
 * Homomorphic Encryption and CKKS", Sec. 4.1 Table "CKKS primitives").
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or constant generator with the GPU library; it is plain,
 * slow, exact integer code: every modular product goes through a 128-bit
 * intermediate and a '%' reduction.
 *
 * The paper states none of the ring internals (transform order, root choice,
 * key-switch variant); the conventions here are the textbook ones:
 *   - primes q = 1 mod 2N found by scanning down from 2^bits (Miller-Rabin
 *     with the first twelve prime bases, deterministic below 3.3e24);
 *   - psi = the smallest primitive 2N-th root of unity mod q;
 *   - forward negacyclic NTT:  A[j] = sum_k a_k psi^((2 brv(j) + 1) k),
 *     computed by the radix-2 Cooley-Tukey recursion with bit-reversed
 *     output (Longa-Naehrig 2016), inverse by Gentleman-Sande;
 *   - fast basis conversion (Bajard-Eynard-Hasan-Zucca 2016, Cheon-Han-Kim-
 *     Kim-Song 2018) with centred digits (Halevi-Polyakov-Shoup 2019):
 *     y mod m = sum_i [x_i * (Q/q_i)^-1]_{q_i, centred} * (Q/q_i) mod m.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef uint64_t u64;
typedef unsigned __int128 u128;

/* ---------------------------------------------------------------- scalars */

static u64 mulmod(u64 a, u64 b, u64 q) { return (u64)(((u128)a * b) % q); }
static u64 addmod(u64 a, u64 b, u64 q) { u64 s = a + b; return s >= q ? s - q : s; }
static u64 submod(u64 a, u64 b, u64 q) { return a >= b ? a - b : a + (q - b); }

static u64 powmod(u64 a, u64 e, u64 q) {
  u64 r = 1 % q;
  a %= q;
  while (e) {
    if (e & 1) r = mulmod(r, a, q);
    a = mulmod(a, a, q);
    e >>= 1;
  }
  return r;
}

/* q prime: Fermat inverse. */
static u64 invmod(u64 a, u64 q) { return powmod(a, q - 2, q); }

u64 or_mulmod(u64 a, u64 b, u64 q) { return mulmod(a, b, q); }
u64 or_powmod(u64 a, u64 e, u64 q) { return powmod(a, e, q); }
u64 or_invmod(u64 a, u64 q) { return invmod(a, q); }

int or_is_prime(u64 n) {
  static const u64 bases[12] = {2, 3, 5, 7, 11, 13, 17, 19, 23, 29, 31, 37};
  if (n < 2) return 0;
  for (int i = 0; i < 12; ++i) {
    if (n == bases[i]) return 1;
    if (n % bases[i] == 0) return 0;
  }
  u64 d = n - 1;
  int s = 0;
  while ((d & 1) == 0) { d >>= 1; ++s; }
  for (int i = 0; i < 12; ++i) {
    u64 x = powmod(bases[i], d, n);
    if (x == 1 || x == n - 1) continue;
    int composite = 1;
    for (int r = 1; r < s; ++r) {
      x = mulmod(x, x, n);
      if (x == n - 1) { composite = 0; break; }
    }
    if (composite) return 0;
  }
  return 1;
}

/* The `count` largest primes q < 2^bits with q = 1 (mod 2^(log_n+1)),
 * in descending order.  Returns the number found. */
int or_find_primes(int log_n, int bits, int count, u64* out) {
  u64 m = (u64)1 << (log_n + 1);
  u64 top = ((u64)1 << bits) - 1;
  u64 c = (top / m) * m + 1;
  if (c > top) c -= m;
  int found = 0;
  while (found < count && c > m) {
    if (or_is_prime(c)) out[found++] = c;
    c -= m;
  }
  return found;
}

/* Smallest primitive 2N-th root of unity mod q (N = 2^log_n). */
u64 or_min_psi(u64 q, int log_n) {
  u64 two_n = (u64)2 << log_n;
  u64 n = (u64)1 << log_n;
  u64 root = 0;
  for (u64 x = 2; x < q; ++x) {
    u64 r = powmod(x, (q - 1) / two_n, q);
    if (powmod(r, n, q) == q - 1) { root = r; break; }
  }
  /* all primitive 2N-th roots are root^k, k odd */
  u64 r2 = mulmod(root, root, q);
  u64 cur = root, best = root;
  for (u64 k = 1; k < two_n; k += 2) {
    if (cur < best) best = cur;
    cur = mulmod(cur, r2, q);
  }
  return best;
}

/* ------------------------------------------------------------------- NTT */

static u64 brv(u64 x, int bits) {
  u64 r = 0;
  for (int i = 0; i < bits; ++i) { r = (r << 1) | (x & 1); x >>= 1; }
  return r;
}

/* tw[i] = root^brv(i), i < N. */
static u64* brv_power_table(u64 root, int log_n, u64 q) {
  u64 n = (u64)1 << log_n;
  u64* pw = (u64*)malloc(n * sizeof(u64));
  u64* tw = (u64*)malloc(n * sizeof(u64));
  pw[0] = 1;
  for (u64 e = 1; e < n; ++e) pw[e] = mulmod(pw[e - 1], root, q);
  for (u64 i = 0; i < n; ++i) tw[i] = pw[brv(i, log_n)];
  free(pw);
  return tw;
}

/* In place: A[j] = a(psi^(2 brv(j) + 1)), output in bit-reversed order.
 * psi: the primitive 2N-th root defining the transform (or_min_psi). */
void or_ntt_fwd(u64* a, int log_n, u64 q, u64 psi) {
  u64 n = (u64)1 << log_n;
  u64* tw = brv_power_table(psi, log_n, q);
  u64 t = n;
  for (u64 m = 1; m < n; m <<= 1) {
    t >>= 1;
    for (u64 i = 0; i < m; ++i) {
      u64 w = tw[m + i];
      u64 j1 = 2 * i * t;
      for (u64 j = j1; j < j1 + t; ++j) {
        u64 u = a[j];
        u64 v = mulmod(a[j + t], w, q);
        a[j] = addmod(u, v, q);
        a[j + t] = submod(u, v, q);
      }
    }
  }
  free(tw);
}

/* Exact inverse of or_ntt_fwd. */
void or_ntt_inv(u64* a, int log_n, u64 q, u64 psi) {
  u64 n = (u64)1 << log_n;
  u64* tw = brv_power_table(invmod(psi, q), log_n, q);
  u64 t = 1;
  for (u64 m = n >> 1; m >= 1; m >>= 1) {
    for (u64 i = 0; i < m; ++i) {
      u64 w = tw[m + i];
      u64 j1 = 2 * i * t;
      for (u64 j = j1; j < j1 + t; ++j) {
        u64 u = a[j];
        u64 v = a[j + t];
        a[j] = addmod(u, v, q);
        a[j + t] = mulmod(submod(u, v, q), w, q);
      }
    }
    t <<= 1;
  }
  u64 n_inv = invmod(n % q, q);
  for (u64 j = 0; j < n; ++j) a[j] = mulmod(a[j], n_inv, q);
  free(tw);
}

/* Row-batched transforms: row r is a polynomial modulo q[r]. */
void or_ntt_fwd_rows(u64* a, long rows, int log_n, const u64* q, const u64* psi) {
  long n = 1L << log_n;
#pragma omp parallel for schedule(dynamic, 1)
  for (long r = 0; r < rows; ++r) or_ntt_fwd(a + r * n, log_n, q[r], psi[r]);
}

void or_ntt_inv_rows(u64* a, long rows, int log_n, const u64* q, const u64* psi) {
  long n = 1L << log_n;
#pragma omp parallel for schedule(dynamic, 1)
  for (long r = 0; r < rows; ++r) or_ntt_inv(a + r * n, log_n, q[r], psi[r]);
}

/* ----------------------------------------------------------- elementwise */

/* out[r][k] = a[r][k] * b[r][k] mod q[r] */
void or_mul_rows(const u64* a, const u64* b, u64* out, long rows, long n, const u64* q) {
#pragma omp parallel for schedule(static)
  for (long r = 0; r < rows; ++r)
    for (long k = 0; k < n; ++k) out[r * n + k] = mulmod(a[r * n + k], b[r * n + k], q[r]);
}

/* out[r][k] = sum_j a[j][r][k] * b[j][r][k] mod q[r]; pairs are `pairs`
 * blocks of rows*n words, a and b laid out [pair][row][k]. */
void or_mac_rows(const u64* a, const u64* b, u64* out, long pairs, long rows, long n,
                 const u64* q) {
#pragma omp parallel for schedule(static)
  for (long r = 0; r < rows; ++r)
    for (long k = 0; k < n; ++k) {
      u64 acc = 0;
      for (long j = 0; j < pairs; ++j) {
        long o = (j * rows + r) * n + k;
        acc = addmod(acc, mulmod(a[o], b[o], q[r]), q[r]);
      }
      out[r * n + k] = acc;
    }
}

/* out[r][k] = a[r][k] * c[r] mod q[r] */
void or_mul_scalar_rows(const u64* a, u64* out, long rows, long n, const u64* q, const u64* c) {
#pragma omp parallel for schedule(static)
  for (long r = 0; r < rows; ++r)
    for (long k = 0; k < n; ++k) out[r * n + k] = mulmod(a[r * n + k], c[r] % q[r], q[r]);
}

void or_add_rows(const u64* a, const u64* b, u64* out, long rows, long n, const u64* q) {
  for (long r = 0; r < rows; ++r)
    for (long k = 0; k < n; ++k) out[r * n + k] = addmod(a[r * n + k], b[r * n + k], q[r]);
}

void or_sub_rows(const u64* a, const u64* b, u64* out, long rows, long n, const u64* q) {
  for (long r = 0; r < rows; ++r)
    for (long k = 0; k < n; ++k) out[r * n + k] = submod(a[r * n + k], b[r * n + k], q[r]);
}

/* Signed 64-bit integers reduced into each row's modulus: out[r][k] = x[k] mod q[r]. */
void or_lift_signed_rows(const int64_t* x, u64* out, long rows, long n, const u64* q) {
  for (long r = 0; r < rows; ++r)
    for (long k = 0; k < n; ++k) {
      int64_t m = x[k] % (int64_t)q[r];   /* C99: remainder takes the dividend's sign */
      out[r * n + k] = m < 0 ? (u64)(m + (int64_t)q[r]) : (u64)m;
    }
}

/* ----------------------------------------------------------- automorphism */

/* Coefficient-domain Galois automorphism X -> X^g (g odd) on every row:
 * coefficient k moves to g*k mod 2N, negated when it lands in [N, 2N). */
void or_automorph_coef_rows(const u64* a, u64* out, long rows, int log_n, const u64* q, u64 g) {
  u64 n = (u64)1 << log_n;
  u64 mask = 2 * n - 1;
  for (long r = 0; r < rows; ++r) {
    const u64* src = a + r * n;
    u64* dst = out + r * n;
    for (u64 k = 0; k < n; ++k) {
      u64 e = (k * g) & mask;
      if (e < n) dst[e] = src[k];
      else dst[e - n] = src[k] == 0 ? 0 : q[r] - src[k];
    }
  }
}

/* -------------------------------------------------- fast basis conversion */

/* src: ns rows modulo sq[]; dst: nd rows modulo dq[].  With Q = prod sq and
 * x_i = [src_i * (Q/q_i)^-1]_{q_i} taken as the CENTRED representative in
 * (-q_i/2, q_i/2):
 *   dst[m][k] = sum_i x_i * ((Q/q_i) mod dq[m])  mod dq[m].
 * No correction of the Q-multiple: the integer it represents is congruent to
 * the input modulo Q and has absolute value below ns*Q/2 (centred fast basis
 * conversion, Halevi-Polyakov-Shoup, CT-RSA 2019). */
void or_fast_bconv(const u64* src, int ns, const u64* sq, u64* dst, int nd, const u64* dq, long n) {
  if (ns > 64) return;
  u64* qhat_inv = (u64*)malloc(sizeof(u64) * ns);
  u64* qhat_mod = (u64*)malloc(sizeof(u64) * ns * nd);
  for (int i = 0; i < ns; ++i) {
    u64 prod = 1;
    for (int t = 0; t < ns; ++t)
      if (t != i) prod = mulmod(prod, sq[t] % sq[i], sq[i]);
    qhat_inv[i] = invmod(prod, sq[i]);
    for (int m = 0; m < nd; ++m) {
      u64 pm = 1;
      for (int t = 0; t < ns; ++t)
        if (t != i) pm = mulmod(pm, sq[t] % dq[m], dq[m]);
      qhat_mod[m * ns + i] = pm;
    }
  }
#pragma omp parallel for schedule(static)
  for (long k = 0; k < n; ++k) {
    u64 xs[64];
    int neg[64];
    for (int i = 0; i < ns; ++i) {
      u64 x = mulmod(src[(long)i * n + k], qhat_inv[i], sq[i]);
      neg[i] = x > sq[i] / 2;          /* centred value x - q_i < 0 */
      xs[i] = neg[i] ? sq[i] - x : x;  /* magnitude */
    }
    for (int m = 0; m < nd; ++m) {
      u64 acc = 0;
      for (int i = 0; i < ns; ++i) {
        u64 t = mulmod(xs[i], qhat_mod[m * ns + i], dq[m]);
        acc = neg[i] ? submod(acc, t, dq[m]) : addmod(acc, t, dq[m]);
      }
      dst[(long)m * n + k] = acc;
    }
  }
  free(qhat_inv);
  free(qhat_mod);
}

/* ------------------------------------------------- seed-expanded key halves
 *
 * Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC 2011): a counter-based generator; the block function
 * maps a 4-word counter and a 2-word key to 4 words by ten rounds of
 *   (x0, x1, x2, x3) <- (hi(M1 x2) ^ x1 ^ k0, lo(M1 x2), hi(M0 x0) ^ x3 ^ k1,
 *                        lo(M0 x0)),  (k0, k1) += (W0, W1)
 * with M0 = 0xD2E7470EE14C6C93, M1 = 0xCA5A826395121157 and the Weyl
 * increments W0 = 0x9E3779B97F4A7C15, W1 = 0xBB67AE8584CAA73B.
 */
void or_philox4x64(const u64* ctr, u64 k0, u64 k1, u64* out) {
  u64 x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  for (int r = 0; r < 10; ++r) {
    const u128 p0 = (u128)0xD2E7470EE14C6C93ull * x0;
    const u128 p1 = (u128)0xCA5A826395121157ull * x2;
    const u64 y0 = (u64)(p1 >> 64) ^ x1 ^ k0, y1 = (u64)p1;
    const u64 y2 = (u64)(p0 >> 64) ^ x3 ^ k1, y3 = (u64)p0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    k0 += 0x9E3779B97F4A7C15ull;
    k1 += 0xBB67AE8584CAA73Bull;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

static int bitlen(u64 q) {
  int b = 0;
  while (q >> b) ++b;
  return b;
}

/* The uniform half a_j[row][k] of a switching key, regenerated from a
 * 2-word seed instead of being stored.  For coefficient k, extended prime
 * `row_id` (the prime's index in the full chain: q_i -> i, p_k -> L + k),
 * Galois element `elt` (0: relinearisation) and digit block c (digits
 * 3c .. 3c + 2), one Philox call on the counter (k, row_id, c, elt) gives
 * words w0..w3; digit 3c + i takes w_i masked to the bit length of q if that
 * is below q, else the spare w3 (masked) if no earlier digit of the block
 * took it and it is below q, else w_i mod q.
 * out: [dnum][rows][n]; moduli and row_ids: [rows]. */
void or_seeded_key_a(u64* out, int dnum, int rows, long n, const u64* moduli, const u64* row_ids,
                     u64 k0, u64 k1, u64 elt) {
#pragma omp parallel for schedule(static)
  for (long t = 0; t < (long)rows * n; ++t) {
    const int r = (int)(t / n);
    const long k = t % n;
    const u64 q = moduli[r], mask = (q >> 63) ? ~0ull : ((1ull << bitlen(q)) - 1);
    for (int c = 0; 3 * c < dnum; ++c) {
      const u64 ctr[4] = {(u64)k, row_ids[r], (u64)c, elt};
      u64 w[4];
      or_philox4x64(ctr, k0, k1, w);
      int spare = 1;
      for (int i = 0; i < 3 && 3 * c + i < dnum; ++i) {
        u64 v = w[i] & mask;
        if (v >= q) {
          const u64 s = w[3] & mask;
          if (spare && s < q) {
            v = s;
            spare = 0;
          } else {
            v = w[i] % q;
          }
        }
        out[((size_t)(3 * c + i) * rows + r) * n + k] = v;
      }
    }
  }
}
