// Internal definitions shared by the HIP kernels and the host-side library.
//
// Residue arithmetic runs in IEEE fp64 on the VALU: every prime is below 2^50,
// so residues, sums of a few residues and the exact low half of a product
// (recovered with one FMA) are all exact integers in a double.  A modular
// product x*w mod q with a precomputed w' = w/q (Shoup's method carried over
// to floating point, cf. van der Hoeven, Lecerf and Quintin, "Modular SIMD
// arithmetic in Mathemagix", ACM TOMS 2016) is
//     h = x*w;  l = fma(x, w, -h);  c = rint(x*w');  r = fma(-c, q, h) + l
// which is exact and lands in (-1.5q, 1.5q) for |x| < 3q.  Values inside a
// kernel live in this signed, lazily reduced form; only stores to caller
// memory are reduced to the canonical range [0, q) and converted to uint64.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include <map>
#include <set>
#include <string>
#include <vector>

#include "fesc.h"

namespace fesc {

// ------------------------------------------------------------ device math

struct PrimeK {        // per-prime constants read by kernels
  double q;            // the prime
  double qinv;         // fl(1/q)
  double ninv, ninvp;  // N^-1 mod q and fl(N^-1 / q)
  uint64_t qu;         // the prime as an integer
  uint64_t pad[3];
};

__device__ __forceinline__ double mm_shoup(double x, double w, double wp, double q) {
  double h = x * w;
  double l = __builtin_fma(x, w, -h);
  double c = __builtin_rint(x * wp);
  double d = __builtin_fma(-c, q, h);
  return d + l;
}

__device__ __forceinline__ double mm_var(double x, double y, double q, double qinv) {
  double h = x * y;
  double l = __builtin_fma(x, y, -h);
  double c = __builtin_rint(h * qinv);
  double d = __builtin_fma(-c, q, h);
  return d + l;
}

// |x| < 2^52 -> congruent value in [-q/2 - eps, q/2 + eps]
__device__ __forceinline__ double red_bal(double x, double q, double qinv) {
  return __builtin_fma(-__builtin_rint(x * qinv), q, x);
}

// |x| < 2^52 -> canonical representative in [0, q)
__device__ __forceinline__ double red_full(double x, double q, double qinv) {
  double r = red_bal(x, q, qinv);
  return r < 0.0 ? r + q : r;
}

// centred representative in (-q/2, q/2) of a canonical value in [0, q)
__device__ __forceinline__ double center(double x, double q) {
  return x > 0.5 * q ? x - q : x;
}

// Galois automorphism X -> X^g (g odd, < 2N) in evaluation form: the value at
// index jp of sigma_g(a) is a[galois_src(jp)], the index whose evaluation
// point psi^(2 brv(j) + 1) is the g-th power of jp's point.
__device__ __forceinline__ uint32_t galois_src(uint32_t jp, uint32_t g, uint32_t log_n) {
  const uint32_t b = __builtin_bitreverse32(jp) >> (32 - log_n);
  const uint32_t e = (g * (2u * b + 1u)) & ((2u << log_n) - 1u);  // wraps mod 2^32 first
  return __builtin_bitreverse32((e - 1u) >> 1) >> (32 - log_n);
}

// Integer <-> double for values below 2^52: the double 2^52 + x has exactly
// x in its 52 mantissa bits, so each direction is one bit operation and one
// fp64 add.
constexpr double kTwo52 = 4503599627370496.0;

// x: residue (below 2^52)
__device__ __forceinline__ double u2d(uint64_t x) {
  return __longlong_as_double((long long)(x | 0x4330000000000000ull)) - kTwo52;
}

// Canonical residue in [0, q) of an integer-valued x, |x| < 2^52, as uint64.
__device__ __forceinline__ uint64_t to_res(double x, double q, double qinv) {
  const double r = red_bal(x, q, qinv);
  const double v = r + (r < 0.0 ? q + kTwo52 : kTwo52);
  return (uint64_t)__double_as_longlong(v) & 0x000FFFFFFFFFFFFFull;
}

// ------------------------------------------------------------- host side

#define FESC_MAX_PRIMES 64
#define FESC_MAX_ALPHA 16

// Per-level constants of basis conversion and rescaling (device arrays
// carved from one allocation `base`); entries are {v, fl(v / m)}.
struct LevelTables {
  void* base = nullptr;
  uint32_t level = 0;
  double2* mu_inv = nullptr;   // [dnum][alpha]             (Q_D/q_a)^-1 mod q_a
  double2* mu_hat = nullptr;   // [dnum][level+alpha][alpha] (Q_D/q_a) mod m_row
  double2* md_inv = nullptr;   // [alpha]                   (P/p_k)^-1 mod p_k
  double2* md_hat = nullptr;   // [level][alpha]            (P/p_k) mod q_i
  double2* md_pinv = nullptr;  // [level]                   P^-1 mod q_i
  double2* pmod = nullptr;     // [L]                       P mod q_i
  double2* rs_inv = nullptr;   // [level]                   q_{level-1}^-1 mod q_i
  double2* mu_inv_n = nullptr; // [level]  N^-1 (Q_D/q_i)^-1 mod q_i (q_i in digit D)
  double2* md_inv_n = nullptr; // [alpha]  N^-1 (P/p_k)^-1 mod p_k
  double2* rs_ninv = nullptr;  // [1]      N^-1 mod q_{level-1}
  double2* one = nullptr;      // [level]  1 (with 1/q_i)
  // ModDown merged with the rescale (division by M = P q_{level-1}); digit
  // sources m_0 = q_{level-1}, m_{1+k} = p_k
  double2* mr_inv_n = nullptr; // [alpha+1]  N^-1 (M/m_j)^-1 mod m_j (m_0: N^-1, the row holding x P^-1)
  double2* mr_hat = nullptr;   // [level-1][alpha+1]  (M/m_j) mod q_i
  // int8 operands of the matrix-core basis conversion (k_bconv_mfma, alpha
  // <= 8): per target row 512 bytes [tau 8][lane group 4][16]; byte b of
  // (tau, lg) is the balanced base-256 digit tau of 256^s hat_a mod m_row,
  // a = 2 lg + b / 8, s = b % 8 (zero for s = 7 and past the digit's primes)
  int8_t* mu_bytes = nullptr;  // [dnum][level+alpha][512]  of mu_hat
  int8_t* md_bytes = nullptr;  // [level][512]              of md_hat
  int8_t* mr_bytes = nullptr;  // [level-1][512]            of mr_hat, digit sources 0..7
};

struct Context {
  int device = 0;
  uint32_t log_n = 0, n = 0;
  uint32_t L = 0, alpha = 0, dnum = 0;
  std::vector<uint64_t> primes;   // ext order: q_0..q_{L-1}, p_0..p_{alpha-1}
  std::vector<uint64_t> psi;      // smallest primitive 2N-th root per prime
  PrimeK* d_pk = nullptr;         // [L+alpha]
  // [L+alpha][N] {w, w/q}, w = psi^brv(i) (inverse: psi^-brv(i)) as the
  // balanced representative in [-q/2, q/2]
  double2* d_tw_fwd = nullptr;
  double2* d_tw_inv = nullptr;
  // the powers used by the radix-16 step on index bits 3..0 of the 4096-point
  // inner NTT blocks, re-ordered [L+alpha][N/4096][15][256] (see ntt.hip)
  double* d_tw3_fwd = nullptr;
  double* d_tw3_inv = nullptr;
  // device encoding: T[k] = exp(-i pi k / N) for k < 2N, and the inverse slot
  // map (position p of the length-N transform input holds z_j if inv[p] = j,
  // conj(z_j) if inv[p] = ~j)
  double2* d_enc_tw = nullptr;
  int32_t* d_enc_inv = nullptr;
  // device decoding's mixed-radix CRT: [L][L], entry [i][j] (j < i) =
  // q_j^-1 mod q_i as {w, w / q_i}, w the balanced representative
  double2* d_garner = nullptr;
  // keys: Galois element (0 = relinearisation) -> device [dnum][L+alpha][2][N]
  // (seed-expanded keys: the compact layout, see seedkey.hpp)
  std::map<uint32_t, uint64_t*> keys;
  std::map<const uint64_t*, size_t> key_alloc;  // key buffer -> words allocated
  std::set<const uint64_t*> key_seeded;          // key buffers in the compact layout
  // keys uploaded over a chain prefix: key buffer -> the highest level it
  // serves (keys absent here serve every level)
  std::map<const uint64_t*, uint32_t> key_cap;
  // basis-conversion / rescale constants, built on first use per level
  std::map<uint32_t, LevelTables> level_tabs;
  // scratch (grown on demand, freed with the context)
  void* scratch = nullptr;
  size_t scratch_bytes = 0;
  // device address of the statically allocated scratch array on this
  // context's device (the rotation batch that allocates nothing)
  uint64_t* static_scratch = nullptr;
  hipStream_t stream = nullptr;   // default stream when callers pass null

  size_t ext_count() const { return primes.size(); }
};

// thread-local error message, set by fail()
int fail(int code, const std::string& msg);
int hip_check(hipError_t e, const char* what);

void* scratch_get(Context* c, size_t bytes, int* err);

// host number theory
uint64_t h_mulmod(uint64_t a, uint64_t b, uint64_t m);
uint64_t h_powmod(uint64_t a, uint64_t e, uint64_t m);
uint64_t h_inv(uint64_t a, uint64_t p);
bool h_is_prime(uint64_t n);
uint64_t h_min_root(uint64_t q, uint32_t log_n);

// Row selection of a batched NTT launch (see ntt.hip).
struct RowSel {
  uint64_t* base;
  size_t batch_stride, limb_stride;
  uint32_t prime0, split, prime1;
  uint32_t skip_alpha, skip_limit, skip_mod;
  __device__ uint64_t* row() const;
  __device__ uint32_t prime() const;
  __device__ bool skip() const;
};

// kernel launchers (ntt.hip)
hipError_t launch_ntt_rows(const Context* c, const RowSel& rs, uint32_t batch, uint32_t limbs,
                           bool inverse, hipStream_t s);
hipError_t launch_ntt(const Context* c, uint64_t* d, uint32_t batch, size_t batch_stride,
                      uint32_t limbs, size_t limb_stride, uint32_t prime0, bool inverse,
                      hipStream_t s);

}  // namespace fesc

// The opaque handle of the C ABI is the context itself.
struct fesc_ctx : public fesc::Context {};

namespace fesc {
int create(const fesc_params* p, fesc_ctx** out);
void destroy(Context* c);
const char* last_error();
hipError_t launch_mac(const Context* c, const uint64_t* a, const uint64_t* b, uint64_t* out,
                      uint32_t pairs, size_t pair_stride, uint32_t limbs, uint32_t prime0,
                      hipStream_t s);
}  // namespace fesc
