// Negacyclic NTT / inverse NTT over word-sized primes, batched over rows.
//
// Definition (the forward transform's output order is bit-reversed):
//     A[j] = sum_k a_k psi^((2 brv(j) + 1) k)  mod q,
// psi the smallest primitive 2N-th root of unity mod q.  The transform is the
// radix-2 Cooley-Tukey network whose butterfly on the pair (j, j + t) uses the
// twiddle psi^brv((N + j) / 2t); the inverse is the Gentleman-Sande network
// with psi^-1 and a final scaling by N^-1.
//
// gfx950 mapping.  N = M * 4096 with M = 2^(log N - 12) in [1, 16].  At most
// two passes over HBM, each over independent sub-transforms held on chip:
//   outer pass (M > 1): the first log M stages couple only indices that agree
//               mod 4096, i.e. M-point "columns" at stride 4096.  A thread
//               keeps whole columns in registers; a wavefront reads and writes
//               64 adjacent columns, so every access is a contiguous 512-byte
//               run (2 KB per workgroup) and no LDS is needed.  The twiddles of
//               these stages do not depend on the column (M - 1 values).
//   inner pass: the last 12 stages couple only indices inside a contiguous
//               4096-element block, one block per 256-thread workgroup.  The
//               block is processed as three radix-16 register steps on index
//               bits 11..8, 7..4 and 3..0, with LDS transposes in between, so
//               loads and stores of the forward pass are fully coalesced.
// Between the passes the row holds the signed fp64 intermediate in place of
// the uint64 residues (same 8 bytes per value), so no conversion or full
// reduction is spent on it.  For N = 4096 the inner pass alone is the whole
// transform.
//
// Twiddles: the outer passes read the bit-reversed power table (uniform per
// stage); an inner pass stages its block's 255 twiddles of bits 11..4 in LDS
// next to the data and generates those of bits 3..0 from one power per
// thread (Context::d_tw3_*), so that no global load is waited on
// between its butterflies.
#include <type_traits>

#include "butterfly.hpp"
#include "fesc_internal.hpp"
#include "ops.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;
constexpr uint32_t kBlock = 4096;

// LDS layout of a 4096-value block: one pad word after every 16 values, so
// value k sits at k + k/16.  All three access patterns below then reduce to a
// per-thread base plus a compile-time offset (no address arithmetic per
// access), and 16 consecutive lanes always hit 16 distinct 8-byte bank slots.
//   lds_row(t, r):    value t + 256 r        (bits 11..8 in registers)
//   lds_mid(a, b, r): value 256 a + 16 r + b (bits 7..4 in registers)
//   lds_col(t, r):    value 16 t + r         (bits 3..0 in registers)
__device__ __forceinline__ uint32_t lds_row(uint32_t t, uint32_t r) {
  return (t + (t >> 4)) + 272 * r;
}
__device__ __forceinline__ uint32_t lds_mid(uint32_t a, uint32_t b, uint32_t r) {
  return (272 * a + b) + 17 * r;
}
__device__ __forceinline__ uint32_t lds_col(uint32_t t, uint32_t r) { return 17 * t + r; }
constexpr int kLds = kBlock + kBlock / 16;

// Inner passes: the twiddles of bits 11..4 staged in LDS per block.  For
// index bits 11..8 (register distance H, distance 256 H) the group twiddle is
// psi_rev[(N + B) / 512H + gi]; for bits 7..4 (distance 16 H) with a = bits
// 11..8 of the thread's values it is psi_rev[(N + B) / 32H + a * 8/H + gi]
// (B the block offset in the row): eight contiguous runs of the table, 255
// values.  Entry t < 255 of the staging array lies in segment k = floor(log2(t + 1))
// (the 2^k group twiddles of one stage) at index t + 1 - 2^k, i.e.
// psi_rev[(N + B) / 2^(12 - k) + t + 1 - 2^k]; entries 255..261 are
// psi_rev[1..7].  For bits 11..8 (distance 256 H) the stage of H uses
// segment log2(8/H); for bits 7..4 (distance 16 H) segment 4 + log2(8/H), at
// a * 8/H + gi.
constexpr int kTwL = 262;
__device__ __forceinline__ double2 block_twiddle(const double2* tw, uint32_t nb, uint32_t t) {
  const uint32_t k = 31 - __builtin_clz(t + 1);  // t < 255
  return tw[(nb >> (12 - k)) + t + 1 - (1u << k)];
}
struct TwL {
  const double2* lt;
  uint32_t off;
  __device__ __forceinline__ double2 operator()(int gi) const { return lt[off + gi]; }
};

// Bits 3..0, generated instead of loaded: thread t's 16 consecutive values
// are positions 16 j + r with j = (N + B) / 16 + t; brv(j) has its three low
// bits clear, so psi_rev[j 8/H + gi] = psi_rev[j 8/H] psi_rev[gi] and
// psi_rev[j 8/H] = b^(8/H) with b = psi_rev[8 j].  Each twiddle is formed as
// the balanced representative (the table's value) and w' = w / q as w qinv
// (as for the loaded ones).
struct TwGen {
  double base;         // psi_rev[j 8/H], balanced
  const double2* c;    // psi_rev[1..7] (LDS)
  double q, qinv;
  __device__ __forceinline__ double2 operator()(int gi) const {
    const double w =
        gi == 0 ? base : red_bal(mm_shoup(base, c[gi - 1].x, c[gi - 1].y, q), q, qinv);
    return double2{w, w * qinv};
  }
};
__device__ __forceinline__ double sq_bal(double b, double q, double qinv) {
  return red_bal(mm_shoup(b, b, b * qinv, q), q, qinv);
}

}  // namespace

// Row selection of a batched transform launch.  blockIdx.y = batch index b,
// blockIdx.z = limb index i (the batch varies fastest between workgroups, so
// the twiddle tables of one prime stay resident in L2 across the batch).
// Limb i < split uses prime prime0 + i, limb i >= split prime1 + (i - split).
// If skip_alpha != 0, limbs [d*skip_alpha, min((d+1)*skip_alpha, skip_limit))
// of batch element b, d = b mod skip_mod, are left untouched (the own-digit
// rows of digit d in a batch of ModUp outputs).
__device__ __forceinline__ uint64_t* RowSel::row() const {
  return base + (size_t)blockIdx.y * batch_stride + (size_t)blockIdx.z * limb_stride;
}
__device__ __forceinline__ uint32_t RowSel::prime() const {
  const uint32_t i = blockIdx.z;
  return i < split ? prime0 + i : prime1 + (i - split);
}
__device__ __forceinline__ bool RowSel::skip() const {
  if (!skip_alpha) return false;
  const uint32_t lo = (blockIdx.y % skip_mod) * skip_alpha;
  const uint32_t hi = min(lo + skip_alpha, skip_limit);
  return blockIdx.z >= lo && blockIdx.z < hi;
}

namespace {

// ------------------------------------------------------------- outer pass

// M = 2^LOGM point columns at stride 4096; a thread holds C = 16/M columns,
// c0 + 256 j (j < C), value m of column j in x[j*M + m].  Grid x = M.
// Stage s (distance 4096 * M/2^(s+1)) uses psi_rev[2^s + m / 2^(LOGM-s)].
// Forward stages reduce lazily as in ct_st (even s reduce).
template <int LOGM>
__global__ __launch_bounds__(kThreads) void k_fwd_outer(RowSel rs, uint32_t log_n,
                                                        const PrimeK* __restrict__ pk,
                                                        const double2* __restrict__ twf) {
  constexpr int M = 1 << LOGM, C = 16 / M;
  if (rs.skip()) return;
  const uint32_t n = 1u << log_n;
  const uint32_t prime = rs.prime();
  const double q = pk[prime].q, qinv = pk[prime].qinv;
  const double2* tw = twf + (size_t)prime * n;
  uint64_t* row = rs.row();
  const uint32_t c0 = blockIdx.x * (kThreads * C) + threadIdx.x;
  double x[16];
#pragma unroll
  for (int j = 0; j < C; ++j)
#pragma unroll
    for (int m = 0; m < M; ++m) x[j * M + m] = u2d(row[c0 + kThreads * j + kBlock * m]);
#pragma unroll
  for (int s = 0; s < LOGM; ++s) {
    const int H = M >> (s + 1);
#pragma unroll
    for (int m = 0; m < M; ++m) {
      if (m & H) continue;
      const double2 w = tw[(1 << s) + (m >> (LOGM - s))];
#pragma unroll
      for (int j = 0; j < C; ++j) {
        const double u = (s % 2 == 0) ? red_bal(x[j * M + m], q, qinv) : x[j * M + m];
        const double v = mm_shoup(x[j * M + m + H], w.x, w.y, q);
        x[j * M + m] = u + v;
        x[j * M + m + H] = u - v;
      }
    }
  }
  double* rowd = reinterpret_cast<double*>(row);
#pragma unroll
  for (int j = 0; j < C; ++j)
#pragma unroll
    for (int m = 0; m < M; ++m) rowd[c0 + kThreads * j + kBlock * m] = x[j * M + m];
}

// Final store of an inverse transform: N^-1 x as a canonical uint64 residue.
struct InvCanon {
  __device__ __forceinline__ void operator()(uint64_t* row, uint32_t k, double x,
                                             const PrimeK& P) const {
    row[k] = to_res(mm_shoup(x, P.ninv, P.ninvp, P.q), P.q, P.qinv);
  }
};

// Final store of an inverse transform that feeds a fast basis conversion: the
// centred digit [N^-1 f_i x]_q in (-q/2, q/2), stored as fp64 in place of the
// residue.  f holds {N^-1 f_i mod q_i, /q_i} per limb i (blockIdx.z), where
// f_i is the conversion's (Q_D/q_i)^-1.
struct InvDigit {
  const double2* f;
  __device__ __forceinline__ void operator()(uint64_t* row, uint32_t k, double x,
                                             const PrimeK& P) const {
    const double2 c = f[blockIdx.z];
    reinterpret_cast<double*>(row)[k] =
        center(red_full(mm_shoup(x, c.x, c.y, P.q), P.q, P.qinv), P.q);
  }
};

// Inverse: stages in reverse order (every other one reducing, as in gs_st),
// then the final store (N^-1 scaling included).
template <int LOGM, class St>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(5))) void k_inv_outer(RowSel rs, uint32_t log_n,
                                                        const PrimeK* __restrict__ pk,
                                                        const double2* __restrict__ twi, St st) {
  constexpr int M = 1 << LOGM, C = 16 / M;
  if (rs.skip()) return;
  const uint32_t n = 1u << log_n;
  const uint32_t prime = rs.prime();
  const PrimeK P = pk[prime];
  const double2* tw = twi + (size_t)prime * n;
  uint64_t* row = rs.row();
  const double* rowd = reinterpret_cast<const double*>(row);
  const uint32_t c0 = blockIdx.x * (kThreads * C) + threadIdx.x;
  double x[16];
#pragma unroll
  for (int j = 0; j < C; ++j)
#pragma unroll
    for (int m = 0; m < M; ++m) x[j * M + m] = rowd[c0 + kThreads * j + kBlock * m];
#pragma unroll
  for (int s = LOGM - 1; s >= 0; --s) {
    const int H = M >> (s + 1);
#pragma unroll
    for (int m = 0; m < M; ++m) {
      if (m & H) continue;
      const double2 w = tw[(1 << s) + (m >> (LOGM - s))];
#pragma unroll
      for (int j = 0; j < C; ++j) {
        const double u = x[j * M + m], v = x[j * M + m + H];
        x[j * M + m] = ((LOGM - 1 - s) % 2 == 0) ? red_bal(u + v, P.q, P.qinv) : u + v;
        x[j * M + m + H] = mm_shoup(u - v, w.x, w.y, P.q);
      }
    }
  }
#pragma unroll
  for (int j = 0; j < C; ++j)
#pragma unroll
    for (int m = 0; m < M; ++m) st(row, c0 + kThreads * j + kBlock * m, x[j * M + m], P);
}

// ------------------------------------------ basis conversion + outer pass

// Fused fast basis conversion and first forward pass.  For group g
// (blockIdx.z) and targets t = T blockIdx.y .. T blockIdx.y + T - 1 of the
// map, value k of target row t (prime m) is
//     y_k = sum_{a < aj} x_a[k] * hat_a  mod m,
// x_a the centred digits stored by the inverse transform (InvDigit, fp64).
// The first log M forward stages then run on the thread's columns exactly as
// in k_fwd_outer and the fp64 intermediate is stored; for M = 1 (no outer
// pass) the canonical residue is stored instead.  Targets vary fastest after
// the column block, so all targets of a column block run together and read
// its digit rows from L2; with M a multiple of 8 a column block also stays on
// one XCD (workgroups are dealt to the 8 XCDs round-robin).
template <int LOGM, int T, class Map>
__global__ __launch_bounds__(kThreads) void k_bconv_outer(Map map, uint32_t log_n,
                                                          const PrimeK* __restrict__ pk,
                                                          const double2* __restrict__ twf) {
  constexpr int M = 1 << LOGM, C = 16 / M;
  const uint32_t g = blockIdx.z, t0 = blockIdx.y * T;
  const uint32_t nt = map.targets(g);
  if (t0 >= nt) return;
  const uint32_t n = 1u << log_n;
  const uint32_t aj = map.aj(g);
  uint32_t prime[T];
  const double2* hat[T];
#pragma unroll
  for (int i = 0; i < T; ++i) {
    const uint32_t row = map.row(g, min(t0 + i, nt - 1));
    prime[i] = map.prime(row);
    hat[i] = map.hat(g, row);
  }
  const double* dig = map.digits(g);
  const uint32_t c0 = blockIdx.x * (kThreads * C) + threadIdx.x;
  double y[T][16];
#pragma unroll
  for (int i = 0; i < T; ++i)
#pragma unroll
    for (int v = 0; v < 16; ++v) y[i][v] = 0.0;
  // |x_a| < 2^49 and hat_a < m: each Shoup product lies within 0.625 m, so
  // eight terms and a carried reduced sum stay below 2^53
  for (uint32_t a = 0; a < map.alpha; ++a) {
    const uint32_t ac = a < aj ? a : aj - 1;
    const double* da = dig + (size_t)ac * n + c0;
    double x[16];
#pragma unroll
    for (int j = 0; j < C; ++j)
#pragma unroll
      for (int m = 0; m < M; ++m) x[j * M + m] = da[kThreads * j + kBlock * m];
#pragma unroll
    for (int i = 0; i < T; ++i) {
      const double q = pk[prime[i]].q;
      const double2 h = a < aj ? hat[i][ac] : double2{0.0, 0.0};
#pragma unroll
      for (int v = 0; v < 16; ++v) y[i][v] += mm_shoup(x[v], h.x, h.y, q);
    }
    if ((a & 7) == 7) {
#pragma unroll
      for (int i = 0; i < T; ++i) {
        const double q = pk[prime[i]].q, qinv = pk[prime[i]].qinv;
#pragma unroll
        for (int v = 0; v < 16; ++v) y[i][v] = red_bal(y[i][v], q, qinv);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < T; ++i) {
    if (t0 + i >= nt) break;
    const uint32_t row = map.row(g, t0 + i);
    const double q = pk[prime[i]].q, qinv = pk[prime[i]].qinv;
    uint64_t* out = map.out(g, row);
    double (&x)[16] = y[i];
    if constexpr (LOGM == 0) {
#pragma unroll
      for (int v = 0; v < 16; ++v) out[c0 + kThreads * v] = to_res(x[v], q, qinv);
    } else {
      const double2* tw = twf + (size_t)prime[i] * n;
#pragma unroll
      for (int v = 0; v < 16; ++v) x[v] = red_bal(x[v], q, qinv);
#pragma unroll
      for (int s = 0; s < LOGM; ++s) {
        const int H = M >> (s + 1);
#pragma unroll
        for (int m = 0; m < M; ++m) {
          if (m & H) continue;
          const double2 w = tw[(1 << s) + (m >> (LOGM - s))];
#pragma unroll
          for (int j = 0; j < C; ++j) {
            const double u = (s % 2 == 0) ? red_bal(x[j * M + m], q, qinv) : x[j * M + m];
            const double v = mm_shoup(x[j * M + m + H], w.x, w.y, q);
            x[j * M + m] = u + v;
            x[j * M + m + H] = u - v;
          }
        }
      }
      double* outd = reinterpret_cast<double*>(out);
#pragma unroll
      for (int j = 0; j < C; ++j)
#pragma unroll
        for (int m = 0; m < M; ++m) outd[c0 + kThreads * j + kBlock * m] = x[j * M + m];
    }
  }
}

// ModUp: group g = s * dnum + j (source s, digit j = primes [lo, lo + aj)),
// targets = the extended rows outside the digit, digits = cc[s][lo ..].
struct ModupMap {
  const double* cc;
  uint64_t* ext;
  const double2* mu_hat;
  uint32_t level, L, alpha, dnum_l, n;
  const int8_t* mu_bytes;  // matrix-core operands (LevelTables::mu_bytes), or null
  __device__ uint32_t lo(uint32_t g) const { return (g % dnum_l) * alpha; }
  __device__ uint32_t aj(uint32_t g) const { return min(alpha, level - lo(g)); }
  __device__ uint32_t targets(uint32_t g) const { return level + alpha - aj(g); }
  __device__ uint32_t row(uint32_t g, uint32_t t) const {
    const uint32_t l = lo(g);
    return t < l ? t : t + aj(g);
  }
  __device__ uint32_t prime(uint32_t r) const { return r < level ? r : L + (r - level); }
  __device__ const double* digits(uint32_t g) const {
    return cc + ((size_t)(g / dnum_l) * level + lo(g)) * n;
  }
  __device__ const double2* hat(uint32_t g, uint32_t r) const {
    return mu_hat + ((size_t)(g % dnum_l) * (level + alpha) + r) * alpha;
  }
  __device__ uint64_t* out(uint32_t g, uint32_t r) const {
    return ext + ((size_t)g * (level + alpha) + r) * n;
  }
  __device__ const int8_t* bytes(uint32_t g, uint32_t r) const {
    return mu_bytes + ((size_t)(g % dnum_l) * (level + alpha) + r) * 512;
  }
};

// ModDown: group g = 2 * job + component, digits = the alpha special-prime
// rows of acc[g], targets = the level rows of y[g].
struct ModdownMap {
  const uint64_t* acc;
  uint64_t* y;
  const double2* md_hat;
  uint32_t level, alpha, n;
  const int8_t* md_bytes;  // matrix-core operands (LevelTables::md_bytes), or null
  __device__ uint32_t aj(uint32_t) const { return alpha; }
  __device__ uint32_t targets(uint32_t) const { return level; }
  __device__ uint32_t row(uint32_t, uint32_t t) const { return t; }
  __device__ uint32_t prime(uint32_t r) const { return r; }
  __device__ const double* digits(uint32_t g) const {
    return reinterpret_cast<const double*>(acc + ((size_t)g * (level + alpha) + level) * n);
  }
  __device__ const double2* hat(uint32_t, uint32_t r) const { return md_hat + (size_t)r * alpha; }
  __device__ uint64_t* out(uint32_t g, uint32_t r) const {
    return y + ((size_t)g * level + r) * n;
  }
  __device__ const int8_t* bytes(uint32_t, uint32_t r) const { return md_bytes + (size_t)r * 512; }
};

// ModDown merged with the rescale: group g = 2 * job + component, digits =
// the alpha + 1 rows level-1 .. level+alpha-1 of acc[g] (q_{level-1}, then the
// special primes), targets = rows 0 .. rows-1 (< level - 1) of y[g], stored
// [g][level-1][N].
struct ModdownRescaleMap {
  const uint64_t* acc;
  uint64_t* y;
  const double2* mr_hat;
  uint32_t level, E, alpha, rows, n;  // alpha = number of digits (special primes + 1)
  const int8_t* mr_bytes;  // matrix-core operands of digits 0..7 (LevelTables::mr_bytes), or null
  __device__ uint32_t aj(uint32_t) const { return alpha; }
  __device__ uint32_t targets(uint32_t) const { return rows; }
  __device__ uint32_t row(uint32_t, uint32_t t) const { return t; }
  __device__ uint32_t prime(uint32_t r) const { return r; }
  __device__ const double* digits(uint32_t g) const {
    return reinterpret_cast<const double*>(acc + ((size_t)g * E + level - 1) * n);
  }
  __device__ const double2* hat(uint32_t, uint32_t r) const { return mr_hat + (size_t)r * alpha; }
  __device__ uint64_t* out(uint32_t g, uint32_t r) const {
    return y + ((size_t)g * (level - 1) + r) * n;
  }
  __device__ const int8_t* bytes(uint32_t, uint32_t r) const { return mr_bytes + (size_t)r * 512; }
};

// Rescale lift: group g = 2 b + t (component t of ciphertext b), one digit =
// the centred last limb v[g] (|v| < q_last / 2), weight 1 for every target,
// targets = rows 0 .. rows-1 of w[g]: each target row gets v mod q_i.
struct RescaleMap {
  const double* v;
  uint64_t* w;
  const double2* one;  // {1, 1/q_i}
  uint32_t last, rows, n;
  static constexpr uint32_t alpha = 1;
  __device__ uint32_t aj(uint32_t) const { return 1; }
  __device__ uint32_t targets(uint32_t) const { return rows; }
  __device__ uint32_t row(uint32_t, uint32_t t) const { return t; }
  __device__ uint32_t prime(uint32_t r) const { return r; }
  __device__ const double* digits(uint32_t g) const { return v + (size_t)g * n; }
  __device__ const double2* hat(uint32_t, uint32_t r) const { return one + r; }
  __device__ uint64_t* out(uint32_t g, uint32_t r) const { return w + ((size_t)g * last + r) * n; }
};

// ------------------------- basis conversion on the matrix cores (N = 2^16)

typedef int v4i __attribute__((ext_vector_type(4)));

// Balanced base-256 digits of an integer-valued x, |x| < 2^49, as 8 signed
// bytes (the top one zero): the bytes of x + B, B = 0x80 in each of the low
// seven bytes, each less 128 (x + 1.5 2^52 holds x in its low bits).
__device__ __forceinline__ uint64_t bal_bytes(double x) {
  const int64_t xi = __double_as_longlong(x + 6755399441055744.0) - 0x4338000000000000ll;
  return (uint64_t)(xi + 0x0080808080808080ll) ^ 0x0080808080808080ull;
}

// The conversion of k_bconv_outer for N = 2^16 and digits of at most 8
// primes (a ninth source, for ModDown merged with the rescale, as one
// Shoup product per value on the VALU), as an integer matrix product.  With x_a = sum_s x_a^s 256^s and
// c_(a,s) = 256^s hat_a mod m = sum_tau c^tau_(a,s) 256^tau (balanced
// base-256 digits, LevelTables::mu_bytes),
//     y = sum_a x_a hat_a = sum_tau 256^tau Q_tau  (mod m),
//     Q_tau = sum_(a,s) x_a^s c^tau_(a,s),
// an exact int32 (56 products of magnitude <= 2^14).  A wavefront owns the
// 16 columns c0 .. c0 + 15 of the outer pass (values c0 + u + 4096 m) for
// every target of its group.  Per quad of targets and index m, two
// 16 x 16 x 64 int8 products (rows: 4 targets x tau 0..3, then tau 4..7;
// columns: u; k: 8 sources x 8 digit bytes) give every Q, so that lane
// (g, u) ends up with y of target g at c0 + u + 4096 m for all 16 m: the
// column of the outer pass, which then runs in registers as in
// k_bconv_outer.
template <class Map, bool NINTH>
__device__ __forceinline__ void bconv_mfma(const Map& map, const PrimeK* __restrict__ pk,
                                           const double2* __restrict__ twf) {
  constexpr uint32_t n = 1u << 16, LOGM = 4, M = 16;
  const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint32_t lg = lane >> 4, col = lane & 15;
  const uint32_t g = blockIdx.z;
  const uint32_t c = (blockIdx.x * (kThreads / 64) + wave) * 16 + col;  // this lane's column
  const uint32_t aj = map.aj(g), nt = map.targets(g);
  // a ninth digit source (ModDown merged with the rescale: q_{l-1} and eight
  // special primes) is added on the VALU
  const double* d8 = map.digits(g) + (size_t)8 * n + c;  // read only with NINTH (aj = 9)
  // B operands: column col of product m holds value c + 4096 m of sources
  // 2 lg (bytes 0..7) and 2 lg + 1 (bytes 8..15); a source past the digit
  // reads a valid row and contributes zero
  v4i b[16];
  {
    const double* dig = map.digits(g);
    const uint32_t a0 = 2 * lg, a1 = a0 + 1;
    const double* r0 = dig + (size_t)min(a0, aj - 1) * n + c;
    const double* r1 = dig + (size_t)min(a1, aj - 1) * n + c;
    const uint64_t k0 = a0 < aj ? ~0ull : 0ull, k1 = a1 < aj ? ~0ull : 0ull;
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const uint64_t p0 = bal_bytes(r0[kBlock * m]) & k0, p1 = bal_bytes(r1[kBlock * m]) & k1;
      b[m] = v4i{(int)(uint32_t)p0, (int)(uint32_t)(p0 >> 32), (int)(uint32_t)p1,
                 (int)(uint32_t)(p1 >> 32)};
    }
  }
  for (uint32_t q0 = 0; q0 < nt; q0 += 4) {
    // A operands: product row col = target q0 + col / 4, digit tau = col % 4
    // (first product) or 4 + col % 4 (second)
    const int8_t* tb = map.bytes(g, map.row(g, min(q0 + col / 4, nt - 1)));
    const v4i alo = *reinterpret_cast<const v4i*>(tb + ((col % 4) * 4 + lg) * 16);
    const v4i ahi = *reinterpret_cast<const v4i*>(tb + ((4 + col % 4) * 4 + lg) * 16);
    // this lane's results: target q0 + lg (rows 4 lg .. 4 lg + 3 of each
    // product); in a partial last quad the idle lane groups still join the
    // products (a product needs the whole wavefront) and store nothing
    const uint32_t tt = q0 + lg;
    const uint32_t trow = map.row(g, min(tt, nt - 1));
    const uint32_t prime = map.prime(trow);
    const double q = pk[prime].q, qinv = pk[prime].qinv, k32 = 4294967296.0 * qinv;
    double2 h8{0.0, 0.0};
    if constexpr (NINTH) h8 = map.hat(g, trow)[8];
    const v4i zero = {0, 0, 0, 0};
    double x[16];
#pragma unroll
    for (int m = 0; m < 16; ++m) {
      const v4i dl = __builtin_amdgcn_mfma_i32_16x16x64_i8(alo, b[m], zero, 0, 0, 0);
      const v4i dh = __builtin_amdgcn_mfma_i32_16x16x64_i8(ahi, b[m], zero, 0, 0, 0);
      // R = hi 2^32 + lo exactly (|lo| < 2^45, |hi| < 2^37), each |Q_tau| <=
      // 64 * 2^14 = 2^20, so digit pairs Q_t + 256 Q_t+1 still fit an int32
      // and are combined before the conversion to fp64; y = R - c q with
      // c = round(R / q), formed exactly (the fma's result is below 2^51)
      const double lo = __builtin_fma((double)(dl[2] + dl[3] * 256), 65536.0,
                                      (double)(dl[0] + dl[1] * 256));
      const double hi = __builtin_fma((double)dh[2], 65536.0, (double)(dh[0] + dh[1] * 256));
      const double cq = __builtin_rint(__builtin_fma(hi, k32, lo * qinv));
      double r = __builtin_fma(-cq, q, hi * 4294967296.0) + lo;
      if constexpr (NINTH) r += mm_shoup(d8[kBlock * m], h8.x, h8.y, q);  // |r| < 1.2 q
      x[m] = red_bal(r, q, qinv);
      // consume each pair of products here: otherwise the combination sinks
      // below the branch on tt and all 32 products (128 registers of
      // results) are held at once
      asm volatile("" : "+v"(x[m]));
    }
    if (tt >= nt) continue;
    const double2* tw = twf + (size_t)prime * n;
#pragma unroll
    for (int s = 0; s < LOGM; ++s) {
      const int H = M >> (s + 1);
#pragma unroll
      for (int m = 0; m < M; ++m) {
        if (m & H) continue;
        const double2 w = tw[(1 << s) + (m >> (LOGM - s))];
        const double u = (s % 2 == 0) ? red_bal(x[m], q, qinv) : x[m];
        const double v = mm_shoup(x[m + H], w.x, w.y, q);
        x[m] = u + v;
        x[m + H] = u - v;
      }
    }
    double* outd = reinterpret_cast<double*>(map.out(g, map.row(g, tt)));
#pragma unroll
    for (int m = 0; m < 16; ++m) outd[c + kBlock * m] = x[m];
  }
}

// Three waves per SIMD fit without spilling; the ninth-digit variant keeps
// two (its extra loads would spill at three).
template <class Map>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(3))) void k_bconv_mfma(
    Map map, const PrimeK* __restrict__ pk, const double2* __restrict__ twf) {
  bconv_mfma<Map, false>(map, pk, twf);
}

template <class Map>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void k_bconv_mfma9(
    Map map, const PrimeK* __restrict__ pk, const double2* __restrict__ twf) {
  bconv_mfma<Map, true>(map, pk, twf);
}

// ------------------------------------------------------------- inner pass

// The last 12 forward stages on block B (offset of its first value) of
// `row`: on return thread t holds the values at block positions 16 t + r in
// x[r].  Uses all of `lds`; the caller needs a barrier before touching it
// again unless it only writes the words it is handed (positions 16 t + r).
// Thread t's values t + 256 r of block B: uint64 residues (SINGLE) or the
// outer pass's fp64 intermediate.
template <bool SINGLE>
__device__ __forceinline__ void fwd_load(const uint64_t* row, uint32_t B, double (&x)[16]) {
  const uint32_t t = threadIdx.x;
  if constexpr (SINGLE) {
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = u2d(row[B + t + 256 * r]);
  } else {
    const double* src = reinterpret_cast<const double*>(row) + B + t;
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = src[256 * r];
  }
}

// The 12 stages on values already loaded by fwd_load; lt: the block's
// staged twiddles (visible to every thread), b: psi_rev[(N + B) / 2 + 8 t].
__device__ __forceinline__ void fwd_transform(const double2* lt, double b, double q, double qinv,
                                              double* lds, double (&x)[16]) {
  const uint32_t t = threadIdx.x, a = t >> 4, bb = t & 15;
  // bits 11..8
  ct_st<8, true>(x, TwL{lt, 0}, q, qinv);
  ct_st<4, false>(x, TwL{lt, 1}, q, qinv);
  ct_st<2, true>(x, TwL{lt, 3}, q, qinv);
  ct_st<1, false>(x, TwL{lt, 7}, q, qinv);
#pragma unroll
  for (int r = 0; r < 16; ++r) lds[lds_row(t, r)] = x[r];
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = lds[lds_mid(a, bb, r)];
  // bits 7..4
  ct_st<8, true>(x, TwL{lt, 15 + a}, q, qinv);
  ct_st<4, false>(x, TwL{lt, 31 + 2 * a}, q, qinv);
  ct_st<2, true>(x, TwL{lt, 63 + 4 * a}, q, qinv);
  ct_st<1, false>(x, TwL{lt, 127 + 8 * a}, q, qinv);
#pragma unroll
  for (int r = 0; r < 16; ++r) lds[lds_mid(a, bb, r)] = x[r];
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = lds[lds_col(t, r)];
  // bits 3..0
  const double b2 = sq_bal(b, q, qinv), b4 = sq_bal(b2, q, qinv);
  ct_st<8, true>(x, TwGen{sq_bal(b4, q, qinv), lt + 255, q, qinv}, q, qinv);
  ct_st<4, false>(x, TwGen{b4, lt + 255, q, qinv}, q, qinv);
  ct_st<2, true>(x, TwGen{b2, lt + 255, q, qinv}, q, qinv);
  ct_st<1, false>(x, TwGen{b, lt + 255, q, qinv}, q, qinv);
}

// An epilogue with nothing to load ahead of the transform.
struct NoPre {};

// Forward 4096-point blocks.  Thread t starts with values t + 256 r (bits
// 11..8 in registers), moves to a*256 + 16 r + b (a = t/16, b = t%16; bits
// 7..4) and to 16 t + r (bits 3..0); fwd_transform ends there.  Each transpose
// writes exactly the LDS words the thread read in the previous one, so only
// the reads need a barrier.  The kernel hands values t + 256 r to the
// epilogue.
//
// SINGLE: N = 4096, the pass reads uint64 residues; otherwise it reads the
// outer pass's fp64 intermediate.  No global load is waited on inside the
// transform: the block's twiddles of bits 11..4 are staged in LDS with the
// data loads, those of bits 3..0 generated from one loaded power.
template <bool SINGLE, class Epi>
__global__ __launch_bounds__(kThreads) void k_fwd_inner(RowSel rs, uint32_t log_n,
                                                        const PrimeK* __restrict__ pk,
                                                        const double2* __restrict__ twf,
                                                        const double* __restrict__ tw3, Epi epi) {
  __shared__ double lds[kLds];
  __shared__ double2 lt[kTwL];
  if (rs.skip()) return;
  const uint32_t n = 1u << log_n;
  const uint32_t prime = rs.prime();
  const double q = pk[prime].q, qinv = pk[prime].qinv;
  uint64_t* row = rs.row();
  const uint32_t t = threadIdx.x;
  const uint32_t B = blockIdx.x * kBlock;
  const double2* tw = twf + (size_t)prime * n;
  if (t < 255) lt[t] = block_twiddle(tw, n + B, t);
  if (t < 7) lt[255 + t] = tw[t + 1];
  // psi_rev[(N + B) / 2 + 8 t]
  const double b = tw3[((size_t)prime * (n / kBlock) + blockIdx.x) * kThreads + t];
  // operands of the epilogue loaded before the transform, so that their
  // latency overlaps the butterflies
  const typename Epi::Pre pv = epi.pre(B + t, n);
  double x[16];
  fwd_load<SINGLE>(row, B, x);
  __syncthreads();
  fwd_transform(lt, b, q, qinv, lds, x);
#pragma unroll
  for (int r = 0; r < 16; ++r) lds[lds_col(t, r)] = x[r];
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = lds[lds_row(t, r)];
  epi(row, B + t, x, q, qinv, n, pv);
}

// Epilogue of the forward transform: canonical residues, value r at k0 + 256 r.
struct StoreResidues {
  using Pre = NoPre;
  __device__ __forceinline__ Pre pre(uint32_t, uint32_t) const { return {}; }
  __device__ __forceinline__ void operator()(uint64_t* row, uint32_t k0, const double (&x)[16],
                                             double q, double qinv, uint32_t, Pre) const {
#pragma unroll
    for (int r = 0; r < 16; ++r) row[k0 + 256 * r] = to_res(x[r], q, qinv);
  }
};

// 16 consecutive residues at p (two 16-byte loads per pair).
__device__ __forceinline__ void load16(const uint64_t* p, double (&x)[16]) {
  const ulonglong2* v = reinterpret_cast<const ulonglong2*>(p);
#pragma unroll
  for (int r = 0; r < 16; r += 2) {
    const ulonglong2 w = v[r / 2];
    x[r] = u2d(w.x);
    x[r + 1] = u2d(w.y);
  }
}

// Source of the inverse inner pass: the row itself (in place).
struct LoadRow {
  __device__ __forceinline__ void operator()(const uint64_t* row, uint32_t off, double (&x)[16],
                                             double, double) const {
    load16(row + off, x);
  }
};

// Source of the inverse inner pass: row blockIdx.z of source blockIdx.y of a
// key-switch table (out of place; the row receives the result).  A product
// source (src_y set) is formed here, x y mod q in (-q/2, q/2] (balanced
// values sit inside the inverse butterflies' input bound).
struct LoadSources {
  KsTable tab;
  __device__ __forceinline__ void operator()(const uint64_t*, uint32_t off, double (&x)[16],
                                             double q, double qinv) const {
    const size_t o = (size_t)blockIdx.z * tab.src_stride[blockIdx.y] + off;
    load16(tab.src_in[blockIdx.y] + o, x);
    if (const uint64_t* y = tab.src_y[blockIdx.y]) {
      double z[16];
      load16(y + o, z);
#pragma unroll
      for (int r = 0; r < 16; ++r) x[r] = mm_var(x[r], z[r], q, qinv);
    }
  }
};

// Inverse 4096-point blocks: the mirror image of k_fwd_inner (twiddles of
// bits 11..4 staged in LDS, those of bits 3..0 generated).  Reads uint64
// residues (16 consecutive values per thread), writes fp64 for the outer pass
// or, if SINGLE, applies the final store St.
template <bool SINGLE, class Ld, class St>
__global__ __launch_bounds__(kThreads) void k_inv_inner(RowSel rs, uint32_t log_n,
                                                        const PrimeK* __restrict__ pk,
                                                        const double2* __restrict__ twi,
                                                        const double* __restrict__ tw3, Ld ld,
                                                        St st) {
  __shared__ double lds[kLds];
  __shared__ double2 lt[kTwL];
  if (rs.skip()) return;
  const uint32_t n = 1u << log_n;
  const uint32_t prime = rs.prime();
  const PrimeK P = pk[prime];
  const double q = P.q, qinv = P.qinv;
  const double2* tw = twi + (size_t)prime * n;
  uint64_t* row = rs.row();
  const uint32_t t = threadIdx.x, a = t >> 4, b = t & 15;
  const uint32_t B = blockIdx.x * kBlock;
  if (t < 255) lt[t] = block_twiddle(tw, n + B, t);
  if (t < 7) lt[255 + t] = tw[t + 1];
  // psi_rev[(N + B) / 2 + 8 t] (inverse powers)
  const double b1 = tw3[((size_t)prime * (n / kBlock) + blockIdx.x) * kThreads + t];
  double x[16];
  ld(row, B + 16 * t, x, q, qinv);
  __syncthreads();
  // bits 3..0
  const double b2 = sq_bal(b1, q, qinv), b4 = sq_bal(b2, q, qinv);
  gs_st<1, true>(x, TwGen{b1, lt + 255, q, qinv}, q, qinv);
  gs_st<2, false>(x, TwGen{b2, lt + 255, q, qinv}, q, qinv);
  gs_st<4, true>(x, TwGen{b4, lt + 255, q, qinv}, q, qinv);
  gs_st<8, false>(x, TwGen{sq_bal(b4, q, qinv), lt + 255, q, qinv}, q, qinv);
#pragma unroll
  for (int r = 0; r < 16; ++r) lds[lds_col(t, r)] = x[r];
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = lds[lds_mid(a, b, r)];
  // bits 7..4
  gs_st<1, true>(x, TwL{lt, 127 + 8 * a}, q, qinv);
  gs_st<2, false>(x, TwL{lt, 63 + 4 * a}, q, qinv);
  gs_st<4, true>(x, TwL{lt, 31 + 2 * a}, q, qinv);
  gs_st<8, false>(x, TwL{lt, 15 + a}, q, qinv);
#pragma unroll
  for (int r = 0; r < 16; ++r) lds[lds_mid(a, b, r)] = x[r];
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = lds[lds_row(t, r)];
  // bits 11..8
  gs_st<1, true>(x, TwL{lt, 7}, q, qinv);
  gs_st<2, false>(x, TwL{lt, 3}, q, qinv);
  gs_st<4, true>(x, TwL{lt, 1}, q, qinv);
  gs_st<8, false>(x, TwL{lt, 0}, q, qinv);
  if constexpr (SINGLE) {
#pragma unroll
    for (int r = 0; r < 16; ++r) st(row, B + t + 256 * r, x[r], P);
  } else {
    double* dst = reinterpret_cast<double*>(row) + B + t;
#pragma unroll
    for (int r = 0; r < 16; ++r) dst[256 * r] = x[r];
  }
}

}  // namespace

// Epilogue fusing the key-switch combine into the forward transform of the
// ModDown conversion y: for u = 2*job + t (blockIdx.y) and limb i
// (blockIdx.z), out_job[i][t] = (acc[u][i] - NTT(y)[u][i]) * P^-1 + adds,
// with the adds of the job table (sigma_g-permuted `add`, plain `add2`).  If
// tab.fold the inner product has already stored acc * P^-1 + add, and only
// NTT(y) * P^-1 is subtracted here.  With qlinv (ModDown merged with the
// rescale, fold only) the difference is also multiplied by q_{level-1}^-1
// before add2 is added.
struct KsCombine {
  KsTable tab;
  const uint64_t* acc;
  const double2* pinv;
  const double2* qlinv;
  uint32_t level, alpha, log_n;
  struct Pre {
    uint64_t a[16];  // acc[u][i] at k0 + 256 r
  };
  __device__ __forceinline__ Pre pre(uint32_t k0, uint32_t n) const {
    const uint64_t* a = acc + ((size_t)blockIdx.y * (level + alpha) + blockIdx.z) * n + k0;
    Pre p;
#pragma unroll
    for (int r = 0; r < 16; ++r) p.a[r] = a[256 * r];
    return p;
  }
  __device__ __forceinline__ void operator()(uint64_t*, uint32_t k0, const double (&x)[16],
                                             double q, double qinv, uint32_t n,
                                             const Pre& pa) const {
    const uint32_t u = blockIdx.y, i = blockIdx.z, job = u >> 1, t = u & 1;
    const double2 f = pinv[i];
    const size_t o = ((size_t)2 * i + t) * n;
    const bool use_add = (tab.add_mask[job] >> t) & 1u;
    const uint32_t g = tab.add_galois[job];
    const uint64_t* add = use_add ? tab.add[job] + o : nullptr;
    const uint64_t* add2 = tab.add2[job];
    uint64_t* out = tab.out[job] + o;
    if (tab.fold) {
      const double2 h = qlinv ? qlinv[i] : double2{0.0, 0.0};
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const uint32_t k = k0 + 256 * r;
        double v = u2d(pa.a[r]) - mm_shoup(x[r], f.x, f.y, q);  // |v| < 2.5 q
        if (qlinv) v = mm_shoup(v, h.x, h.y, q);
        if (add2) v += u2d(add2[o + k]);
        out[k] = to_res(v, q, qinv);
      }
      return;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const uint32_t k = k0 + 256 * r;
      double v = mm_shoup(u2d(pa.a[r]) - x[r], f.x, f.y, q);
      if (use_add) v += u2d(add[g ? galois_src(k, g, log_n) : k]);
      if (add2) v += u2d(add2[o + k]);
      out[k] = to_res(v, q, qinv);
    }
  }
};

// Epilogue fusing the rescale combine into the forward transform of the
// lifted last limbs: for u = 2 b + t (blockIdx.y) and limb i (blockIdx.z),
// out_b[i][t] = (in_b[i][t] - NTT(w)[u][i]) * q_last^-1 (+ add_b[i][t]).
// out_b may alias in_b or add_b (same element, same thread).
struct RsCombine {
  RsTable tab;
  const double2* qlinv;
  using Pre = NoPre;
  __device__ __forceinline__ Pre pre(uint32_t, uint32_t) const { return {}; }
  __device__ __forceinline__ void operator()(uint64_t*, uint32_t k0, const double (&x)[16],
                                             double q, double qinv, uint32_t n, Pre) const {
    const uint32_t u = blockIdx.y, i = blockIdx.z, b = u >> 1, t = u & 1;
    const double2 f = qlinv[i];
    const size_t o = ((size_t)2 * i + t) * n;
    const uint64_t* in = tab.in[b] + o;
    const uint64_t* add = tab.add[b];
    uint64_t* out = tab.out[b] + o;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const uint32_t k = k0 + 256 * r;
      double v = mm_shoup(u2d(in[k]) - x[r], f.x, f.y, q);
      if (add) v += u2d(add[o + k]);
      out[k] = to_res(v, q, qinv);
    }
  }
};

namespace {

hipError_t launch_fwd_outer(const Context* c, const RowSel& rs, uint32_t batch, uint32_t limbs,
                            hipStream_t s) {
  const dim3 grid(c->n / kBlock, batch, limbs), blk(kThreads);
  const double2* tw = c->d_tw_fwd;
  switch (c->log_n) {
    case 12: return hipSuccess;
    case 13: hipLaunchKernelGGL(k_fwd_outer<1>, grid, blk, 0, s, rs, c->log_n, c->d_pk, tw); break;
    case 14: hipLaunchKernelGGL(k_fwd_outer<2>, grid, blk, 0, s, rs, c->log_n, c->d_pk, tw); break;
    case 15: hipLaunchKernelGGL(k_fwd_outer<3>, grid, blk, 0, s, rs, c->log_n, c->d_pk, tw); break;
    case 16: hipLaunchKernelGGL(k_fwd_outer<4>, grid, blk, 0, s, rs, c->log_n, c->d_pk, tw); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class St>
hipError_t launch_inv_outer(const Context* c, const RowSel& rs, uint32_t batch, uint32_t limbs,
                            const St& st, hipStream_t s) {
  const dim3 grid(c->n / kBlock, batch, limbs), blk(kThreads);
  const double2* tw = c->d_tw_inv;
  switch (c->log_n) {
    case 12: return hipSuccess;
    case 13: k_inv_outer<1, St><<<grid, blk, 0, s>>>(rs, c->log_n, c->d_pk, tw, st); break;
    case 14: k_inv_outer<2, St><<<grid, blk, 0, s>>>(rs, c->log_n, c->d_pk, tw, st); break;
    case 15: k_inv_outer<3, St><<<grid, blk, 0, s>>>(rs, c->log_n, c->d_pk, tw, st); break;
    case 16: k_inv_outer<4, St><<<grid, blk, 0, s>>>(rs, c->log_n, c->d_pk, tw, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <class Epi>
hipError_t launch_fwd_inner(const Context* c, const RowSel& rs, uint32_t batch, uint32_t limbs,
                            const Epi& epi, hipStream_t s) {
  const uint32_t nblk = c->n / kBlock;
  const dim3 blk(kThreads);
  if (c->log_n == 12) {
    k_fwd_inner<true, Epi><<<dim3(nblk, batch, limbs), blk, 0, s>>>(
        rs, c->log_n, c->d_pk, c->d_tw_fwd, c->d_tw3_fwd, epi);
  } else {
    k_fwd_inner<false, Epi><<<dim3(nblk, batch, limbs), blk, 0, s>>>(
        rs, c->log_n, c->d_pk, c->d_tw_fwd, c->d_tw3_fwd, epi);
  }
  return hipGetLastError();
}

// Inverse transform: inner pass (reading through Ld), then the outer pass; St
// is the final store of whichever pass is last.
template <class Ld, class St>
hipError_t launch_inverse(const Context* c, const RowSel& rs, uint32_t batch, uint32_t limbs,
                          const Ld& ld, const St& st, hipStream_t s) {
  const dim3 grid(c->n / kBlock, batch, limbs), blk(kThreads);
  if (c->log_n == 12)
    k_inv_inner<true, Ld, St><<<grid, blk, 0, s>>>(rs, c->log_n, c->d_pk, c->d_tw_inv,
                                                    c->d_tw3_inv, ld, st);
  else
    k_inv_inner<false, Ld, St><<<grid, blk, 0, s>>>(rs, c->log_n, c->d_pk, c->d_tw_inv,
                                                     c->d_tw3_inv, ld, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_inv_outer(c, rs, batch, limbs, st, s);
}

constexpr int kBconvTargets = 3;

// The matrix-core conversion serves N = 2^16 for the maps that carry its
// operand tables (ModUp, ModDown and ModDown merged with the rescale, with
// digits of at most 8 primes plus at most one on the VALU).
template <class Map>
constexpr bool kMfmaMap = false;
template <>
constexpr bool kMfmaMap<ModupMap> = true;
template <>
constexpr bool kMfmaMap<ModdownMap> = true;
template <>
constexpr bool kMfmaMap<ModdownRescaleMap> = true;

__host__ inline const int8_t* mfma_bytes(const ModupMap& m) { return m.mu_bytes; }
__host__ inline const int8_t* mfma_bytes(const ModdownMap& m) { return m.md_bytes; }
__host__ inline const int8_t* mfma_bytes(const ModdownRescaleMap& m) {
  return m.alpha <= 9 ? m.mr_bytes : nullptr;  // at most one digit past the eight
}

template <class Map>
hipError_t launch_bconv_outer(const Context* c, const Map& map, uint32_t targets, uint32_t groups,
                              hipStream_t s) {
  constexpr int T = kBconvTargets;
  if constexpr (kMfmaMap<Map>) {
    if (c->log_n == 16 && mfma_bytes(map)) {
      const dim3 grid(kBlock / (16 * (kThreads / 64)), 1, groups);
      if constexpr (std::is_same_v<Map, ModdownRescaleMap>) {
        if (map.alpha > 8) {  // q_{l-1} and eight special primes
          k_bconv_mfma9<Map><<<grid, kThreads, 0, s>>>(map, c->d_pk, c->d_tw_fwd);
          return hipGetLastError();
        }
      }
      k_bconv_mfma<Map><<<grid, kThreads, 0, s>>>(map, c->d_pk, c->d_tw_fwd);
      return hipGetLastError();
    }
  }
  const dim3 grid(c->n / kBlock, (targets + T - 1) / T, groups), blk(kThreads);
  const double2* tw = c->d_tw_fwd;
  switch (c->log_n) {
    case 12: k_bconv_outer<0, T, Map><<<grid, blk, 0, s>>>(map, c->log_n, c->d_pk, tw); break;
    case 13: k_bconv_outer<1, T, Map><<<grid, blk, 0, s>>>(map, c->log_n, c->d_pk, tw); break;
    case 14: k_bconv_outer<2, T, Map><<<grid, blk, 0, s>>>(map, c->log_n, c->d_pk, tw); break;
    case 15: k_bconv_outer<3, T, Map><<<grid, blk, 0, s>>>(map, c->log_n, c->d_pk, tw); break;
    case 16: k_bconv_outer<4, T, Map><<<grid, blk, 0, s>>>(map, c->log_n, c->d_pk, tw); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

// Inverse transform of the first `level` rows of each key-switch source into
// cc[s][level][N] (out of place: the first pass reads the sources directly),
// stored as the centred ModUp digits [N^-1 (Q_D/q_i)^-1 x]_{q_i} (fp64);
// f = LevelTables::mu_inv_n.
hipError_t launch_ntt_inv_sources(const Context* c, const KsTable& tab, uint32_t nsrc,
                                  uint64_t* cc, uint32_t level, const double2* f, hipStream_t s) {
  RowSel rs{cc, (size_t)level * c->n, (size_t)c->n, 0, level, 0, 0, 0, 0};
  return launch_inverse(c, rs, nsrc, level, LoadSources{tab}, InvDigit{f}, s);
}

// Rescale, step 1: inverse transform of nrows single rows under prime
// `last`, row r read from tab.src_in[r], stored into v[r][N] as the centred
// coefficients [N^-1 x]_{q_last} (fp64; ninv = {N^-1 mod q_last, /q_last}).
hipError_t launch_ntt_inv_rescale_last(const Context* c, const KsTable& tab, uint32_t nrows,
                                       uint64_t* v, uint32_t last, const double2* ninv,
                                       hipStream_t s) {
  RowSel rs{v, (size_t)c->n, (size_t)c->n, last, 1, 0, 0, 0, 0};
  return launch_inverse(c, rs, nrows, 1, LoadSources{tab}, InvDigit{ninv}, s);
}

// Rescale, step 2: each centred last limb lifted to rows 0 .. rows-1 (a
// conversion with one digit and weight 1) fused with their first forward
// pass, into w[g][last][N].
hipError_t launch_rescale_outer(const Context* c, const uint64_t* v, uint64_t* w, uint32_t groups,
                                uint32_t last, uint32_t rows, const double2* one, hipStream_t s) {
  const RescaleMap map{reinterpret_cast<const double*>(v), w, one, last, rows, c->n};
  return launch_bconv_outer(c, map, rows, groups, s);
}

// Rescale, step 3: second forward pass of w with the combine
// out_b = (in_b - w) * q_last^-1 (+ add_b) as the epilogue, first `rows` limbs.
hipError_t launch_ntt_fwd_rs_combine(const Context* c, uint64_t* w, uint32_t count, uint32_t last,
                                     uint32_t rows, const RsTable& tab, const double2* qlinv,
                                     hipStream_t s) {
  RowSel rs{w, (size_t)last * c->n, (size_t)c->n, 0, rows, 0, 0, 0, 0};
  return launch_fwd_inner(c, rs, 2 * count, rows, RsCombine{tab, qlinv}, s);
}

// Inverse transform of the rows rs selects (in place), stored as centred
// digits [N^-1 f_i x]_{q_i} (fp64), f per limb.
hipError_t launch_ntt_inv_digits(const Context* c, const RowSel& rs, uint32_t batch,
                                 uint32_t limbs, const double2* f, hipStream_t s) {
  return launch_inverse(c, rs, batch, limbs, LoadRow{}, InvDigit{f}, s);
}

// ModUp of every source (digits from launch_ntt_inv_sources) fused with the
// first forward pass of the extended rows (own-digit rows are not written).
hipError_t launch_modup_outer(const Context* c, const LevelTables& T, const uint64_t* cc,
                              uint64_t* ext, uint32_t nsrc, uint32_t level, hipStream_t s) {
  const uint32_t dnum_l = (level + c->alpha - 1) / c->alpha;
  const uint32_t aj_min = level - (dnum_l - 1) * c->alpha;
  const ModupMap map{reinterpret_cast<const double*>(cc), ext, T.mu_hat, level, c->L, c->alpha,
                     dnum_l, c->n, T.mu_bytes};
  return launch_bconv_outer(c, map, level + c->alpha - aj_min, nsrc * dnum_l, s);
}

// ModDown conversion of the special-prime rows of acc (digits from
// launch_ntt_inv_digits) fused with the first forward pass of y.
hipError_t launch_moddown_outer(const Context* c, const LevelTables& T, const uint64_t* acc,
                                uint64_t* y, uint32_t njobs, uint32_t level, hipStream_t s) {
  const ModdownMap map{acc, y, T.md_hat, level, c->alpha, c->n, T.md_bytes};
  return launch_bconv_outer(c, map, level, 2 * njobs, s);
}

// Second forward pass of rows whose first pass has run (launch_modup_outer).
hipError_t launch_ntt_fwd_inner_rows(const Context* c, const RowSel& rs, uint32_t batch,
                                     uint32_t limbs, hipStream_t s) {
  return launch_fwd_inner(c, rs, batch, limbs, StoreResidues{}, s);
}

// ModDown merged with the rescale: conversion of the alpha + 1 digit rows of
// acc (launch_ntt_inv_digits with mr_inv_n) to rows 0 .. rows-1, fused with
// the first forward pass of y[2*njobs][level-1][N].
hipError_t launch_moddown_rescale_outer(const Context* c, const LevelTables& T,
                                        const uint64_t* acc, uint64_t* y, uint32_t njobs,
                                        uint32_t level, uint32_t rows, hipStream_t s) {
  const ModdownRescaleMap map{acc, y, T.mr_hat, level, level + c->alpha, c->alpha + 1, rows,
                              c->n, T.mr_bytes};
  return launch_bconv_outer(c, map, rows, 2 * njobs, s);
}

// Second forward pass of the ModDown conversions y[2*njobs][ystride][N]
// (first pass: launch_moddown_outer or launch_moddown_rescale_outer) with the
// key-switch combine as the epilogue; writes rows 0 .. rows-1 of the jobs'
// outputs.  qlinv: null, or q_{level-1}^-1 per row (merged rescale).
hipError_t launch_ntt_fwd_ks_combine(const Context* c, uint64_t* y, uint32_t njobs,
                                     uint32_t level, uint32_t rows, uint32_t ystride,
                                     const KsTable& tab, const uint64_t* acc,
                                     const double2* pinv, const double2* qlinv, hipStream_t s) {
  RowSel rs{y, (size_t)ystride * c->n, (size_t)c->n, 0, rows, 0, 0, 0, 0};
  return launch_fwd_inner(c, rs, 2 * njobs, rows,
                          KsCombine{tab, acc, pinv, qlinv, level, c->alpha, c->log_n}, s);
}

// (Splitting a large batch into cache-sized chunks, so that the second pass
// would read the first pass's output back from the 256 MB Infinity Cache,
// measured no faster on MI355X than one launch per pass over the whole batch.)
hipError_t launch_ntt_rows(const Context* c, const RowSel& rs, uint32_t batch, uint32_t limbs,
                           bool inverse, hipStream_t s) {
  if (inverse) return launch_inverse(c, rs, batch, limbs, LoadRow{}, InvCanon{}, s);
  hipError_t e = launch_fwd_outer(c, rs, batch, limbs, s);
  if (e != hipSuccess) return e;
  return launch_fwd_inner(c, rs, batch, limbs, StoreResidues{}, s);
}

hipError_t launch_ntt(const Context* c, uint64_t* d, uint32_t batch, size_t batch_stride,
                      uint32_t limbs, size_t limb_stride, uint32_t prime0, bool inverse,
                      hipStream_t s) {
  RowSel rs{d, batch_stride, limb_stride, prime0, limbs, 0, 0, 0, 0};
  return launch_ntt_rows(c, rs, batch, limbs, inverse, s);
}

}  // namespace fesc
