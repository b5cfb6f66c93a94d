// Hybrid key switching (digit decomposition with special primes): ModUp by
// fast basis conversion, inner product with the switching key, ModDown.
//
// Basis conversion uses centred digits: for a digit D with product Q_D and
// x_a = [c_a * (Q_D/q_a)^-1]_{q_a} taken in (-q_a/2, q_a/2),
//     y mod m = sum_a x_a * ((Q_D/q_a) mod m)  mod m.
// With centred digits the conversion is an odd map, so it commutes with the
// signed coefficient permutations of the Galois group: ModUp once, then apply
// sigma_g to the extended digits (evaluation-form index permutation) for any
// number of rotations of the same ciphertext.
//
// Every kernel here is batched: up to kMaxBatch ModUp sources and key-switch
// jobs run in one launch (tables passed by value in the kernel arguments), so
// independent key switches fill the GPU together instead of one at a time.
// Loops over digit primes and digits are unrolled over compile-time bounds
// (alpha, dnum) with clamped indices instead of bounds branches, so that all
// loads of a loop are issued together.
//
// The transforms around these kernels carry two more steps of the pipeline
// (ntt.hip): the inverse NTT of the sources reads the callers' ciphertexts
// directly (no gather copy), and the forward NTT of the ModDown conversion y
// ends in the combine (acc - y) * P^-1 + sigma_g(c0) that writes the outputs.
//
// Extended basis at level l: rows 0..l-1 are q_0..q_{l-1}, rows l..l+alpha-1
// are p_0..p_{alpha-1} (extended prime index L + k).
#include "fesc_internal.hpp"
#include "ops.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;

// Basis-conversion launches split the target rows over gridDim.z only as far
// as needed to reach about kTargetBlocks workgroups: every split recomputes
// the centred digits of its coefficients.
constexpr uint32_t kTargetBlocks = 4096;
constexpr uint32_t kMinRowsPerZ = 4;

uint32_t row_splits(uint32_t xy_blocks, uint32_t rows) {
  uint32_t z = (kTargetBlocks + xy_blocks - 1) / xy_blocks;
  const uint32_t zmax = (rows + kMinRowsPerZ - 1) / kMinRowsPerZ;
  return z < 1 ? 1 : (z > zmax ? zmax : z);
}

__device__ __forceinline__ uint32_t ext_prime(uint32_t row, uint32_t level, uint32_t L) {
  return row < level ? row : L + (row - level);
}

// centred [v * f]_q of a canonical residue pair
__device__ __forceinline__ void centred_digit(const ulonglong2 v, const double2 f, const PrimeK& P,
                                              double& y0, double& y1) {
  y0 = center(red_full(mm_shoup(u2d(v.x), f.x, f.y, P.q), P.q, P.qinv), P.q);
  y1 = center(red_full(mm_shoup(u2d(v.y), f.x, f.y, P.q), P.q, P.qinv), P.q);
}

// sum_a x_a * h_a mod M for A terms, reduced every 8 terms; canonical result
template <int A>
__device__ __forceinline__ void conv_row(const double (&x0)[A], const double (&x1)[A],
                                         const double2* __restrict__ h, const PrimeK& M,
                                         uint64_t* dst) {
  double s0 = 0.0, s1 = 0.0;
#pragma unroll
  for (int a = 0; a < A; ++a) {
    const double2 w = h[a];
    s0 += mm_shoup(x0[a], w.x, w.y, M.q);
    s1 += mm_shoup(x1[a], w.x, w.y, M.q);
    if ((a & 7) == 7 && a + 1 < A) {
      s0 = red_bal(s0, M.q, M.qinv);
      s1 = red_bal(s1, M.q, M.qinv);
    }
  }
  ulonglong2 o;
  o.x = to_res(s0, M.q, M.qinv);
  o.y = to_res(s1, M.q, M.qinv);
  *reinterpret_cast<ulonglong2*>(dst) = o;
}

// ModUp: coefficient-form rows cc[s][0..level) -> ext[s][j][row] for every
// row outside digit j (coefficient form; transformed afterwards).
// blockIdx.y = s * dnum_l + j.  A = alpha; a short last digit (aj < A) reads
// its last row again for the missing terms and zeroes them.
template <int A>
__global__ __launch_bounds__(kThreads) void k_modup(const uint64_t* __restrict__ cc,
                                                    uint64_t* __restrict__ ext, uint32_t level,
                                                    uint32_t L, uint32_t dnum_l, uint32_t n,
                                                    const PrimeK* __restrict__ pk,
                                                    const double2* __restrict__ mu_inv,
                                                    const double2* __restrict__ mu_hat) {
  const uint32_t s = blockIdx.y / dnum_l, j = blockIdx.y % dnum_l;
  const uint32_t lo = j * A, hi = min(lo + (uint32_t)A, level), aj = hi - lo;
  const uint32_t E = level + A;
  const uint32_t k = 2 * (blockIdx.x * kThreads + threadIdx.x);
  if (k >= n) return;
  const uint64_t* src = cc + (size_t)s * level * n;
  uint64_t* dst = ext + ((size_t)s * dnum_l + j) * E * n;
  double x0[A], x1[A];
#pragma unroll
  for (int a = 0; a < A; ++a) {
    const uint32_t ac = min((uint32_t)a, aj - 1);
    const ulonglong2 v = *reinterpret_cast<const ulonglong2*>(src + (size_t)(lo + ac) * n + k);
    double y0, y1;
    centred_digit(v, mu_inv[j * A + ac], pk[lo + ac], y0, y1);
    x0[a] = (uint32_t)a < aj ? y0 : 0.0;
    x1[a] = (uint32_t)a < aj ? y1 : 0.0;
  }
  const uint32_t per = (E + gridDim.z - 1) / gridDim.z;
  const uint32_t r0 = blockIdx.z * per, r1 = min(r0 + per, E);
  for (uint32_t row = r0; row < r1; ++row) {
    if (row >= lo && row < hi) continue;
    conv_row<A>(x0, x1, mu_hat + ((size_t)j * E + row) * A, pk[ext_prime(row, level, L)],
                dst + (size_t)row * n + k);
  }
}

// Inner product with the key, sigma_g applied to the extended digits on the
// fly: acc[job][t][row][k] = sum_j d_j[row][src(k)] * key[j][prime(row)][t][k].
// Own-digit rows of d_j are the source polynomial itself.  blockIdx.z = job.
// D = number of digits at this level (compile time), A = alpha.
template <int D>
__global__ __launch_bounds__(kThreads) void k_ip(KsTable tab, const uint64_t* __restrict__ ext,
                                                 uint64_t* __restrict__ acc, uint32_t level,
                                                 uint32_t L, uint32_t alpha, uint32_t log_n,
                                                 const PrimeK* __restrict__ pk) {
  const uint32_t n = 1u << log_n;
  const uint32_t row = blockIdx.y, job = blockIdx.z;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const uint32_t E = level + alpha, KE = L + alpha;
  const uint32_t s = tab.job_src[job], galois = tab.galois[job];
  const uint64_t* key = tab.key[job];
  const uint64_t* in = tab.src_in[s];
  const size_t in_stride = tab.src_stride[s];
  const uint64_t* ex = ext + (size_t)s * D * E * n;
  const uint32_t prime = ext_prime(row, level, L);
  const PrimeK M = pk[prime];
  const uint32_t src = galois ? galois_src(k, galois, log_n) : k;
  const uint32_t own = row < level ? row / alpha : D;  // digit whose rows hold `row`
  uint64_t dv[D], kb[D], ka[D];
#pragma unroll
  for (int j = 0; j < D; ++j) {
    const uint64_t* p = (uint32_t)j == own ? in + (size_t)row * in_stride
                                           : ex + ((size_t)j * E + row) * n;
    dv[j] = p[src];
    const size_t ko = (((size_t)j * KE + prime) * 2) * n + k;
    kb[j] = key[ko];
    ka[j] = key[ko + n];
  }
  double ab = 0.0, aa = 0.0;
#pragma unroll
  for (int j = 0; j < D; ++j) {
    const double d = u2d(dv[j]);
    ab += mm_var(d, u2d(kb[j]), M.q, M.qinv);
    aa += mm_var(d, u2d(ka[j]), M.q, M.qinv);
    if ((j & 3) == 3 && j + 1 < D) {
      ab = red_bal(ab, M.q, M.qinv);
      aa = red_bal(aa, M.q, M.qinv);
    }
  }
  uint64_t* out = acc + (size_t)job * 2 * E * n;
  out[(size_t)row * n + k] = to_res(ab, M.q, M.qinv);
  out[((size_t)E + row) * n + k] = to_res(aa, M.q, M.qinv);
}

// ModDown conversion: for u = 2*job + t (blockIdx.y), the P-rows of acc[u]
// (coefficient form) -> y[u][i], i < level.  A = alpha.
template <int A>
__global__ __launch_bounds__(kThreads) void k_moddown_bconv(const uint64_t* __restrict__ acc,
                                                            uint64_t* __restrict__ y,
                                                            uint32_t level, uint32_t L,
                                                            uint32_t n,
                                                            const PrimeK* __restrict__ pk,
                                                            const double2* __restrict__ md_inv,
                                                            const double2* __restrict__ md_hat) {
  const uint32_t u = blockIdx.y;
  const uint32_t E = level + A;
  const uint32_t k = 2 * (blockIdx.x * kThreads + threadIdx.x);
  if (k >= n) return;
  double x0[A], x1[A];
#pragma unroll
  for (int a = 0; a < A; ++a) {
    const ulonglong2 v =
        *reinterpret_cast<const ulonglong2*>(acc + ((size_t)u * E + level + a) * n + k);
    centred_digit(v, md_inv[a], pk[L + a], x0[a], x1[a]);
  }
  const uint32_t per = (level + gridDim.z - 1) / gridDim.z;
  const uint32_t i0 = blockIdx.z * per, i1 = min(i0 + per, level);
  for (uint32_t i = i0; i < i1; ++i)
    conv_row<A>(x0, x1, md_hat + (size_t)i * A, pk[i], y + ((size_t)u * level + i) * n + k);
}

// Dispatch on a runtime value to a template instantiation 1..16.
template <template <int> class K, typename... Args>
void dispatch16(uint32_t a, Args&&... args) {
  switch (a) {
#define FESC_CASE(v) \
  case v: K<v>::run(args...); break;
    FESC_CASE(1) FESC_CASE(2) FESC_CASE(3) FESC_CASE(4) FESC_CASE(5) FESC_CASE(6) FESC_CASE(7)
    FESC_CASE(8) FESC_CASE(9) FESC_CASE(10) FESC_CASE(11) FESC_CASE(12) FESC_CASE(13)
    FESC_CASE(14) FESC_CASE(15) FESC_CASE(16)
#undef FESC_CASE
    default: break;
  }
}

template <int A>
struct ModupL {
  static void run(dim3 g, hipStream_t s, const uint64_t* cc, uint64_t* ext, uint32_t level,
                  uint32_t L, uint32_t dnum_l, uint32_t n, const PrimeK* pk, const double2* mi,
                  const double2* mh) {
    hipLaunchKernelGGL(k_modup<A>, g, dim3(kThreads), 0, s, cc, ext, level, L, dnum_l, n, pk, mi,
                       mh);
  }
};

template <int A>
struct ModdownL {
  static void run(dim3 g, hipStream_t s, const uint64_t* acc, uint64_t* y, uint32_t level,
                  uint32_t L, uint32_t n, const PrimeK* pk, const double2* mi,
                  const double2* mh) {
    hipLaunchKernelGGL(k_moddown_bconv<A>, g, dim3(kThreads), 0, s, acc, y, level, L, n, pk, mi,
                       mh);
  }
};

template <int D>
struct IpL {
  static void run(dim3 g, hipStream_t s, const KsTable& tab, const uint64_t* ext, uint64_t* acc,
                  uint32_t level, uint32_t L, uint32_t alpha, uint32_t log_n, const PrimeK* pk) {
    hipLaunchKernelGGL(k_ip<D>, g, dim3(kThreads), 0, s, tab, ext, acc, level, L, alpha, log_n,
                       pk);
  }
};

}  // namespace

hipError_t k_modup_launch(const Context* c, const LevelTables& T, const uint64_t* cc,
                          uint64_t* ext, uint32_t nsrc, uint32_t level, hipStream_t s) {
  const uint32_t dnum_l = (level + c->alpha - 1) / c->alpha;
  const uint32_t E = level + c->alpha;
  const uint32_t xb = (c->n / 2 + kThreads - 1) / kThreads;
  dim3 grid(xb, nsrc * dnum_l, row_splits(xb * nsrc * dnum_l, E));
  dispatch16<ModupL>(c->alpha, grid, s, cc, ext, level, c->L, dnum_l, c->n, c->d_pk, T.mu_inv,
                     T.mu_hat);
  return hipGetLastError();
}

hipError_t k_ip_launch(const Context* c, const KsTable& tab, uint32_t njobs, const uint64_t* ext,
                       uint64_t* acc, uint32_t level, hipStream_t s) {
  const uint32_t dnum_l = (level + c->alpha - 1) / c->alpha;
  if (dnum_l > 16) return hipErrorInvalidValue;
  dim3 grid((c->n + kThreads - 1) / kThreads, level + c->alpha, njobs);
  dispatch16<IpL>(dnum_l, grid, s, tab, ext, acc, level, c->L, c->alpha, c->log_n, c->d_pk);
  return hipGetLastError();
}

hipError_t k_moddown_bconv_launch(const Context* c, const LevelTables& T, const uint64_t* acc,
                                  uint64_t* y, uint32_t njobs, uint32_t level, hipStream_t s) {
  const uint32_t xb = (c->n / 2 + kThreads - 1) / kThreads;
  dim3 grid(xb, 2 * njobs, row_splits(xb * 2 * njobs, level));
  dispatch16<ModdownL>(c->alpha, grid, s, acc, y, level, c->L, c->n, c->d_pk, T.md_inv,
                       T.md_hat);
  return hipGetLastError();
}

}  // namespace fesc
