// Hybrid key switching (digit decomposition with special primes): the key
// inner product.  The rest of the pipeline lives with the transforms
// (ntt.hip), fused into their passes:
//   1. inverse NTT of each source polynomial, reading the caller's rows
//      directly; its last pass stores the centred ModUp digits
//          x_a = [c_a * (Q_D/q_a)^-1]_{q_a} in (-q_a/2, q_a/2)  (fp64);
//   2. ModUp: y mod m = sum_a x_a * ((Q_D/q_a) mod m) for every extended row
//      m outside digit D, fused with the first forward pass; second pass;
//   3. k_ip (here): acc_t = sum_j sigma_g(D_j) * key_j[t], the own-digit rows
//      of D_j being the source rows themselves;
//   4. inverse NTT of the special-prime rows of acc to centred ModDown digits,
//      the conversion to the level rows fused with the first forward pass of
//      y, and a second pass whose epilogue is the combine
//          out = (acc - y) * P^-1 + sigma_g(c0) (+ an optional addend).
// With centred digits the conversion is an odd map, so it commutes with the
// signed coefficient permutations of the Galois group: ModUp once, then apply
// sigma_g to the extended digits (evaluation-form index permutation) for any
// number of rotations of the same ciphertext.
//
// Every step is batched: up to kMaxBatch ModUp sources and key-switch jobs
// run in one launch (tables passed by value in the kernel arguments), so
// independent key switches fill the GPU together instead of one at a time.
// The digit loop of the inner product is unrolled over a compile-time dnum.
//
// Extended basis at level l: rows 0..l-1 are q_0..q_{l-1}, rows l..l+alpha-1
// are p_0..p_{alpha-1} (extended prime index L + k).
#include "fesc_internal.hpp"
#include "ops.hpp"
#include "seedkey.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t ext_prime(uint32_t row, uint32_t level, uint32_t L) {
  return row < level ? row : L + (row - level);
}

// Key-stationary inner product with sigma_g applied to the extended digits on
// the fly: for every job j of key group blockIdx.z (jobs sharing one switching
// key and Galois element g),
//     acc[j][t][row][k] = sum_d D_d(src_j)[row][gsrc(k)] * key[d][prime(row)][t][k],
// D_d(src) the ModUp digit d of the job's source, whose own-digit rows are the
// source polynomial itself.  The key values of a coefficient are loaded once
// and reused by every job of the group.  With tab.fold == 1 the level rows
// (row < level) store acc * P^-1 plus the job's addend components instead
// (the addend read through the same permutation), so that the combine only
// has to subtract y * P^-1.  With tab.fold == 2 (extended-basis outputs, no
// ModDown) every row goes to the job's output [2][level+alpha][N] and the
// level rows add the addend times P (pinv then holds P mod q_row).  A seed-expanded key (bit kg of tab.kg_seeded)
// stores only its b half; its a half is regenerated here from the seed, which
// halves the key bytes read.  D = number of digits at this level (compile
// time).
template <int D>
__global__ __launch_bounds__(kThreads) void k_ip(KsTable tab, const uint64_t* __restrict__ ext,
                                                 uint64_t* __restrict__ acc, uint32_t level,
                                                 uint32_t L, uint32_t alpha, uint32_t log_n,
                                                 const PrimeK* __restrict__ pk,
                                                 const double2* __restrict__ pinv) {
  const uint32_t n = 1u << log_n;
  const uint32_t row = blockIdx.y, kg = blockIdx.z;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  const uint32_t E = level + alpha, KE = L + alpha;
  const uint32_t j0 = tab.kg_first[kg], j1 = j0 + tab.kg_count[kg];
  const uint32_t galois = tab.galois[j0];
  const uint64_t* key = tab.key[j0];
  const uint32_t prime = ext_prime(row, level, L);
  const PrimeK M = pk[prime];
  const uint32_t src = galois ? galois_src(k, galois, log_n) : k;
  const uint32_t own = row < level ? row / alpha : D;  // digit whose rows hold `row`
  double kb[D], ka[D];
  if ((tab.kg_seeded >> kg) & 1u) {
    // seed-expanded key: b read from the compact rows, a regenerated
    const uint64_t s0 = key[0], s1 = key[1], elt = key[2];
#pragma unroll
    for (int j = 0; j < D; ++j)
      kb[j] = u2d(key[kSeedHeaderWords + ((size_t)j * KE + prime) * n + k]);
#pragma unroll
    for (int c = 0; 3 * c < D; ++c) {
      uint64_t blk[3] = {0, 0, 0};
      seeded_key_block(blk, k, prime, c, elt, s0, s1, D, M);
#pragma unroll
      for (int t = 0; t < 3 && 3 * c + t < D; ++t) ka[3 * c + t] = u2d(blk[t]);
    }
  } else {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      const size_t ko = (((size_t)j * KE + prime) * 2) * n + k;
      kb[j] = u2d(key[ko]);
      ka[j] = u2d(key[ko + n]);
    }
  }
  for (uint32_t job = j0; job < j1; ++job) {
    const uint32_t s = tab.job_src[job];
    const size_t so = (size_t)row * tab.src_stride[s] + src;
    const uint64_t* ex = ext + ((size_t)s * D * E + row) * n + src;
    const uint64_t* y = tab.src_y[s];
    double dv[D];
#pragma unroll
    for (int j = 0; j < D; ++j) {
      if ((uint32_t)j != own) {
        dv[j] = u2d(ex[(size_t)j * E * n]);
      } else {  // own digit: the source row itself (a product source formed here)
        dv[j] = u2d(tab.src_in[s][so]);
        if (y) dv[j] = mm_var(dv[j], u2d(y[so]), M.q, M.qinv);
      }
    }
    double ab = 0.0, aa = 0.0;
#pragma unroll
    for (int j = 0; j < D; ++j) {
      ab += mm_var(dv[j], kb[j], M.q, M.qinv);
      aa += mm_var(dv[j], ka[j], M.q, M.qinv);
      if ((j & 3) == 3 && j + 1 < D) {
        ab = red_bal(ab, M.q, M.qinv);
        aa = red_bal(aa, M.q, M.qinv);
      }
    }
    if (tab.fold == 2 && row < level) {
      // extended-basis output: the addend enters multiplied by P (pinv holds
      // P mod q_row here), no ModDown follows
      const double2 f = pinv[row];
      const uint64_t* add = tab.add[job];
      const uint32_t mask = tab.add_mask[job];
      const size_t o0 = (size_t)2 * row * n + src, o1 = o0 + n;
      if (add && (mask & 1u)) ab += mm_shoup(u2d(add[o0]), f.x, f.y, M.q);
      if (add && (mask & 2u)) aa += mm_shoup(u2d(add[o1]), f.x, f.y, M.q);
    } else if (tab.fold && row < level) {
      const double2 f = pinv[row];
      ab = mm_shoup(ab, f.x, f.y, M.q);
      aa = mm_shoup(aa, f.x, f.y, M.q);
      const uint64_t* add = tab.add[job];
      const uint32_t mask = tab.add_mask[job];
      const size_t o0 = (size_t)2 * row * n + src, o1 = o0 + n;
      if (const uint64_t* ay = tab.add_y[job]) {
        // tensor addend (d0, d1) = (x0 y0, x0 y1 + x1 y0), |each| < q
        const double x0 = u2d(add[o0]), x1 = u2d(add[o1]);
        const double y0 = u2d(ay[o0]), y1 = u2d(ay[o1]);
        if (mask & 1u) ab += mm_var(x0, y0, M.q, M.qinv);
        if (mask & 2u) aa += mm_var(x0, y1, M.q, M.qinv) + mm_var(x1, y0, M.q, M.qinv);
      } else {
        if (add && (mask & 1u)) ab += u2d(add[o0]);
        if (add && (mask & 2u)) aa += u2d(add[o1]);
      }
    }
    uint64_t* out = tab.fold == 2 ? tab.out[job] : acc + (size_t)job * 2 * E * n;
    out[(size_t)row * n + k] = to_res(ab, M.q, M.qinv);
    out[((size_t)E + row) * n + k] = to_res(aa, M.q, M.qinv);
  }
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

template <int D>
struct IpL {
  static void run(dim3 g, hipStream_t s, const KsTable& tab, const uint64_t* ext, uint64_t* acc,
                  uint32_t level, uint32_t L, uint32_t alpha, uint32_t log_n, const PrimeK* pk,
                  const double2* pinv) {
    hipLaunchKernelGGL(k_ip<D>, g, dim3(kThreads), 0, s, tab, ext, acc, level, L, alpha, log_n,
                       pk, pinv);
  }
};

}  // namespace

hipError_t k_ip_launch(const Context* c, const KsTable& tab, uint32_t nkeys, const uint64_t* ext,
                       uint64_t* acc, uint32_t level, const double2* pinv, hipStream_t s) {
  const uint32_t dnum_l = (level + c->alpha - 1) / c->alpha;
  if (dnum_l > 16) return hipErrorInvalidValue;
  dim3 grid((c->n + kThreads - 1) / kThreads, level + c->alpha, nkeys);
  dispatch16<IpL>(dnum_l, grid, s, tab, ext, acc, level, c->L, c->alpha, c->log_n, c->d_pk,
                  pinv);
  return hipGetLastError();
}

}  // namespace fesc
