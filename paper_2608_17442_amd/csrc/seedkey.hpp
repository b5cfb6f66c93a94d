// Seed-expanded switching keys: the uniform half a_j of a key is not stored
// but regenerated wherever it is read, from two 64-bit seed words, with the
// counter-based generator Philox4x64-10 (Salmon, Moraes, Dror and Shaw,
// "Parallel random numbers: as easy as 1, 2, 3", SC 2011).
//
// For coefficient k (evaluation-form index), extended prime `prime` (its index
// in the full chain: q_i -> i, p_k -> L + k), Galois element `elt` (0 for the
// relinearisation key) and digit block c (digits 3c, 3c+1, 3c+2), one Philox
// block of the counter (k, prime, c, elt) under the key (seed0, seed1) gives
// words w0..w3.  Digit 3c+i takes w_i masked to the bit length of q when that
// is below q; otherwise the spare word w3 (masked) when no earlier digit of the
// block has taken it and it is below q; otherwise w_i mod q.
//
// Compact key layout (device): words 0, 1 the seed, word 2 the element, words
// 3..31 zero, then the b half [dnum][L+alpha][N] from word kSeedHeaderWords.
#pragma once

#include "fesc_internal.hpp"

namespace fesc {

constexpr size_t kSeedHeaderWords = 32;  // 256 bytes: keeps the b rows aligned

__device__ __forceinline__ void philox4x64_10(uint64_t x[4], uint64_t k0, uint64_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t m0 = 0xD2E7470EE14C6C93ull, m1 = 0xCA5A826395121157ull;
    const uint64_t lo0 = m0 * x[0], hi0 = __umul64hi(m0, x[0]);
    const uint64_t lo1 = m1 * x[2], hi1 = __umul64hi(m1, x[2]);
    const uint64_t y0 = hi1 ^ x[1] ^ k0, y2 = hi0 ^ x[3] ^ k1;
    x[0] = y0;
    x[1] = lo1;
    x[2] = y2;
    x[3] = lo0;
    k0 += 0x9E3779B97F4A7C15ull;  // Weyl increments of the key
    k1 += 0xBB67AE8584CAA73Bull;
  }
}

// w mod q for a full 64-bit w (the rare fallback of the residue rule), exact:
// w = hi 2^32 + lo, hi 2^32 reduced with one fp64 product (exact, as 2^32 is
// a power of two) and the sum brought to [0, q).
__device__ __forceinline__ uint64_t mod_u64(uint64_t w, double q, double qinv) {
  const double hi = (double)(uint32_t)(w >> 32), lo = (double)(uint32_t)w;
  return to_res(mm_var(hi, 4294967296.0, q, qinv) + lo, q, qinv);
}

// Digits 3c .. min(3c + 3, digits) - 1 of the uniform half at (k, prime, elt):
// a[i] for i < 3 (entries at or beyond `digits` - 3c are left untouched).
__device__ __forceinline__ void seeded_key_block(uint64_t a[3], uint32_t k, uint32_t prime,
                                                 uint32_t c, uint64_t elt, uint64_t s0,
                                                 uint64_t s1, uint32_t digits,
                                                 const PrimeK& M) {
  uint64_t w[4] = {k, prime, c, elt};
  philox4x64_10(w, s0, s1);
  const uint64_t q = M.qu, mask = ~0ull >> __builtin_clzll(q);
  bool spare = true;
#pragma unroll
  for (uint32_t i = 0; i < 3; ++i) {
    if (3 * c + i >= digits) break;
    uint64_t v = w[i] & mask;
    if (v >= q) {
      const uint64_t sp = w[3] & mask;
      if (spare && sp < q) {
        v = sp;
        spare = false;
      } else {
        v = mod_u64(w[i], M.q, M.qinv);
      }
    }
    a[i] = v;
  }
}

}  // namespace fesc
