// Compositions of the ciphertext operations (ops.cpp): the scan-contract
// slice, HEConv and the fused post-SSM path.  Every launch is asynchronous on
// the caller's stream; temporaries live in the context scratch.
#include <algorithm>
#include <climits>
#include <vector>

#include "fesc_internal.hpp"
#include "ops.hpp"
#include "scratch.hpp"

#define HIPCK(expr)                                    \
  do {                                                 \
    hipError_t e_ = (expr);                            \
    if (e_ != hipSuccess) return hip_check(e_, #expr); \
  } while (0)

namespace fesc {

// Scan-contract slice (see fesc.h): per (token, chunk),
//   t = RS(relin(RS(relin(decay * h)) * c))     (decay given; level - 2)
//   t = RS(relin(h * c))                        (contraction only; level - 1)
// each relinearised product divided by P q_{l-1} in one merged key switch;
// chunk pairs packed as chi = t_2l + i t_2l+1, reduced over the d_s axis by
// rotate-and-add, and split by one conjugation into 2 Sigma(t_2l) and
// 2 Sigma(t_2l+1).
int op_scan_contract(Context* c, const uint64_t* const* h, const uint64_t* const* decay,
                     const uint64_t* const* cfac, uint32_t K, uint32_t T, uint32_t d_s,
                     uint64_t* const* out, uint32_t level, hipStream_t s) {
  int err;
  const uint32_t lo = decay ? level - 2 : level - 1;
  const size_t n = c->n;
  // The batched layout is taken first: the calls below request no more, so
  // the ciphertext region S.cts stays in place while it is in use.
  Scratch S;
  if ((err = scratch(c, &S, 2))) return err;
  if (S.cap < 2) return fail(FESC_ERR_OOM, "scan-contract needs batched scratch");
  const size_t W = (size_t)2 * c->L * n;
  const uint32_t G = S.cap & ~1u;
  const uint32_t KT = K * T;
  if (K % 2 && T > S.cap) return fail(FESC_ERR_ARG, "at most 32 tokens with an odd chunk count");
  // the products of every (token, chunk) in groups of G; the decay product's
  // level - 1 intermediates live in S.cts, the last product writes out
  for (uint32_t g0 = 0; g0 < KT; g0 += G) {
    const uint32_t m = std::min(G, KT - g0);
    if (!decay) {
      if ((err = op_prod_rescale_many(c, m, h + g0, cfac + g0, out + g0, nullptr, level,
                                      level - 1, s)))
        return err;
      continue;
    }
    std::vector<uint64_t*> t(m);
    for (uint32_t k = 0; k < m; ++k) t[k] = S.cts + (size_t)k * W;
    if ((err = op_prod_rescale_many(c, m, decay + g0, h + g0, t.data(), nullptr, level,
                                    level - 1, s)))
      return err;
    const std::vector<const uint64_t*> tc(t.begin(), t.end());
    if ((err = op_prod_rescale_many(c, m, tc.data(), cfac + g0, out + g0, nullptr, level - 1,
                                    level - 2, s)))
      return err;
  }
  const uint32_t P = K / 2;  // complex pairs (2l, 2l+1); an odd last chunk is reduced alone
  const uint32_t R = P + (K % 2);
  if (R == 0) return FESC_OK;
  // Reduction of every token at once.  Pair l of token u is reduced in its own
  // two output buffers (x: the value, y: the partner; rotate-and-add
  // ping-pongs between them); an odd chunk's partner is a scratch slot.
  std::vector<uint64_t*> x, y;
  for (uint32_t u = 0; u < T; ++u) {
    uint64_t* const* o = out + (size_t)u * K;
    for (uint32_t l = 0; l < P; ++l) {
      x.push_back(o[2 * l]);
      y.push_back(o[2 * l + 1]);
    }
    if (K % 2) {
      x.push_back(o[K - 1]);
      y.push_back(S.cts + (size_t)u * W);
    }
  }
  const std::vector<uint64_t*> first = x;  // where out_2l (or the odd output) lives
  // pair entries (an odd chunk has none), kPairBatch per launch
  auto pairs = [&](bool split) -> int {
    PairTable tab{};
    uint32_t m = 0;
    for (uint32_t r = 0; r < R * T; ++r) {
      if (K % 2 && r % R == P) continue;
      tab.x[m] = x[r];
      tab.y[m] = y[r];
      // out_2l goes to the buffer it started in, out_2l+1 to the other
      tab.first[m] = first[r];
      tab.second[m] = first[r] == x[r] ? y[r] : x[r];
      if (++m == kPairBatch) {
        HIPCK(k_pair_launch(c, tab, m, split, lo, s));
        m = 0;
      }
    }
    if (m) HIPCK(k_pair_launch(c, tab, m, split, lo, s));
    return FESC_OK;
  };
  // chi_l = t_2l + i t_2l+1 (i = X^(N/2)), formed in x
  if ((err = pairs(false))) return err;
  for (uint32_t st = d_s / 2; st >= 1; st /= 2) {
    const std::vector<int32_t> steps(R * T, (int32_t)st);
    // y = x + rot(x, st)
    if ((err = op_rotate_batch(c, R * T, x.data(), steps.data(), y.data(), x.data(), lo, s)))
      return err;
    std::swap(x, y);
  }
  if (P > 0) {
    std::vector<uint64_t*> xp, yp;
    for (uint32_t r = 0; r < R * T; ++r)
      if (!(K % 2 && r % R == P)) {
        xp.push_back(x[r]);
        yp.push_back(y[r]);
      }
    const std::vector<int32_t> cj(xp.size(), INT32_MIN);
    if ((err = op_rotate_batch(c, (uint32_t)xp.size(), xp.data(), cj.data(), yp.data(), nullptr,
                               lo, s)))
      return err;
    // out_2l = chi + conj(chi);  out_2l+1 = -i (chi - conj(chi)) = X^(3N/2) (chi - conj(chi)),
    // in place in the pair's two buffers (x = chi, y = conj(chi))
    if ((err = pairs(true))) return err;
  }
  if (K % 2)
    for (uint32_t u = 0; u < T; ++u) {
      const uint32_t r = u * R + P;
      if (x[r] != first[r])
        HIPCK(hipMemcpyAsync(first[r], x[r], (size_t)2 * lo * n * 8, hipMemcpyDeviceToDevice, s));
    }
  return FESC_OK;
}


// HEConv (Sec. "Causal Depthwise Convolution"): the taps' rotations share one
// ModUp (hoisted), one pass accumulates sum_r M_r (.) rho(q; delta_r) with the
// bias folded in as q_{l-1} b, and a rescale divides by q_{l-1}:
//     out = RS(sum_r M_r (.) rho(q; delta_r)) + b            (level - 1)
int op_heconv(Context* c, const uint64_t* q, uint32_t taps, const int32_t* deltas,
              const uint64_t* const* masks, const uint64_t* bias, uint64_t* out, uint32_t level,
              hipStream_t s) {
  Scratch S;
  int err;
  if ((err = scratch(c, &S, 2))) return err;  // batched layout: S.cts stays in place
  if (taps + 1 > S.cap) return fail(FESC_ERR_ARG, "too many taps");
  const size_t W = (size_t)2 * c->L * c->n;
  std::vector<uint64_t*> rot(taps);
  for (uint32_t r = 0; r < taps; ++r) rot[r] = S.cts + (size_t)r * W;
  uint64_t* acc = S.cts + (size_t)taps * W;
  if ((err = op_rotate_many(c, q, taps, deltas, rot.data(), level, s))) return err;
  ConvTable tab{};
  for (uint32_t r = 0; r < taps; ++r) {
    tab.rot[r] = rot[r];
    tab.mask[r] = masks[r];
  }
  tab.taps = taps;
  HIPCK(k_conv_acc_launch(c, tab, bias, acc, level, s));
  const uint64_t* in = acc;
  return op_rescale_many(c, 1, &in, &out, level, s);
}

// Fused post-SSM path (Appendix "Fused Post-SSM Path"):
//     y = RS(D (.) x_skip) + m          (level - 1; m through its leading limbs)
//     out = y (.) g / (P q_{level-2})   (level - 2; one merged key switch)
int op_post_ssm(Context* c, const uint64_t* m, const uint64_t* x_skip, const uint64_t* d_skip,
                const uint64_t* g, uint64_t* out, uint32_t level, hipStream_t s) {
  Scratch S;
  int err;
  if ((err = scratch(c, &S, 2))) return err;
  const size_t W = (size_t)2 * c->L * c->n;
  uint64_t* t = S.cts;
  uint64_t* y = S.cts + W;
  HIPCK(k_mul_plain_launch(c, x_skip, d_skip, t, level, s));
  const uint64_t* tin = t;
  if ((err = op_rescale_add_many(c, 1, &tin, &y, &m, level, level - 1, s))) return err;
  const uint64_t* yin = y;
  return op_prod_rescale_many(c, 1, &yin, &g, &out, nullptr, level - 1, level - 2, s);
}

int op_add_plain(Context* c, const uint64_t* ct, const uint64_t* pt, uint64_t* out,
                 uint32_t level, hipStream_t s) {
  HIPCK(k_add_plain_launch(c, ct, pt, out, level, s));
  return FESC_OK;
}

}  // namespace fesc

namespace fesc {

// The batched scratch ciphertext slots ([cap][L][2][N] words) for callers
// outside this file (device encoding).
int scratch_slots(Context* c, uint64_t** cts, uint32_t* cap) {
  Scratch S;
  int err;
  if ((err = scratch(c, &S, 2))) return err;
  *cts = S.cts;
  *cap = S.cap;
  return FESC_OK;
}

}  // namespace fesc
