// Host drivers of the ciphertext operations: per-level constant tables,
// scratch layout, and the launch sequences of key switching, rotation,
// relinearisation, rescaling (separate, or merged with ModDown), key
// generation and encryption (the compositions built on them are in
// compose.cpp).  Every launch is
// asynchronous on the caller's stream; only a growth of the context scratch
// synchronises the device (before the old allocation is freed).
#include <algorithm>
#include <functional>
#include <string>
#include <vector>

#include "fesc_internal.hpp"
#include "ops.hpp"
#include "scratch.hpp"
#include "seedkey.hpp"

namespace fesc {

// ------------------------------------------------------------ level tables

namespace {

uint64_t prod_mod_except(const std::vector<uint64_t>& ps, size_t skip, uint64_t m) {
  uint64_t r = 1 % m;
  for (size_t b = 0; b < ps.size(); ++b)
    if (b != skip) r = h_mulmod(r, ps[b] % m, m);
  return r;
}

double2 entry(uint64_t v, uint64_t m) { return double2{(double)v, (double)v / (double)m}; }

// The 512 operand bytes of one target row of the matrix-core conversion
// (LevelTables::mu_bytes): hats[a] for a < aj (aj <= 8), target prime m.
void conversion_bytes(int8_t* dst, const uint64_t* hats, uint32_t aj, uint64_t m) {
  for (uint32_t a = 0; a < 8; ++a)
    for (uint32_t s = 0; s < 8; ++s) {
      int64_t v = (a < aj && s < 7) ? (int64_t)h_mulmod(hats[a] % m, h_powmod(2, 8 * s, m), m) : 0;
      for (uint32_t tau = 0; tau < 8; ++tau) {
        const int64_t d = ((v + 128) & 255) - 128;  // balanced digit in [-128, 127]
        v = (v - d) / 256;
        dst[(tau * 4 + a / 2) * 16 + (a % 2) * 8 + s] = (int8_t)d;
      }
    }
}

}  // namespace

const LevelTables* level_tables(Context* c, uint32_t level, int* err) {
  *err = FESC_OK;
  auto it = c->level_tabs.find(level);
  if (it != c->level_tabs.end()) return &it->second;
  const uint32_t L = c->L, alpha = c->alpha, E = level + alpha;
  const uint32_t dnum_l = (level + alpha - 1) / alpha;
  auto ext_prime = [&](uint32_t row) { return c->primes[row < level ? row : L + (row - level)]; };
  std::vector<uint64_t> ps(c->primes.begin() + L, c->primes.end());

  std::vector<double2> mu_inv((size_t)dnum_l * alpha), mu_hat((size_t)dnum_l * E * alpha),
      mu_inv_n(level);
  const bool mfma = alpha <= 8;  // the matrix-core conversion's operand tables
  std::vector<int8_t> mu_bytes(mfma ? (size_t)dnum_l * E * 512 : 0),
      md_bytes(mfma ? (size_t)level * 512 : 0), mr_bytes(mfma ? (size_t)(level - 1) * 512 : 0);
  for (uint32_t j = 0; j < dnum_l; ++j) {
    const uint32_t lo = j * alpha, hi = std::min(lo + alpha, level);
    std::vector<uint64_t> dq(c->primes.begin() + lo, c->primes.begin() + hi);
    for (uint32_t a = 0; a < hi - lo; ++a) {
      const uint64_t inv = h_inv(prod_mod_except(dq, a, dq[a]), dq[a]);
      mu_inv[j * alpha + a] = entry(inv, dq[a]);
      mu_inv_n[lo + a] = entry(h_mulmod(inv, h_inv(c->n % dq[a], dq[a]), dq[a]), dq[a]);
      for (uint32_t row = 0; row < E; ++row) {
        const uint64_t m = ext_prime(row);
        mu_hat[((size_t)j * E + row) * alpha + a] = entry(prod_mod_except(dq, a, m), m);
      }
    }
    if (mfma)
      for (uint32_t row = 0; row < E; ++row) {
        const uint64_t m = ext_prime(row);
        uint64_t hats[8];
        for (uint32_t a = 0; a < hi - lo; ++a) hats[a] = prod_mod_except(dq, a, m);
        conversion_bytes(mu_bytes.data() + ((size_t)j * E + row) * 512, hats, hi - lo, m);
      }
  }
  std::vector<double2> md_inv(alpha), md_hat((size_t)level * alpha), md_pinv(level), pmod(L),
      rs_inv(level), md_inv_n(alpha);
  for (uint32_t a = 0; a < alpha; ++a) {
    const uint64_t inv = h_inv(prod_mod_except(ps, a, ps[a]), ps[a]);
    md_inv[a] = entry(inv, ps[a]);
    md_inv_n[a] = entry(h_mulmod(inv, h_inv(c->n % ps[a], ps[a]), ps[a]), ps[a]);
  }
  for (uint32_t i = 0; i < L; ++i) {
    const uint64_t q = c->primes[i];
    const uint64_t P = prod_mod_except(ps, ps.size(), q);
    pmod[i] = entry(P, q);
    if (i < level) {
      md_pinv[i] = entry(h_inv(P, q), q);
      uint64_t hats[FESC_MAX_ALPHA];
      for (uint32_t a = 0; a < alpha; ++a) {
        hats[a] = prod_mod_except(ps, a, q);
        md_hat[(size_t)i * alpha + a] = entry(hats[a], q);
      }
      if (mfma) conversion_bytes(md_bytes.data() + (size_t)i * 512, hats, alpha, q);
      if (i + 1 < level) rs_inv[i] = entry(h_inv(c->primes[level - 1] % q, q), q);
    }
  }
  std::vector<double2> rs_ninv(1), one(level), mr_inv_n(alpha + 1),
      mr_hat((size_t)(level - 1) * (alpha + 1));
  {
    const uint64_t ql = c->primes[level - 1];
    rs_ninv[0] = entry(h_inv(c->n % ql, ql), ql);
    for (uint32_t i = 0; i < level; ++i) one[i] = entry(1, c->primes[i]);
    // m_0 = q_{level-1}: the inner product stores x P^-1 on that row, which is
    // already x (M/m_0)^-1, so its constant is N^-1 alone
    mr_inv_n[0] = entry(h_inv(c->n % ql, ql), ql);
    for (uint32_t a = 0; a < alpha; ++a) {
      const uint64_t pa = ps[a];
      const uint64_t mh = h_mulmod(prod_mod_except(ps, a, pa), ql % pa, pa);  // M/p_a mod p_a
      mr_inv_n[1 + a] = entry(h_mulmod(h_inv(mh, pa), h_inv(c->n % pa, pa), pa), pa);
    }
    for (uint32_t i = 0; i + 1 < level; ++i) {
      const uint64_t q = c->primes[i];
      uint64_t hats[FESC_MAX_ALPHA + 1];
      hats[0] = prod_mod_except(ps, ps.size(), q);  // P
      for (uint32_t a = 0; a < alpha; ++a)
        hats[1 + a] = h_mulmod(prod_mod_except(ps, a, q), ql % q, q);  // (P/p_a) q_{l-1}
      for (uint32_t a = 0; a <= alpha; ++a) mr_hat[(size_t)i * (alpha + 1) + a] = entry(hats[a], q);
      // sources 0..7 on the matrix cores (the ninth, p_7 for alpha = 8, on the VALU)
      if (mfma) conversion_bytes(mr_bytes.data() + (size_t)i * 512, hats, std::min(alpha + 1, 8u), q);
    }
  }
  std::vector<double2> all;
  LevelTables T;
  T.level = level;
  size_t off[13];
  const std::vector<double2>* parts[13] = {&mu_inv,   &mu_hat,  &md_inv,   &md_hat, &md_pinv,
                                           &pmod,     &rs_inv,  &mu_inv_n, &md_inv_n,
                                           &rs_ninv,  &one,     &mr_inv_n, &mr_hat};
  for (int p = 0; p < 13; ++p) {
    off[p] = all.size();
    all.insert(all.end(), parts[p]->begin(), parts[p]->end());
  }
  // one allocation: the double2 tables, then the conversion bytes
  const size_t words = sizeof(double2) * all.size();
  const size_t total = words + mu_bytes.size() + md_bytes.size() + mr_bytes.size();
  double2* d = nullptr;
  if (hipMalloc(&d, total) != hipSuccess) {
    *err = fail(FESC_ERR_OOM, "level table allocation failed");
    return nullptr;
  }
  int8_t* bytes = reinterpret_cast<int8_t*>(d) + words;
  if ((*err = hip_check(hipMemcpy(d, all.data(), words, hipMemcpyHostToDevice), "hipMemcpy")) ||
      (mfma && ((*err = hip_check(hipMemcpy(bytes, mu_bytes.data(), mu_bytes.size(),
                                            hipMemcpyHostToDevice), "hipMemcpy")) ||
                (*err = hip_check(hipMemcpy(bytes + mu_bytes.size(), md_bytes.data(),
                                            md_bytes.size(), hipMemcpyHostToDevice),
                                  "hipMemcpy")) ||
                (*err = hip_check(hipMemcpy(bytes + mu_bytes.size() + md_bytes.size(),
                                            mr_bytes.data(), mr_bytes.size(),
                                            hipMemcpyHostToDevice),
                                  "hipMemcpy"))))) {
    (void)hipFree(d);
    return nullptr;
  }
  if (mfma) {
    T.mu_bytes = bytes;
    T.md_bytes = bytes + mu_bytes.size();
    T.mr_bytes = bytes + mu_bytes.size() + md_bytes.size();
  }
  T.base = d;
  T.mu_inv = d + off[0];
  T.mu_hat = d + off[1];
  T.md_inv = d + off[2];
  T.md_hat = d + off[3];
  T.md_pinv = d + off[4];
  T.pmod = d + off[5];
  T.rs_inv = d + off[6];
  T.mu_inv_n = d + off[7];
  T.md_inv_n = d + off[8];
  T.rs_ninv = d + off[9];
  T.one = d + off[10];
  T.mr_inv_n = d + off[11];
  T.mr_hat = d + off[12];
  return &(c->level_tabs[level] = T);
}

// ------------------------------------------------------------------ scratch

int scratch(Context* c, Scratch* s, uint32_t batch) {
  const size_t n = c->n, L = c->L, E = c->L + c->alpha;
  size_t B = batch <= 1 ? 1 : kMaxBatch;
  if (c->scratch_bytes) {  // keep the larger capacity once allocated
    const size_t per_b = (L + c->dnum * E + 2 * E + 2 * L + 2 * L) * n * 8;
    const size_t fixed = (2 * L + L + 2 + 2 * L) * n * 8;
    if (c->scratch_bytes >= fixed + kMaxBatch * per_b) B = kMaxBatch;
  }
  const size_t sizes[9] = {2 * L * n,     B * L * n, B * c->dnum * E * n, B * 2 * E * n,
                           B * 2 * L * n, L * n,     2 * n,               2 * L * n,
                           B * 2 * L * n};
  size_t total = 0;
  for (size_t x : sizes) total += x;
  int err;
  uint64_t* base = static_cast<uint64_t*>(scratch_get(c, total * sizeof(uint64_t), &err));
  if (!base) return err;
  s->cap = (uint32_t)B;
  uint64_t** dst[9] = {&s->cin, &s->cc, &s->ext, &s->acc, &s->y, &s->d2, &s->v, &s->w, &s->cts};
  for (int i = 0; i < 9; ++i) {
    *dst[i] = base;
    base += sizes[i];
  }
  return FESC_OK;
}

namespace {

#define HIPCK(expr)                                    \
  do {                                                 \
    hipError_t e_ = (expr);                            \
    if (e_ != hipSuccess) return hip_check(e_, #expr); \
  } while (0)

hipError_t ntt_rows(const Context* c, uint64_t* d, uint32_t batch, size_t batch_stride,
                    uint32_t limbs, uint32_t prime0, bool inverse, hipStream_t s) {
  RowSel rs{d, batch_stride, (size_t)c->n, prime0, limbs, 0, 0, 0, 0};
  return launch_ntt_rows(c, rs, batch, limbs, inverse, s);
}

}  // namespace

// --------------------------------------------------------- key switch engine

int key_switch_batch(Context* c, uint32_t level, const std::vector<KsSource>& srcs,
                     const std::vector<KsJob>& jobs, hipStream_t s, uint32_t rescale_rows,
                     const Scratch* given, bool ext_out) {
  if (jobs.empty()) return FESC_OK;
  if (ext_out && rescale_rows) return fail(FESC_ERR_ARG, "extended outputs take no rescale");
  if (rescale_rows && (level < 2 || rescale_rows > level - 1))
    return fail(FESC_ERR_LEVEL, "merged rescale needs level >= 2 and rows <= level - 1");
  if (srcs.size() > kMaxBatch) return fail(FESC_ERR_ARG, "too many key-switch sources");
  int err;
  const LevelTables* T = level_tables(c, level, &err);
  if (!T) return err;
  Scratch S;
  if (given)
    S = *given;
  else if ((err = scratch(c, &S, (uint32_t)std::max(srcs.size(), jobs.size()))))
    return err;
  const size_t n = c->n;
  const uint32_t E = level + c->alpha, dnum_l = (level + c->alpha - 1) / c->alpha;
  KsTable tab{};
  for (size_t i = 0; i < srcs.size(); ++i) {
    tab.src_in[i] = srcs[i].in;
    tab.src_stride[i] = srcs[i].stride;
    tab.src_y[i] = srcs[i].y;
  }
  // ModUp of every source (the scratch capacity covers all of them)
  const uint32_t ns = (uint32_t)srcs.size();
  if (ns > S.cap) return fail(FESC_ERR_ARG, "key-switch sources exceed the scratch capacity");
  for (const KsJob& J : jobs) {
    if (J.src >= ns) return fail(FESC_ERR_ARG, "key-switch job names a missing source");
    auto cap = c->key_cap.find(J.key);
    if (cap != c->key_cap.end() && level > cap->second)
      return fail(FESC_ERR_LEVEL, "switching key uploaded for levels up to " +
                                      std::to_string(cap->second) + ", used at level " +
                                      std::to_string(level));
  }
  // iNTT of the sources, stored as centred ModUp digits; ModUp fused with the
  // first forward pass of the extended rows; second pass (own-digit rows are
  // never written: the inner product reads them from the source)
  HIPCK(launch_ntt_inv_sources(c, tab, ns, S.cc, level, T->mu_inv_n, s));
  HIPCK(launch_modup_outer(c, *T, S.cc, S.ext, ns, level, s));
  RowSel rs{S.ext, (size_t)E * n, n, 0, level, c->L, c->alpha, level, dnum_l};
  HIPCK(launch_ntt_fwd_inner_rows(c, rs, ns * dnum_l, E, s));
  // jobs
  // jobs ordered by (key, Galois element): each group of kMaxBatch jobs then
  // holds few distinct keys, and the inner product reads each key once
  std::vector<uint32_t> order(jobs.size());
  for (uint32_t j = 0; j < order.size(); ++j) order[j] = j;
  std::stable_sort(order.begin(), order.end(), [&](uint32_t x, uint32_t y) {
    const KsJob &a = jobs[x], &b = jobs[y];
    return a.key != b.key ? std::less<const uint64_t*>()(a.key, b.key) : a.galois < b.galois;
  });
  for (size_t j0 = 0; j0 < jobs.size(); j0 += S.cap) {
    const uint32_t nj = std::min<uint32_t>(S.cap, (uint32_t)(jobs.size() - j0));
    KsTable t = tab;
    t.fold = 1;
    uint32_t nkeys = 0;
    for (uint32_t j = 0; j < nj; ++j) {
      const KsJob& J = jobs[order[j0 + j]];
      if (j == 0 || J.key != t.key[j - 1] || J.galois != t.galois[j - 1]) {
        if (c->key_seeded.count(J.key)) t.kg_seeded |= 1u << nkeys;
        t.kg_first[nkeys] = j;
        t.kg_count[nkeys++] = 0;
      }
      ++t.kg_count[nkeys - 1];
      t.job_src[j] = J.src;
      t.key[j] = J.key;
      t.galois[j] = J.galois;
      t.add[j] = J.add;
      t.add_mask[j] = J.add ? J.add_mask : 0;
      t.add_galois[j] = J.add_galois;
      if (J.add && J.add_galois != J.galois) t.fold = 0;
      t.add2[j] = J.add2;
      t.out[j] = J.out;
      t.add_y[j] = J.add_y;
    }
    for (uint32_t j = 0; j < nj && !t.fold; ++j)
      if (t.add_y[j]) return fail(FESC_ERR_ARG, "a tensor addend needs the folded combine");
    if (rescale_rows && !t.fold) return fail(FESC_ERR_ARG, "merged rescale needs folded addends");
    if (ext_out) {
      for (uint32_t j = 0; j < nj; ++j)
        if (t.add_y[j]) return fail(FESC_ERR_ARG, "extended outputs take plain addends");
      if (!t.fold) return fail(FESC_ERR_ARG, "extended outputs need addends under the job's element");
      t.fold = 2;
      HIPCK(k_ip_launch(c, t, nkeys, S.ext, S.acc, level, T->pmod, s));
      continue;
    }
    HIPCK(k_ip_launch(c, t, nkeys, S.ext, S.acc, level, T->md_pinv, s));
    if (rescale_rows) {
      // rows q_{level-1}, p_0 .. p_{alpha-1} (adjacent in acc): iNTT to the
      // centred digits of M = P q_{level-1}; conversion to the kept rows fused
      // with the first forward pass; combine times q_{level-1}^-1
      const RowSel rp{S.acc + (size_t)(level - 1) * n, (size_t)E * n, n, level - 1, 1, c->L,
                      0, 0, 0};
      HIPCK(launch_ntt_inv_digits(c, rp, 2 * nj, c->alpha + 1, T->mr_inv_n, s));
      HIPCK(launch_moddown_rescale_outer(c, *T, S.acc, S.y, nj, level, rescale_rows, s));
      HIPCK(launch_ntt_fwd_ks_combine(c, S.y, nj, level, rescale_rows, level - 1, t, S.acc,
                                      T->md_pinv, T->rs_inv, s));
      continue;
    }
    // special-prime rows: iNTT to centred ModDown digits, conversion fused
    // with the first forward pass of y, second pass ending in the combine
    const RowSel rp{S.acc + (size_t)level * n, (size_t)E * n, n, c->L, c->alpha, 0, 0, 0, 0};
    HIPCK(launch_ntt_inv_digits(c, rp, 2 * nj, c->alpha, T->md_inv_n, s));
    HIPCK(launch_moddown_outer(c, *T, S.acc, S.y, nj, level, s));
    HIPCK(launch_ntt_fwd_ks_combine(c, S.y, nj, level, level, level, t, S.acc, T->md_pinv,
                                    nullptr, s));
  }
  return FESC_OK;
}

int op_moddown_many(Context* c, uint32_t count, uint64_t* ext, uint64_t* const* outs,
                    uint32_t level, hipStream_t s) {
  int err;
  const LevelTables* T = level_tables(c, level, &err);
  if (!T) return err;
  Scratch S;
  if ((err = scratch(c, &S, count))) return err;
  const size_t n = c->n, E = level + c->alpha;
  // the ciphertexts play the inner products' part (component-major rows
  // over the extended basis): inverse transform of the special-prime rows to
  // centred digits (in place), conversion to the level rows fused with the
  // first forward pass, second pass with the combine (acc - y) P^-1
  for (uint32_t j0 = 0; j0 < count; j0 += S.cap) {
    const uint32_t nj = std::min(S.cap, count - j0);
    uint64_t* acc = ext + (size_t)j0 * 2 * E * n;
    KsTable t{};
    for (uint32_t j = 0; j < nj; ++j) t.out[j] = outs[j0 + j];
    const RowSel rp{acc + (size_t)level * n, E * n, n, c->L, c->alpha, 0, 0, 0, 0};
    HIPCK(launch_ntt_inv_digits(c, rp, 2 * nj, c->alpha, T->md_inv_n, s));
    HIPCK(launch_moddown_outer(c, *T, acc, S.y, nj, level, s));
    HIPCK(launch_ntt_fwd_ks_combine(c, S.y, nj, level, level, level, t, acc, T->md_pinv,
                                    nullptr, s));
  }
  return FESC_OK;
}

// ------------------------------------------------------------------- drivers

uint32_t galois_of_step(const Context* c, int32_t step) {
  const uint64_t two_n = 2ull * c->n;
  if (step == INT32_MIN) return (uint32_t)(two_n - 1);
  const int64_t half = c->n / 2;
  const int64_t r = ((int64_t)step % half + half) % half;
  if (r == 0) return 1;
  return (uint32_t)h_powmod(5, (uint64_t)r, two_n);
}

static int key_of(Context* c, uint32_t g, const uint64_t** key) {
  auto it = c->keys.find(g);
  if (it == c->keys.end())
    return fail(FESC_ERR_NO_KEY, g == 0 ? std::string("no relinearisation key")
                                        : "no switching key for Galois element " +
                                              std::to_string(g));
  *key = it->second;
  return FESC_OK;
}

// Rotations of one ciphertext sharing one ModUp.
int op_rotate_many(Context* c, const uint64_t* in, uint32_t count, const int32_t* steps,
                   uint64_t* const* outs, uint32_t level, hipStream_t s) {
  const size_t n = c->n, ct_words = (size_t)2 * level * n;
  std::vector<uint32_t> gal(count);
  std::vector<const uint64_t*> keys(count, nullptr);
  int err;
  for (uint32_t r = 0; r < count; ++r) {
    gal[r] = galois_of_step(c, steps[r]);
    if (gal[r] != 1 && (err = key_of(c, gal[r], &keys[r]))) return err;
  }
  Scratch S;
  if ((err = scratch(c, &S, count))) return err;
  // an output that aliases the input would be overwritten while later
  // rotations still read it: work from a private copy then
  const uint64_t* src = in;
  for (uint32_t r = 0; r < count; ++r)
    if (outs[r] == in) {
      HIPCK(hipMemcpyAsync(S.cin, in, ct_words * 8, hipMemcpyDeviceToDevice, s));
      src = S.cin;
      break;
    }
  std::vector<KsJob> jobs;
  for (uint32_t r = 0; r < count; ++r) {
    if (gal[r] == 1) {
      if (outs[r] != src)
        HIPCK(hipMemcpyAsync(outs[r], src, ct_words * 8, hipMemcpyDeviceToDevice, s));
      continue;
    }
    jobs.push_back(KsJob{0, keys[r], gal[r], src, 1u, gal[r], nullptr, outs[r]});
  }
  return key_switch_batch(c, level, {KsSource{src + n, 2 * n}}, jobs, s);
}

// Rotation of `count` different ciphertexts, ins[i] by steps[i] into outs[i]
// (+ add2[i] when given).  Outputs must not alias inputs.
int op_rotate_batch(Context* c, uint32_t count, const uint64_t* const* ins,
                    const int32_t* steps, uint64_t* const* outs, const uint64_t* const* add2,
                    uint32_t level, hipStream_t s, const Scratch* given) {
  const size_t n = c->n, ct_words = (size_t)2 * level * n;
  const uint32_t group = given ? given->cap : kMaxBatch;
  int err;
  for (uint32_t b0 = 0; b0 < count; b0 += group) {
    const uint32_t nb = std::min(group, count - b0);
    std::vector<KsSource> srcs;
    std::vector<KsJob> jobs;
    for (uint32_t i = b0; i < b0 + nb; ++i) {
      const uint32_t g = galois_of_step(c, steps[i]);
      const uint64_t* a2 = add2 ? add2[i] : nullptr;
      if (g == 1) {
        if (a2)
          HIPCK(k_binary_launch(c, ins[i], a2, outs[i], 2 * level, 1, 0, s));
        else if (outs[i] != ins[i])
          HIPCK(hipMemcpyAsync(outs[i], ins[i], ct_words * 8, hipMemcpyDeviceToDevice, s));
        continue;
      }
      const uint64_t* key;
      if ((err = key_of(c, g, &key))) return err;
      jobs.push_back(KsJob{(uint32_t)srcs.size(), key, g, ins[i], 1u, g, a2, outs[i]});
      srcs.push_back(KsSource{ins[i] + n, 2 * n});
    }
    if ((err = key_switch_batch(c, level, srcs, jobs, s, 0, given))) return err;
  }
  return FESC_OK;
}

// Products a_i * b_i relinearised, in groups of up to kMaxBatch, each group
// one batched key switch (all jobs share the relinearisation key) whose
// source is d2 = a1 b1 and whose addend is (d0, d1) = (a0 b0, a0 b1 + a1 b0),
// both formed from the operands where they are read: the tensor is never
// stored.  out_i may alias a_i or b_i (all operands of a group are read
// before its combine writes).
int op_mul_relin_many(Context* c, uint32_t count, const uint64_t* const* as,
                      const uint64_t* const* bs, uint64_t* const* outs, uint32_t level,
                      hipStream_t s) {
  const uint64_t* key;
  int err;
  if ((err = key_of(c, 0, &key))) return err;
  Scratch S;
  if ((err = scratch(c, &S, count))) return err;
  const size_t n = c->n;
  for (uint32_t b0 = 0; b0 < count; b0 += S.cap) {
    const uint32_t m = std::min(S.cap, count - b0);
    // the tensor is never stored: the source d2 = a1 b1 is formed by the
    // inverse transform and the inner product, (d0, d1) by the fold
    std::vector<KsSource> srcs;
    std::vector<KsJob> jobs;
    for (uint32_t b = 0; b < m; ++b) {
      const uint64_t *x = as[b0 + b], *y = bs[b0 + b];
      srcs.push_back(KsSource{x + n, 2 * n, y + n});
      jobs.push_back(KsJob{b, key, 0, x, 3u, 0, nullptr, outs[b0 + b], y});
    }
    if ((err = key_switch_batch(c, level, srcs, jobs, s))) return err;
  }
  return FESC_OK;
}

int op_mul_relin(Context* c, const uint64_t* a, const uint64_t* b, uint64_t* out,
                 uint32_t level, hipStream_t s) {
  return op_mul_relin_many(c, 1, &a, &b, &out, level, s);
}

// Rescale (c - [c mod q_last]) / q_last of up to kRescaleBatch ciphertexts
// per launch sequence: inverse NTT of every last limb (read in place), lift
// of the centred coefficients to the other primes, forward NTT, combine.
int op_rescale_add_many(Context* c, uint32_t count, const uint64_t* const* ins,
                        uint64_t* const* outs, const uint64_t* const* adds, uint32_t level,
                        uint32_t out_rows, hipStream_t s) {
  if (level < 2 || out_rows < 1 || out_rows > level - 1)
    return fail(FESC_ERR_LEVEL, "rescale needs level >= 2 and 1 <= rows <= level - 1");
  int err;
  const LevelTables* T = level_tables(c, level, &err);
  if (!T) return err;
  Scratch S;
  if ((err = scratch(c, &S, count))) return err;
  if (count > 1 && S.cap < kMaxBatch) return fail(FESC_ERR_ARG, "rescale batch needs scratch");
  const size_t n = c->n;
  const uint32_t last = level - 1;
  // the key-switch regions are idle here: last limbs in cc, lifted rows in ext
  uint64_t* v = count > 1 ? S.cc : S.v;
  uint64_t* w = count > 1 ? S.ext : S.w;
  for (uint32_t b0 = 0; b0 < count; b0 += kRescaleBatch) {
    const uint32_t m = std::min(kRescaleBatch, count - b0);
    KsTable tab{};
    RsTable rt{};
    for (uint32_t b = 0; b < m; ++b) {
      tab.src_in[2 * b] = ins[b0 + b] + (size_t)2 * last * n;
      tab.src_in[2 * b + 1] = ins[b0 + b] + ((size_t)2 * last + 1) * n;
      rt.in[b] = ins[b0 + b];
      rt.out[b] = outs[b0 + b];
      rt.add[b] = adds ? adds[b0 + b] : nullptr;
    }
    // last limbs to centred coefficients (fp64), lifted to the kept rows
    // inside the first forward pass, combined in the second pass's epilogue
    HIPCK(launch_ntt_inv_rescale_last(c, tab, 2 * m, v, last, T->rs_ninv, s));
    HIPCK(launch_rescale_outer(c, v, w, 2 * m, last, out_rows, T->one, s));
    HIPCK(launch_ntt_fwd_rs_combine(c, w, m, last, out_rows, rt, T->rs_inv, s));
  }
  return FESC_OK;
}

int op_rescale_many(Context* c, uint32_t count, const uint64_t* const* ins, uint64_t* const* outs,
                    uint32_t level, hipStream_t s) {
  return op_rescale_add_many(c, count, ins, outs, nullptr, level, level - 1, s);
}

uint32_t prod_group(Context* c, int* err) {
  Scratch S;
  if ((*err = scratch(c, &S, 2))) return 0;
  return S.cap & ~1u;
}

int op_prod_rescale_many(Context* c, uint32_t count, const uint64_t* const* xs,
                         const uint64_t* const* ys, uint64_t* const* outs,
                         const uint64_t* const* adds, uint32_t level, uint32_t out_rows,
                         hipStream_t s) {
  if (level < 2 || out_rows < 1 || out_rows > level - 1)
    return fail(FESC_ERR_LEVEL, "product needs level >= 2 and 1 <= rows <= level - 1");
  const uint64_t* key;
  int err;
  if ((err = key_of(c, 0, &key))) return err;
  Scratch S;
  if ((err = scratch(c, &S, 2))) return err;
  const uint32_t G = S.cap & ~1u;
  if (G < 2) return fail(FESC_ERR_OOM, "batched products need batched scratch");
  const size_t n = c->n;
  // one key switch per group: tensor formed inside (source x1 y1, folded
  // addend (x0 y0, x0 y1 + x1 y0)), ModDown merged with the rescale, add_i
  // added in the combine
  for (uint32_t g0 = 0; g0 < count; g0 += G) {
    const uint32_t m = std::min(G, count - g0);
    std::vector<KsSource> srcs;
    std::vector<KsJob> jobs;
    for (uint32_t b = 0; b < m; ++b) {
      const uint64_t *x = xs[g0 + b], *y = ys[g0 + b];
      srcs.push_back(KsSource{x + n, 2 * n, y + n});
      jobs.push_back(
          KsJob{b, key, 0, x, 3u, 0, adds ? adds[g0 + b] : nullptr, outs[g0 + b], y});
    }
    if ((err = key_switch_batch(c, level, srcs, jobs, s, out_rows))) return err;
  }
  return FESC_OK;
}

int op_rescale(Context* c, const uint64_t* in, uint64_t* out, uint32_t level, hipStream_t s) {
  return op_rescale_many(c, 1, &in, &out, level, s);
}

size_t full_key_words(const Context* c) {
  return (size_t)c->dnum * (c->L + c->alpha) * 2 * c->n;
}

size_t seeded_key_words(const Context* c) {
  return kSeedHeaderWords + (size_t)c->dnum * (c->L + c->alpha) * c->n;
}

int key_buffer(Context* c, uint32_t galois, size_t words, uint64_t** out) {
  auto it = c->keys.find(galois);
  if (it != c->keys.end() && c->key_alloc[it->second] < words) {
    uint64_t* old = it->second;
    // work in flight may still read the old key
    const int rc = hip_check(hipDeviceSynchronize(), "key replacement");
    if (rc) return rc;
    c->key_alloc.erase(old);
    c->key_cap.erase(old);
    c->key_seeded.erase(old);
    c->keys.erase(it);
    (void)hipFree(old);
    it = c->keys.end();
  }
  if (it == c->keys.end()) {
    uint64_t* key = nullptr;
    if (hipMalloc(&key, words * 8) != hipSuccess) return fail(FESC_ERR_OOM, "key allocation failed");
    it = c->keys.emplace(galois, key).first;
    c->key_alloc[key] = words;
  }
  c->key_cap.erase(it->second);
  c->key_seeded.erase(it->second);
  *out = it->second;
  return FESC_OK;
}

int op_keygen(Context* c, uint32_t galois, const int8_t* sk, const uint64_t* a, const int64_t* e,
              const uint64_t* seed, hipStream_t s) {
  const size_t n = c->n;
  const uint32_t E = c->L + c->alpha;
  int err;
  const LevelTables* T = level_tables(c, c->L, &err);
  if (!T) return err;
  Scratch S;
  if ((err = scratch(c, &S))) return err;
  uint64_t* key = nullptr;
  if ((err = key_buffer(c, galois, seed ? seeded_key_words(c) : full_key_words(c), &key)))
    return err;
  // recorded before any launch: should one fail, the buffer is still read
  // with the layout it was allocated for
  if (seed) c->key_seeded.insert(key);
  uint64_t* s_ext = S.acc;            // [E][N]
  uint64_t* s_from = S.acc + E * n;   // [E][N]
  uint64_t* e_ntt = S.ext;            // [dnum][E][N]
  HIPCK(k_lift_launch(c, nullptr, sk, s_ext, E, 0, E, 0, s));
  HIPCK(ntt_rows(c, s_ext, 1, 0, E, 0, false, s));
  if (galois == 0)
    HIPCK(k_binary_launch(c, s_ext, s_ext, s_from, E, 0, 2, s));
  else
    HIPCK(k_galois_launch(c, s_ext, s_from, E, galois, s));
  for (uint32_t j = 0; j < c->dnum; ++j)
    HIPCK(k_lift_launch(c, e + (size_t)j * n, nullptr, e_ntt + (size_t)j * E * n, E, 0, E, 0, s));
  HIPCK(ntt_rows(c, e_ntt, c->dnum, (size_t)E * n, E, 0, false, s));
  KeySeed sd{};
  if (seed) sd = KeySeed{seed[0], seed[1], galois, c->dnum, 1u};
  HIPCK(k_keygen_launch(c, a, e_ntt, s_ext, s_from, key, T->pmod, sd, s));
  return FESC_OK;
}

int op_encrypt(Context* c, const int8_t* sk, const int64_t* m, const uint64_t* a,
               const int64_t* e, uint64_t* ct, uint32_t level, hipStream_t s) {
  Scratch S;
  int err;
  if ((err = scratch(c, &S))) return err;
  uint64_t* me = S.cc;
  uint64_t* et = S.y;
  uint64_t* sl = S.d2;
  HIPCK(k_lift_launch(c, m, nullptr, me, level, 0, level, 0, s));
  HIPCK(k_lift_launch(c, e, nullptr, et, level, 0, level, 0, s));
  HIPCK(k_binary_launch(c, me, et, me, level, 0, 0, s));
  HIPCK(ntt_rows(c, me, 1, 0, level, 0, false, s));
  HIPCK(k_lift_launch(c, nullptr, sk, sl, level, 0, level, 0, s));
  HIPCK(ntt_rows(c, sl, 1, 0, level, 0, false, s));
  HIPCK(k_encrypt_launch(c, a, sl, me, ct, level, s));
  return FESC_OK;
}

int op_plain_from_coeffs(Context* c, const int64_t* m, uint64_t* pt, uint32_t level,
                         hipStream_t s) {
  HIPCK(k_lift_launch(c, m, nullptr, pt, level, 0, level, 0, s));
  HIPCK(ntt_rows(c, pt, 1, 0, level, 0, false, s));
  return FESC_OK;
}

}  // namespace fesc
