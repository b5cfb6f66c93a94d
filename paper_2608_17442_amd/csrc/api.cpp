// extern "C" entry points: argument validation, then dispatch to the
// launchers.  No allocation happens here except through scratch_get().
#include <algorithm>
#include <cmath>
#include <string>
#include <vector>

#include "fesc_internal.hpp"

using namespace fesc;

namespace {

inline hipStream_t S(void* s) { return reinterpret_cast<hipStream_t>(s); }

int check_rows(const fesc_ctx* c, uint32_t limbs, uint32_t prime0) {
  if (!c) return fail(FESC_ERR_ARG, "null context");
  if (limbs == 0 || (size_t)prime0 + limbs > c->ext_count())
    return fail(FESC_ERR_ARG, "prime range [" + std::to_string(prime0) + ", " +
                                  std::to_string(prime0 + limbs) + ") outside the " +
                                  std::to_string(c->ext_count()) + " extended primes");
  return FESC_OK;
}

}  // namespace

extern "C" {

int fesc_ctx_create(const fesc_params* params, fesc_ctx** out) { return create(params, out); }

void fesc_ctx_destroy(fesc_ctx* ctx) { destroy(ctx); }

const char* fesc_last_error(void) { return last_error(); }

int fesc_find_primes(uint32_t log_n, uint32_t bits, uint32_t count, uint64_t* out) {
  if (!out || bits < log_n + 2 || bits > 62) return fail(FESC_ERR_ARG, "bad prime request");
  const uint64_t m = 2ull << log_n;
  uint64_t c = (((1ull << bits) - 1) / m) * m + 1;
  if (c >= (1ull << bits)) c -= m;
  uint32_t found = 0;
  for (; found < count && c > m; c -= m)
    if (h_is_prime(c)) out[found++] = c;
  return (int)found;
}

int fesc_root_of_unity(uint32_t log_n, uint64_t q, uint64_t* psi) {
  if (!psi || log_n < 1 || log_n > 30 || q % (2ull << log_n) != 1 || !h_is_prime(q))
    return fail(FESC_ERR_ARG, "q must be a prime = 1 mod 2N");
  *psi = h_min_root(q, log_n);
  return FESC_OK;
}

int fesc_get_psi(const fesc_ctx* ctx, uint32_t idx, uint64_t* psi) {
  if (!ctx || !psi || idx >= ctx->ext_count()) return fail(FESC_ERR_ARG, "bad prime index");
  *psi = ctx->psi[idx];
  return FESC_OK;
}

static int ntt_common(fesc_ctx* ctx, uint64_t* d, uint32_t batch, size_t batch_stride,
                      uint32_t limbs, size_t limb_stride, uint32_t prime0, void* stream,
                      bool inverse) {
  int rc = check_rows(ctx, limbs, prime0);
  if (rc) return rc;
  if (!d || batch == 0 || batch > 65535 || limbs > 65535)
    return fail(FESC_ERR_ARG, "bad NTT batch");
  return hip_check(launch_ntt(ctx, d, batch, batch_stride, limbs, limb_stride, prime0, inverse,
                              S(stream)),
                   inverse ? "ntt_inv launch" : "ntt_fwd launch");
}

int fesc_ntt_fwd(fesc_ctx* ctx, uint64_t* d, uint32_t batch, size_t batch_stride,
                 uint32_t limbs, size_t limb_stride, uint32_t prime0, void* stream) {
  return ntt_common(ctx, d, batch, batch_stride, limbs, limb_stride, prime0, stream, false);
}

int fesc_ntt_inv(fesc_ctx* ctx, uint64_t* d, uint32_t batch, size_t batch_stride,
                 uint32_t limbs, size_t limb_stride, uint32_t prime0, void* stream) {
  return ntt_common(ctx, d, batch, batch_stride, limbs, limb_stride, prime0, stream, true);
}

int fesc_mac(fesc_ctx* ctx, const uint64_t* a, const uint64_t* b, uint64_t* out,
             uint32_t pairs, size_t pair_stride, uint32_t limbs, uint32_t prime0,
             void* stream) {
  int rc = check_rows(ctx, limbs, prime0);
  if (rc) return rc;
  if (!a || !b || !out || pairs == 0) return fail(FESC_ERR_ARG, "bad MAC arguments");
  return hip_check(launch_mac(ctx, a, b, out, pairs, pair_stride, limbs, prime0, S(stream)),
                   "mac launch");
}

}  // extern "C"

// ------------------------------------------------------ ciphertext operations

namespace fesc {
int op_rotate_many(Context* c, const uint64_t* in, uint32_t count, const int32_t* steps,
                   uint64_t* const* outs, uint32_t level, hipStream_t s);
int op_mul_relin(Context* c, const uint64_t* a, const uint64_t* b, uint64_t* out,
                 uint32_t level, hipStream_t s);
int op_rescale(Context* c, const uint64_t* in, uint64_t* out, uint32_t level, hipStream_t s);
int op_encrypt(Context* c, const int8_t* sk, const int64_t* m, const uint64_t* a,
               const int64_t* e, uint64_t* ct, uint32_t level, hipStream_t s);
int op_plain_from_coeffs(Context* c, const int64_t* m, uint64_t* pt, uint32_t level,
                         hipStream_t s);
uint32_t galois_of_step(const Context* c, int32_t step);
int op_scan_contract(Context* c, const uint64_t* const* h, const uint64_t* const* decay,
                     const uint64_t* const* cfac, uint32_t K, uint32_t T, uint32_t d_s,
                     uint64_t* const* out, uint32_t level, hipStream_t s);
int encode(uint32_t log_n, const double* re, const double* im, double scale, int64_t* out);
int calib_valu(Context* c, int kind, uint32_t iters, double* rate, hipStream_t s);
int calib_hbm(Context* c, int kind, size_t bytes, double* rate, hipStream_t s);
int op_heconv(Context* c, const uint64_t* q, uint32_t taps, const int32_t* deltas,
              const uint64_t* const* masks, const uint64_t* bias, uint64_t* out, uint32_t level,
              hipStream_t s);
int op_post_ssm(Context* c, const uint64_t* m, const uint64_t* x_skip, const uint64_t* d_skip,
                const uint64_t* g, uint64_t* out, uint32_t level, hipStream_t s);
int op_add_plain(Context* c, const uint64_t* ct, const uint64_t* pt, uint64_t* out,
                 uint32_t level, hipStream_t s);
int c2m_level(const uint64_t* q, uint32_t level, uint32_t ell, uint32_t sigma, double delta,
              double bmax, uint32_t* out);
int scratch_slots(Context* c, uint64_t** cts, uint32_t* cap);
int op_encode_plain(Context* c, const double2* z, uint32_t count, double scale, uint64_t* pt,
                    uint32_t level, uint64_t* slots, uint32_t nslots, hipStream_t s, bool ext);
int op_decode_plain(Context* c, const uint64_t* pt, uint32_t count, uint32_t level, double scale,
                    double2* z, uint64_t* slots, uint32_t nslots, hipStream_t s);
int op_affine_scan(Context* c, uint64_t* const* a, uint64_t* const* s, uint32_t L,
                   uint32_t chunks, uint32_t level, bool states_only, uint32_t* out_level,
                   hipStream_t st);
int op_affine_scan_level(Context* c, uint32_t L, uint32_t level, bool states_only,
                         uint32_t* out_level, uint64_t* products);
size_t affine_scan_network(uint32_t L, bool states_only, uint32_t* nodes, size_t cap);
size_t affine_scan_resident_program(uint32_t L, uint32_t block, uint32_t level, uint64_t* words,
                                    size_t cap, int* err);
size_t affine_scan_program(uint32_t L, uint32_t chunks, bool states_only, uint32_t level,
                           uint64_t* words, size_t cap, int* err);
size_t affine_scan_resident_words(const Context* c, uint32_t L, uint32_t chunks, uint32_t block,
                                  uint32_t level);
int op_affine_scan_resident_level(Context* c, uint32_t L, uint32_t block, uint32_t level,
                                  uint32_t* out_level, uint64_t* products);
int op_affine_scan_resident(Context* c, const uint64_t* const* a, const uint64_t* const* s,
                            uint32_t L, uint32_t chunks, uint32_t block, uint64_t* const* h,
                            uint32_t level, uint64_t* ws, uint32_t* out_level, hipStream_t st);
}  // namespace fesc

#include "ops.hpp"

namespace {

int check_level(const fesc_ctx* c, uint32_t level, uint32_t min_level = 1) {
  if (!c) return fail(FESC_ERR_ARG, "null context");
  if (level < min_level || level > c->L)
    return fail(FESC_ERR_LEVEL, "level " + std::to_string(level) + " outside [" +
                                    std::to_string(min_level) + ", " + std::to_string(c->L) + "]");
  return FESC_OK;
}

}  // namespace

extern "C" {

int fesc_add(fesc_ctx* ctx, const uint64_t* a, const uint64_t* b, uint64_t* out, uint32_t level,
             void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!a || !b || !out) return fail(FESC_ERR_ARG, "null buffer");
  return hip_check(k_binary_launch(ctx, a, b, out, 2 * level, 1, 0, S(stream)), "add");
}

int fesc_sub(fesc_ctx* ctx, const uint64_t* a, const uint64_t* b, uint64_t* out, uint32_t level,
             void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!a || !b || !out) return fail(FESC_ERR_ARG, "null buffer");
  return hip_check(k_binary_launch(ctx, a, b, out, 2 * level, 1, 1, S(stream)), "sub");
}

int fesc_mul_plain(fesc_ctx* ctx, const uint64_t* ct, const uint64_t* pt, uint64_t* out,
                   uint32_t level, void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!ct || !pt || !out) return fail(FESC_ERR_ARG, "null buffer");
  return hip_check(k_mul_plain_launch(ctx, ct, pt, out, level, S(stream)), "mul_plain");
}

int fesc_mul_monomial(fesc_ctx* ctx, const uint64_t* in, uint64_t* out, uint32_t level,
                      uint32_t k, void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!in || !out) return fail(FESC_ERR_ARG, "null buffer");
  return hip_check(k_monomial_launch(ctx, in, out, level, k % (2 * ctx->n), S(stream)),
                   "mul_monomial");
}

int fesc_mul_relin(fesc_ctx* ctx, const uint64_t* a, const uint64_t* b, uint64_t* out,
                   uint32_t level, void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!a || !b || !out) return fail(FESC_ERR_ARG, "null buffer");
  return op_mul_relin(ctx, a, b, out, level, S(stream));
}

int fesc_mul_relin_rescale(fesc_ctx* ctx, uint32_t count, const uint64_t* const* a,
                           const uint64_t* const* b, uint64_t* const* out, uint32_t level,
                           void* stream) {
  int rc = check_level(ctx, level, 2);
  if (rc) return rc;
  if (count == 0) return FESC_OK;
  if (!a || !b || !out || count > (1u << 20)) return fail(FESC_ERR_ARG, "bad product arguments");
  // out_i may be a_i or b_i; no output may be another product's operand or output
  std::vector<std::pair<const void*, uint32_t>> outs;
  for (uint32_t i = 0; i < count; ++i) {
    if (!a[i] || !b[i] || !out[i]) return fail(FESC_ERR_ARG, "null buffer");
    outs.emplace_back(out[i], i);
  }
  std::sort(outs.begin(), outs.end());
  for (uint32_t i = 1; i < count; ++i)
    if (outs[i].first == outs[i - 1].first)
      return fail(FESC_ERR_ARG, "product outputs must be distinct");
  for (uint32_t i = 0; i < count; ++i)
    for (const void* p : {(const void*)a[i], (const void*)b[i]}) {
      auto it = std::lower_bound(outs.begin(), outs.end(), std::make_pair(p, 0u));
      if (it != outs.end() && it->first == p && it->second != i)
        return fail(FESC_ERR_ARG, "an output aliases another product's operand");
    }
  if (!ctx->keys.count(0)) return fail(FESC_ERR_NO_KEY, "no relinearisation key");
  return op_prod_rescale_many(ctx, count, a, b, out, nullptr, level, level - 1, S(stream));
}

int fesc_rescale(fesc_ctx* ctx, const uint64_t* in, uint64_t* out, uint32_t level,
                 void* stream) {
  int rc = check_level(ctx, level, 2);
  if (rc) return rc;
  if (!in || !out) return fail(FESC_ERR_ARG, "null buffer");
  return op_rescale(ctx, in, out, level, S(stream));
}

int fesc_galois_element(const fesc_ctx* ctx, int32_t step, uint32_t* elt) {
  if (!ctx || !elt) return fail(FESC_ERR_ARG, "null argument");
  *elt = galois_of_step(ctx, step);
  return FESC_OK;
}

int fesc_rotate(fesc_ctx* ctx, const uint64_t* in, uint64_t* out, uint32_t level, int32_t step,
                void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!in || !out) return fail(FESC_ERR_ARG, "null buffer");
  uint64_t* outs[1] = {out};
  return op_rotate_many(ctx, in, 1, &step, outs, level, S(stream));
}

int fesc_rotate_hoisted(fesc_ctx* ctx, const uint64_t* in, uint32_t count, const int32_t* steps,
                        uint64_t* const* outs, uint32_t level, void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!in || !steps || !outs || count == 0) return fail(FESC_ERR_ARG, "bad hoisted arguments");
  for (uint32_t r = 0; r < count; ++r)
    if (!outs[r]) return fail(FESC_ERR_ARG, "null output");
  return op_rotate_many(ctx, in, count, steps, outs, level, S(stream));
}

static int check_rotate_batch(fesc_ctx* ctx, uint32_t count, const uint64_t* const* ins,
                              const int32_t* steps, uint64_t* const* outs, uint32_t level) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!ins || !steps || !outs || count == 0) return fail(FESC_ERR_ARG, "bad batch arguments");
  for (uint32_t i = 0; i < count; ++i) {
    if (!ins[i] || !outs[i]) return fail(FESC_ERR_ARG, "null buffer");
    for (uint32_t j = 0; j < count; ++j)
      if (outs[i] == ins[j]) return fail(FESC_ERR_ARG, "batched outputs must not alias inputs");
  }
  for (uint32_t i = 0; i < count; ++i) {
    const uint32_t g = galois_of_step(ctx, steps[i]);
    if (g != 1 && !ctx->keys.count(g))
      return fail(FESC_ERR_NO_KEY, "no switching key for Galois element " + std::to_string(g));
  }
  return FESC_OK;
}

int fesc_rotate_batch(fesc_ctx* ctx, uint32_t count, const uint64_t* const* ins,
                      const int32_t* steps, uint64_t* const* outs, uint32_t level,
                      void* stream) {
  int rc = check_rotate_batch(ctx, count, ins, steps, outs, level);
  if (rc) return rc;
  return op_rotate_batch(ctx, count, ins, steps, outs, nullptr, level, S(stream));
}

int fesc_rotate_batch_noalloc(fesc_ctx* ctx, uint32_t count, const uint64_t* const* ins,
                              const int32_t* steps, uint64_t* const* outs, uint32_t level,
                              void* stream) {
  if (ctx && level >= 1 && level <= ctx->L &&
      rotate_scratch_words(ctx, level) * sizeof(uint64_t) > static_scratch_bytes())
    return fail(FESC_ERR_ARG, "one rotation at level " + std::to_string(level) + " needs " +
                                  std::to_string(rotate_scratch_words(ctx, level) * 8) +
                                  " bytes of scratch; the static scratch holds " +
                                  std::to_string(static_scratch_bytes()));
  int rc = check_rotate_batch(ctx, count, ins, steps, outs, level);
  if (rc) return rc;
  return op_rotate_batch_static(ctx, count, ins, steps, outs, level, S(stream));
}

static int check_galois(const fesc_ctx* ctx, uint32_t galois_elt) {
  if (galois_elt != 0 && (galois_elt % 2 == 0 || galois_elt >= 2 * ctx->n || galois_elt == 1))
    return fail(FESC_ERR_ARG, "Galois element must be 0 or odd in (1, 2N)");
  return FESC_OK;
}

int fesc_keygen(fesc_ctx* ctx, uint32_t galois_elt, const int8_t* s, const uint64_t* a,
                const int64_t* e, void* stream) {
  if (!ctx || !s || !a || !e) return fail(FESC_ERR_ARG, "null argument");
  int rc = check_galois(ctx, galois_elt);
  if (rc) return rc;
  return op_keygen(ctx, galois_elt, s, a, e, nullptr, S(stream));
}

int fesc_keygen_seeded(fesc_ctx* ctx, uint32_t galois_elt, const int8_t* s,
                       const uint64_t* seed, const int64_t* e, void* stream) {
  if (!ctx || !s || !seed || !e) return fail(FESC_ERR_ARG, "null argument");
  int rc = check_galois(ctx, galois_elt);
  if (rc) return rc;
  return op_keygen(ctx, galois_elt, s, nullptr, e, seed, S(stream));
}

int fesc_key_load(fesc_ctx* ctx, uint32_t galois_elt, const uint64_t* key, void* stream) {
  if (!ctx || !key) return fail(FESC_ERR_ARG, "null argument");
  int rc = check_galois(ctx, galois_elt);
  if (rc) return rc;
  uint64_t* dst;
  if ((rc = key_buffer(ctx, galois_elt, full_key_words(ctx), &dst))) return rc;
  return hip_check(hipMemcpyAsync(dst, key, full_key_words(ctx) * 8, hipMemcpyDeviceToDevice,
                                  S(stream)),
                   "key_load");
}

int fesc_key_upload(fesc_ctx* ctx, uint32_t galois_elt, const uint64_t* host_key,
                    uint32_t key_level, void* stream) {
  if (!ctx || !host_key) return fail(FESC_ERR_ARG, "null argument");
  int rc = check_galois(ctx, galois_elt);
  if (rc) return rc;
  if (key_level < 1 || key_level > ctx->L)
    return fail(FESC_ERR_LEVEL, "key_level must be in 1 .. L");
  uint64_t* dst;
  if ((rc = key_buffer(ctx, galois_elt, full_key_words(ctx), &dst))) return rc;
  const size_t n = ctx->n, E = ctx->L + ctx->alpha, Ek = key_level + ctx->alpha;
  const uint32_t dk = (key_level + ctx->alpha - 1) / ctx->alpha;
  hipStream_t st = S(stream);
  // rows the prefix key does not hold stay zero; the key-switch driver
  // refuses this key above key_level
  rc = hip_check(hipMemsetAsync(dst, 0, full_key_words(ctx) * 8, st), "key_upload");
  for (uint32_t j = 0; j < dk && !rc; ++j) {
    const uint64_t* src = host_key + (size_t)j * Ek * 2 * n;
    uint64_t* d = dst + (size_t)j * E * 2 * n;
    rc = hip_check(hipMemcpyAsync(d, src, (size_t)key_level * 2 * n * 8, hipMemcpyHostToDevice,
                                  st), "key_upload");
    if (!rc)
      rc = hip_check(hipMemcpyAsync(d + (size_t)ctx->L * 2 * n, src + (size_t)key_level * 2 * n,
                                    (size_t)ctx->alpha * 2 * n * 8, hipMemcpyHostToDevice, st),
                     "key_upload");
  }
  if (!rc) rc = hip_check(hipStreamSynchronize(st), "key_upload");
  if (rc) return rc;
  if (key_level < ctx->L) ctx->key_cap[dst] = key_level;
  return FESC_OK;
}

int fesc_key_store(fesc_ctx* ctx, uint32_t galois_elt, uint64_t* key, void* stream) {
  if (!ctx || !key) return fail(FESC_ERR_ARG, "null argument");
  auto it = ctx->keys.find(galois_elt);
  if (it == ctx->keys.end()) return fail(FESC_ERR_NO_KEY, "no such key");
  if (ctx->key_seeded.count(it->second))  // expanded to the full layout
    return hip_check(k_key_expand_launch(ctx, it->second, key, S(stream)), "key_store");
  return hip_check(hipMemcpyAsync(key, it->second, full_key_words(ctx) * 8,
                                  hipMemcpyDeviceToDevice, S(stream)),
                   "key_store");
}

int fesc_encrypt_sk(fesc_ctx* ctx, const int8_t* s, const int64_t* m, const uint64_t* a,
                    const int64_t* e, uint64_t* ct, uint32_t level, void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!s || !m || !a || !e || !ct) return fail(FESC_ERR_ARG, "null buffer");
  return op_encrypt(ctx, s, m, a, e, ct, level, S(stream));
}

int fesc_plain_from_coeffs(fesc_ctx* ctx, const int64_t* m, uint64_t* pt, uint32_t level,
                           void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!m || !pt) return fail(FESC_ERR_ARG, "null buffer");
  return op_plain_from_coeffs(ctx, m, pt, level, S(stream));
}

int fesc_encode(uint32_t log_n, const double* re, const double* im, double scale,
                int64_t* coeffs) {
  return encode(log_n, re, im, scale, coeffs);
}

int fesc_scan_contract(fesc_ctx* ctx, const uint64_t* const* h, const uint64_t* const* decay,
                       const uint64_t* const* cfac, uint32_t chunks, uint32_t tokens,
                       uint32_t d_state, uint64_t* const* out, uint32_t level, void* stream) {
  int rc = check_level(ctx, level, decay ? 3 : 2);
  if (rc) return rc;
  if (!h || !cfac || !out || chunks == 0 || tokens == 0 || d_state == 0 ||
      (d_state & (d_state - 1)) || d_state > ctx->n / 2 || (uint64_t)chunks * tokens > (1u << 20))
    return fail(FESC_ERR_ARG, "bad scan-contract arguments");
  const size_t KT = (size_t)chunks * tokens;
  std::vector<const void*> outs;
  for (size_t k = 0; k < KT; ++k) {
    if (!h[k] || (decay && !decay[k]) || !cfac[k] || !out[k])
      return fail(FESC_ERR_ARG, "null buffer");
    outs.push_back(out[k]);
  }
  // the outputs are also the reduction's workspace
  std::sort(outs.begin(), outs.end());
  if (std::adjacent_find(outs.begin(), outs.end()) != outs.end())
    return fail(FESC_ERR_ARG, "scan-contract outputs must be distinct");
  for (size_t k = 0; k < KT; ++k)
    for (const void* p : {(const void*)h[k], decay ? (const void*)decay[k] : nullptr,
                          (const void*)cfac[k]})
      if (p && std::binary_search(outs.begin(), outs.end(), p))
        return fail(FESC_ERR_ARG, "scan-contract outputs must not alias inputs");
  if (!ctx->keys.count(0)) return fail(FESC_ERR_NO_KEY, "no relinearisation key");
  for (uint32_t st = d_state / 2; st >= 1; st /= 2)
    if (!ctx->keys.count(galois_of_step(ctx, (int32_t)st)))
      return fail(FESC_ERR_NO_KEY, "no key for rotation " + std::to_string(st));
  if (chunks >= 2 && !ctx->keys.count(2 * ctx->n - 1))
    return fail(FESC_ERR_NO_KEY, "no conjugation key");
  return op_scan_contract(ctx, h, decay, cfac, chunks, tokens, d_state, out, level, S(stream));
}

static int scan_args(fesc_ctx* ctx, uint32_t L, uint32_t chunks, uint32_t level) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (L == 0 || chunks == 0 || (uint64_t)L * chunks > (1u << 24))
    return fail(FESC_ERR_ARG, "need L >= 1, chunks >= 1 and L * chunks <= 2^24");
  if (!ctx->keys.count(0)) return fail(FESC_ERR_NO_KEY, "no relinearisation key");
  return FESC_OK;
}

static bool distinct(std::vector<const void*> p) {
  std::sort(p.begin(), p.end());
  return std::adjacent_find(p.begin(), p.end()) == p.end();
}

int fesc_affine_scan_info(fesc_ctx* ctx, uint32_t L, uint32_t level, uint32_t flags,
                          uint32_t* out_level, uint64_t* key_switches) {
  int rc = scan_args(ctx, L, 1, level);
  if (rc) return rc;
  if (!out_level || !key_switches || (flags & ~FESC_SCAN_STATES_ONLY))
    return fail(FESC_ERR_ARG, "bad argument");
  return op_affine_scan_level(ctx, L, level, flags & FESC_SCAN_STATES_ONLY, out_level,
                              key_switches);
}

int fesc_affine_scan_network(uint32_t L, uint32_t flags, uint32_t* nodes, size_t cap,
                             size_t* count) {
  if (!count || L == 0 || L > (1u << 20) || (flags & ~FESC_SCAN_STATES_ONLY))
    return fail(FESC_ERR_ARG, "bad scan-network arguments");
  *count = affine_scan_network(L, flags & FESC_SCAN_STATES_ONLY, nodes, cap);
  if (nodes && *count > cap) return fail(FESC_ERR_ARG, "node array too small");
  return FESC_OK;
}

int fesc_affine_scan_program(uint32_t L, uint32_t chunks, uint32_t flags, uint64_t* words,
                             size_t cap, size_t* count) {
  if (!count || L == 0 || L > (1u << 16) || chunks == 0 || (uint64_t)chunks * L > (1u << 20) ||
      (flags & ~FESC_SCAN_STATES_ONLY))
    return fail(FESC_ERR_ARG, "bad scan-program arguments");
  int err = FESC_OK;
  *count = affine_scan_program(L, chunks, flags & FESC_SCAN_STATES_ONLY, 64, words, cap, &err);
  if (err) return err;
  if (words && *count > cap) return fail(FESC_ERR_ARG, "program array too small");
  return FESC_OK;
}

int fesc_affine_scan_resident_program(uint32_t L, uint32_t block, uint64_t* words, size_t cap,
                                      size_t* count) {
  if (!count || L == 0 || L > (1u << 16) || block == 0 || block > L)
    return fail(FESC_ERR_ARG, "bad resident-program arguments");
  int err = FESC_OK;
  *count = affine_scan_resident_program(L, block, 64, words, cap, &err);
  if (err) return err;
  if (words && *count > cap) return fail(FESC_ERR_ARG, "program array too small");
  return FESC_OK;
}

int fesc_affine_scan(fesc_ctx* ctx, uint64_t* const* a, uint64_t* const* s, uint32_t L,
                     uint32_t chunks, uint32_t level, uint32_t flags, uint32_t* out_level,
                     void* stream) {
  int rc = scan_args(ctx, L, chunks, level);
  if (rc) return rc;
  if (!a || !s || !out_level) return fail(FESC_ERR_ARG, "null argument");
  if (flags & ~FESC_SCAN_STATES_ONLY) return fail(FESC_ERR_ARG, "unknown flags");
  std::vector<const void*> all;
  for (size_t i = 0; i < (size_t)L * chunks; ++i) {
    if (!a[i] || !s[i]) return fail(FESC_ERR_ARG, "null buffer");
    all.push_back(a[i]);
    all.push_back(s[i]);
  }
  if (!distinct(all)) return fail(FESC_ERR_ARG, "scan buffers must be distinct");
  return op_affine_scan(ctx, a, s, L, chunks, level, flags & FESC_SCAN_STATES_ONLY, out_level,
                        S(stream));
}

int fesc_affine_scan_resident_info(fesc_ctx* ctx, uint32_t L, uint32_t chunks, uint32_t block,
                                   uint32_t level, uint32_t* out_level, size_t* workspace_bytes,
                                   uint64_t* key_switches) {
  int rc = scan_args(ctx, L, chunks, level);
  if (rc) return rc;
  if (block == 0 || !out_level || !workspace_bytes) return fail(FESC_ERR_ARG, "bad argument");
  if ((rc = op_affine_scan_resident_level(ctx, L, block, level, out_level, key_switches)))
    return rc;
  *workspace_bytes = affine_scan_resident_words(ctx, L, chunks, block, level) * 8;
  return FESC_OK;
}

int fesc_affine_scan_resident(fesc_ctx* ctx, const uint64_t* const* a, const uint64_t* const* s,
                              uint32_t L, uint32_t chunks, uint32_t block, uint64_t* const* h,
                              uint32_t level, void* workspace, size_t workspace_bytes,
                              void* stream) {
  uint32_t lo;
  size_t need;
  int rc = fesc_affine_scan_resident_info(ctx, L, chunks, block, level, &lo, &need, nullptr);
  if (rc) return rc;
  if (!a || !s || !h) return fail(FESC_ERR_ARG, "null argument");
  if (need && (!workspace || workspace_bytes < need))
    return fail(FESC_ERR_ARG, "workspace of " + std::to_string(need) + " bytes needed");
  std::vector<const void*> all;
  for (size_t i = 0; i < (size_t)L * chunks; ++i) {
    if (!a[i] || !s[i] || !h[i]) return fail(FESC_ERR_ARG, "null buffer");
    all.push_back(a[i]);
    all.push_back(s[i]);
    all.push_back(h[i]);
  }
  if (!distinct(all)) return fail(FESC_ERR_ARG, "scan buffers must be distinct");
  uint32_t got;
  return op_affine_scan_resident(ctx, a, s, L, chunks, block, h, level,
                                 static_cast<uint64_t*>(workspace), &got, S(stream));
}

int fesc_heconv(fesc_ctx* ctx, const uint64_t* q, uint32_t taps, const int32_t* deltas,
                const uint64_t* const* masks, const uint64_t* bias, uint64_t* out,
                uint32_t level, void* stream) {
  int rc = check_level(ctx, level, 2);
  if (rc) return rc;
  if (!q || !deltas || !masks || !out || taps == 0 || taps > kMaxConvTaps)
    return fail(FESC_ERR_ARG, "bad HEConv arguments (1 <= taps <= 16)");
  if (out == q) return fail(FESC_ERR_ARG, "HEConv output must not alias its input");
  for (uint32_t r = 0; r < taps; ++r) {
    if (!masks[r]) return fail(FESC_ERR_ARG, "null mask");
    if (deltas[r] == FESC_CONJ) return fail(FESC_ERR_ARG, "HEConv offsets are rotations");
    const uint32_t g = galois_of_step(ctx, deltas[r]);
    if (g != 1 && !ctx->keys.count(g))
      return fail(FESC_ERR_NO_KEY, "no key for rotation " + std::to_string(deltas[r]));
  }
  return op_heconv(ctx, q, taps, deltas, masks, bias, out, level, S(stream));
}

int fesc_post_ssm(fesc_ctx* ctx, const uint64_t* m, const uint64_t* x_skip,
                  const uint64_t* d_skip, const uint64_t* g, uint64_t* out, uint32_t level,
                  void* stream) {
  int rc = check_level(ctx, level, 3);
  if (rc) return rc;
  if (!m || !x_skip || !d_skip || !g || !out) return fail(FESC_ERR_ARG, "null buffer");
  if (!ctx->keys.count(0)) return fail(FESC_ERR_NO_KEY, "no relinearisation key");
  return op_post_ssm(ctx, m, x_skip, d_skip, g, out, level, S(stream));
}

int fesc_add_plain(fesc_ctx* ctx, const uint64_t* ct, const uint64_t* pt, uint64_t* out,
                   uint32_t level, void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!ct || !pt || !out) return fail(FESC_ERR_ARG, "null buffer");
  return op_add_plain(ctx, ct, pt, out, level, S(stream));
}

static int encode_plain(fesc_ctx* ctx, const double* z, uint32_t count, double scale,
                        uint64_t* pt, uint32_t level, void* stream, bool ext) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!(std::fabs(scale) < 4611686018427387904.0)) return fail(FESC_ERR_ARG, "bad scale");
  if (count == 0) return FESC_OK;
  if (!z || !pt) return fail(FESC_ERR_ARG, "null buffer");
  uint64_t* slots;
  uint32_t cap;
  if ((rc = scratch_slots(ctx, &slots, &cap))) return rc;
  return op_encode_plain(ctx, reinterpret_cast<const double2*>(z), count, scale, pt, level, slots,
                         cap, S(stream), ext);
}

int fesc_encode_plain(fesc_ctx* ctx, const double* z, uint32_t count, double scale, uint64_t* pt,
                      uint32_t level, void* stream) {
  return encode_plain(ctx, z, count, scale, pt, level, stream, false);
}

int fesc_encode_plain_ext(fesc_ctx* ctx, const double* z, uint32_t count, double scale,
                          uint64_t* pt, uint32_t level, void* stream) {
  return encode_plain(ctx, z, count, scale, pt, level, stream, true);
}

int fesc_decode_plain(fesc_ctx* ctx, const uint64_t* pt, uint32_t count, uint32_t level,
                      double scale, double* z, void* stream) {
  int rc = check_level(ctx, level);
  if (rc) return rc;
  if (!(std::fabs(scale) > 0.0 && std::fabs(scale) < HUGE_VAL)) return fail(FESC_ERR_ARG, "bad scale");
  if (count == 0) return FESC_OK;
  if (!z || !pt) return fail(FESC_ERR_ARG, "null buffer");
  uint64_t* slots;
  uint32_t cap;
  if ((rc = scratch_slots(ctx, &slots, &cap))) return rc;
  return op_decode_plain(ctx, pt, count, level, scale, reinterpret_cast<double2*>(z), slots, cap,
                         S(stream));
}

int fesc_c2m_level(const uint64_t* q, uint32_t level, uint32_t ell, uint32_t sigma, double delta,
                   double bmax, uint32_t* out_level) {
  return c2m_level(q, level, ell, sigma, delta, bmax, out_level);
}

int fesc_calib_valu(fesc_ctx* ctx, int kind, uint32_t iters, double* rate, void* stream) {
  if (!ctx || !rate) return fail(FESC_ERR_ARG, "null argument");
  return calib_valu(ctx, kind, iters, rate, S(stream));
}

int fesc_calib_hbm(fesc_ctx* ctx, int kind, size_t bytes, double* rate, void* stream) {
  if (!ctx || !rate) return fail(FESC_ERR_ARG, "null argument");
  return calib_hbm(ctx, kind, bytes, rate, S(stream));
}

}  // extern "C"
