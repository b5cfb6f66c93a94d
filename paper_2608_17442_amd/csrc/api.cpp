// extern "C" entry points: argument validation, then dispatch to the
// launchers.  No allocation happens here except through scratch_get().
#include <string>

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
