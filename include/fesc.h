/*
 * fesc.h - C ABI of the MI355X (gfx950) RNS-CKKS linear hot path of FESC,
 * "Remodeling Long-Context Private Inference with Encrypted State-Space
 * Models" (arXiv 2608.17442).
 *
 * The paper's encrypted kernels are built from the CKKS primitives of its
 * Sec. 4.1 table (add, ptmul, ctmul, rot, conj), from key switching through
 * special primes and rescaling by one prime per level (Sec. 2.1), and from
 * the BSGS plaintext-ciphertext projection (Appendix "Projection Kernel
 * Breakdown").  This header exposes those computations on one GPU.
 *
 * Conventions common to every call
 * --------------------------------
 *  - Ring R = Z[X]/(X^N + 1), N = 2^log_n, 12 <= log_n <= 16.
 *  - Moduli are given by the caller: L ciphertext primes q_0..q_{L-1} and
 *    alpha special primes p_0..p_{alpha-1}, each below 2^50 and = 1 mod 2N.
 *    The "extended prime index" of q_i is i and of p_k is L + k.
 *  - Every residue is a uint64 in [0, q).  Polynomials are in evaluation
 *    (NTT) form at the API unless a call says otherwise:
 *        A[j] = sum_k a_k psi^((2 brv(j) + 1) k)  mod q,
 *    psi the smallest primitive 2N-th root of unity mod q, brv the log_n-bit
 *    reversal (the output order of the radix-2 Cooley-Tukey network).
 *  - Plaintext at level l:  uint64[l][N].
 *    Ciphertext at level l: uint64[l][2][N] (limb-major; c0 and c1 of limb i
 *    are adjacent), so the ciphertext at level l-1 is a prefix.
 *    Switching key:          uint64[dnum][L+alpha][2][N] (digit, extended
 *    prime, (b, a), coefficient); digit j covers q_{j*alpha}..q_{(j+1)alpha-1}.
 *  - Data pointers (polynomials, ciphertexts, keys) are DEVICE pointers owned
 *    by the caller; the library never frees them.  `stream` is a hipStream_t
 *    (NULL: the null stream); all calls are asynchronous on it.  One context
 *    must not be used from two streams at the same time (its scratch memory
 *    is shared).
 *  - Return value: FESC_OK (0) or a negative FESC_ERR_* code.  Argument
 *    errors are detected before any launch, so nothing is written;
 *    fesc_last_error() returns a thread-local description.
 */
#ifndef FESC_H
#define FESC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FESC_OK 0
#define FESC_ERR_ARG (-1)    /* malformed argument */
#define FESC_ERR_LEVEL (-2)  /* level out of range for the operation */
#define FESC_ERR_NO_KEY (-3) /* required switching key not loaded */
#define FESC_ERR_OOM (-4)    /* device allocation failed */
#define FESC_ERR_HIP (-5)    /* HIP runtime error */

typedef struct fesc_ctx fesc_ctx;

typedef struct fesc_params {
  uint32_t log_n;     /* N = 2^log_n, 12..16 */
  uint32_t num_q;     /* L >= 1 */
  uint32_t num_p;     /* alpha >= 1, L + alpha <= 64 */
  uint32_t dnum;      /* must equal ceil(L / alpha) */
  const uint64_t* q;  /* host array of L primes */
  const uint64_t* p;  /* host array of alpha primes */
} fesc_params;

/* Context: validates the primes (prime, < 2^50, = 1 mod 2N, distinct),
 * derives psi for each and uploads twiddle tables to the current device.
 * Errors: FESC_ERR_ARG, FESC_ERR_OOM, FESC_ERR_HIP. */
int fesc_ctx_create(const fesc_params* params, fesc_ctx** out);
void fesc_ctx_destroy(fesc_ctx* ctx);
const char* fesc_last_error(void);

/* Host helper: the `count` largest primes below 2^bits that are = 1 mod
 * 2^(log_n+1), in descending order, written to host array `out`.
 * Returns the number found (< count if the range is exhausted). */
int fesc_find_primes(uint32_t log_n, uint32_t bits, uint32_t count, uint64_t* out);

/* Host helper: psi, the smallest primitive 2N-th root of unity mod q
 * (q prime, = 1 mod 2N), which defines the transform of every call below. */
int fesc_root_of_unity(uint32_t log_n, uint64_t q, uint64_t* psi);

/* psi of extended prime `idx` of a context. */
int fesc_get_psi(const fesc_ctx* ctx, uint32_t idx, uint64_t* psi);

/* Negacyclic NTT in place (forward: coefficients -> evaluation form in the
 * order above; inverse: the exact inverse).  Row (b, i), b < batch, i < limbs,
 * starts at d + b*batch_stride + i*limb_stride (strides in uint64 words) and
 * uses extended prime prime0 + i.  Inputs must be canonical residues; outputs
 * are canonical.  Rows must not overlap.  FESC_ERR_ARG on bad indices. */
int fesc_ntt_fwd(fesc_ctx* ctx, uint64_t* d, uint32_t batch, size_t batch_stride,
                 uint32_t limbs, size_t limb_stride, uint32_t prime0, void* stream);
int fesc_ntt_inv(fesc_ctx* ctx, uint64_t* d, uint32_t batch, size_t batch_stride,
                 uint32_t limbs, size_t limb_stride, uint32_t prime0, void* stream);

/* Modular Hadamard multiply-accumulate (paper: elementwise product, Sec. 4.1):
 *   out[i][k] = sum_{j < pairs} a_j[i][k] * b_j[i][k]  mod prime(prime0 + i),
 * a_j = a + j*pair_stride, b_j = b + j*pair_stride, rows of N words,
 * i < limbs.  out (uint64[limbs][N]) must not overlap a or b. */
int fesc_mac(fesc_ctx* ctx, const uint64_t* a, const uint64_t* b, uint64_t* out,
             uint32_t pairs, size_t pair_stride, uint32_t limbs, uint32_t prime0,
             void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FESC_H */
