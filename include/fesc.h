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
 * psi and the evaluation order depend only on (N, prime), so two contexts of
 * one N whose ciphertext chains share the prefix q_0..q_{m-1} hold every
 * ciphertext or plaintext of level l <= m in the same buffer format: a buffer
 * may be passed from one to the other as it is.  A context over a short
 * prefix with few special primes (and its own switching keys) makes key
 * switching at low levels cheaper, its extended basis being l + alpha' rows.
 * Its keys must be drawn with randomness independent of the first context's
 * keys: two keys of one Galois element sharing their uniform rows and errors
 * differ on a digit row only by (P - P') s', which reveals the secret.
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
 * order above; inverse: the exact inverse).  The paper works in the ring
 * R_Q = Z_Q[X]/(X^N + 1) with N/2 complex slots (Sec. 2.1) and multiplies
 * ciphertexts and plaintexts elementwise (Sec. 4.1 table: ptmul, ctmul); the
 * evaluation form is the residue of a polynomial at the N roots of X^N + 1
 * mod q, where those products are pointwise, so this transform is the map
 * between the two forms (the paper does not print it; it is standard in RNS
 * CKKS).  Row (b, i), b < batch, i < limbs,
 * starts at d + b*batch_stride + i*limb_stride (strides in uint64 words) and
 * uses extended prime prime0 + i.  Inputs must be canonical residues; outputs
 * are canonical.  Rows must not overlap.  FESC_ERR_ARG on bad indices or an
 * empty batch (batch 0). */
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

/* ------------------------------------------------------------------------
 * Ciphertext operations (paper Sec. 4.1 table: add, ptmul, ctmul, rot, conj;
 * Sec. 2.1: rescale drops one prime).  `level` l counts the primes in use
 * (1 <= l <= L); FESC_ERR_LEVEL otherwise.  Unless stated, `out` may alias an
 * input (element-by-element operations).
 * ------------------------------------------------------------------------ */

/* add: out = a + b;  sub: out = a - b  (ciphertexts [l][2][N]). */
int fesc_add(fesc_ctx* ctx, const uint64_t* a, const uint64_t* b, uint64_t* out,
             uint32_t level, void* stream);
int fesc_sub(fesc_ctx* ctx, const uint64_t* a, const uint64_t* b, uint64_t* out,
             uint32_t level, void* stream);

/* ptmul: out = (c0 * pt, c1 * pt), pt a plaintext with at least l limbs
 * (its first l limbs are used).  The scale of the result is the product of
 * the scales; no rescale. */
int fesc_mul_plain(fesc_ctx* ctx, const uint64_t* ct, const uint64_t* pt, uint64_t* out,
                   uint32_t level, void* stream);

/* out = in * X^k (k taken mod 2N).  X^(N/2) multiplies every slot by i, so
 * k = N/2 and k = 3N/2 are the exact plaintext constants i and -i. */
int fesc_mul_monomial(fesc_ctx* ctx, const uint64_t* in, uint64_t* out, uint32_t level,
                      uint32_t k, void* stream);

/* ctmul with relinearisation: tensor (a0 b0, a0 b1 + a1 b0, a1 b1), then a
 * hybrid key switch of the s^2 part with the relinearisation key (Galois
 * element 0).  No rescale.  FESC_ERR_NO_KEY without the key. */
int fesc_mul_relin(fesc_ctx* ctx, const uint64_t* a, const uint64_t* b, uint64_t* out,
                   uint32_t level, void* stream);

/* Batched relinearised product with the rescale merged into the key switch
 * (the ciphertext products of HEScan: update construction
 * s = br(x) * br(B), affine composition and contraction, Sec. "On-Demand
 * Construction and Contraction"): for i < count,
 *     out_i = (P d_i + KS(d2_i) - FastBConv_{M->Q}(...)) * M^-1,  M = P q_{l-1}
 * i.e. relin(a_i * b_i) divided by P q_{l-1} in one ModDown whose conversion
 * takes q_{l-1} together with the special primes; the result is at level
 * l - 1 ([l-1][2][N]) and differs from rescale(mul_relin(a_i, b_i)) only in
 * the rounding (at most (alpha + 1) / 2 units of one conversion).  a, b, out:
 * host arrays of `count` device pointers; a_i and b_i at `level` >= 2 (a
 * longer operand enters through its leading limbs).  out_i may be a_i or
 * b_i; otherwise outputs are distinct and alias no operand (FESC_ERR_ARG).
 * 32 products share one key-switch launch sequence.  count = 0 is a no-op.
 * FESC_ERR_NO_KEY without the relinearisation key. */
int fesc_mul_relin_rescale(fesc_ctx* ctx, uint32_t count, const uint64_t* const* a,
                           const uint64_t* const* b, uint64_t* const* out, uint32_t level,
                           void* stream);

/* Rescale: out = round(in / q_{l-1}) at level l-1 (written as [l-1][2][N]);
 * l >= 2.  Computed as (c_i - [c mod q_{l-1}]_centred) * q_{l-1}^-1 mod q_i. */
int fesc_rescale(fesc_ctx* ctx, const uint64_t* in, uint64_t* out, uint32_t level,
                 void* stream);

/* Galois element of a rotation: 5^(step mod N/2) mod 2N (1 for the identity),
 * 2N-1 for step == FESC_CONJ. */
#define FESC_CONJ INT32_MIN
int fesc_galois_element(const fesc_ctx* ctx, int32_t step, uint32_t* elt);

/* rot: out = rho(in; step), the left rotation of the N/2 slots by `step`
 * (negative steps rotate right); step = 0 mod N/2 is an exact copy with no
 * key switch; step == FESC_CONJ conjugates.  The automorphism is applied as
 * an evaluation-form index permutation and the c1 part is key-switched with
 * the Galois key sigma_g(s) -> s (hybrid, centred basis conversion).
 * FESC_ERR_NO_KEY without the key.  out may alias in. */
int fesc_rotate(fesc_ctx* ctx, const uint64_t* in, uint64_t* out, uint32_t level, int32_t step,
                void* stream);

/* Hoisted rotations: `count` rotations of one ciphertext sharing a single
 * ModUp; steps is a host array, outs a host array of device pointers (each a
 * [l][2][N] ciphertext).  Results equal fesc_rotate residue for residue. */
int fesc_rotate_hoisted(fesc_ctx* ctx, const uint64_t* in, uint32_t count, const int32_t* steps,
                        uint64_t* const* outs, uint32_t level, void* stream);

/* Batched rotations of `count` independent ciphertexts: outs[i] =
 * rho(ins[i]; steps[i]) (FESC_CONJ allowed).  Up to 32 key switches run in
 * each launch of the pipeline, so the device is filled by the batch rather
 * than by one ciphertext.  ins / outs / steps are host arrays; outputs must
 * not alias inputs (FESC_ERR_ARG).  Results equal fesc_rotate residue for
 * residue. */
int fesc_rotate_batch(fesc_ctx* ctx, uint32_t count, const uint64_t* const* ins,
                      const int32_t* steps, uint64_t* const* outs, uint32_t level,
                      void* stream);

/* For callers that cannot allocate device memory (work under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * rotation batch of fesc_rotate_batch with the same arguments, results
 * (residue for residue) and errors, whose key-switch temporaries live in a
 * statically allocated device array of 256 MiB per GPU (held by each GPU the
 * library runs on until the process ends) instead of the context's scratch.
 * It calls no allocating routine: the context builds its per-level constants
 * and looks up the array's device address when it is created.  Rotations run
 * in groups of as many as fit (two at N = 2^16 with 24 limbs and 8 special
 * primes, 32 on small rings).  FESC_ERR_ARG, before any launch, if one
 * rotation at `level` needs more than the array: level + dnum_l (level +
 * alpha) + 2 (level + alpha) + 2 level rows of N words, dnum_l =
 * ceil(level / alpha).  All calls on one GPU share the array, so calls that
 * overlap on one GPU (two streams, threads or contexts) race. */
int fesc_rotate_batch_noalloc(fesc_ctx* ctx, uint32_t count, const uint64_t* const* ins,
                              const int32_t* steps, uint64_t* const* outs, uint32_t level,
                              void* stream);

/* Switching-key generation on the device from caller-drawn randomness:
 * s: int8[N] ternary secret coefficients; a: uint64[dnum][L+alpha][N] uniform
 * residues (evaluation form); e: int64[dnum][N] error coefficients.  For
 * digit j and extended prime i:
 *   b_j = -a_j s + e_j + [P]_{q_i} s'   (q_i in digit j)
 *   b_j = -a_j s + e_j                  (otherwise)
 * with s' = s^2 (galois_elt == 0, relinearisation) or sigma_g(s).  The key is
 * kept in context memory (allocated on first use, replaced on repeat). */
int fesc_keygen(fesc_ctx* ctx, uint32_t galois_elt, const int8_t* s, const uint64_t* a,
                const int64_t* e, void* stream);

/* The same key with its uniform half drawn from a seed instead of passed in:
 * seed: uint64[2] in HOST memory.  a_j[i][k] comes from the counter-based
 * generator Philox4x64-10 (Salmon et al., SC 2011) keyed by the seed: the
 * block of counter (k, i, c, galois_elt), i the extended prime's index in the
 * full chain (q_i -> i, p_m -> L + m), gives words w0..w3 for digits 3c ..
 * 3c + 2; digit 3c + t takes w_t masked to the bit length of the prime when
 * that is below the prime, else the spare word w3 (masked) if no earlier
 * digit of the block took it and it is below the prime, else w_t mod the
 * prime.  The context stores only the seed and the b half (half the bytes);
 * key switching regenerates a where it reads the key, so rotations,
 * conjugations and relinearisation give the residues they give with the full
 * key.  fesc_key_store writes the full layout. */
int fesc_keygen_seeded(fesc_ctx* ctx, uint32_t galois_elt, const int8_t* s,
                       const uint64_t* seed, const int64_t* e, void* stream);

/* Copy a key (layout above, device memory) into / out of the context.
 * galois_elt: 0 (relinearisation) or odd in (1, 2N), else FESC_ERR_ARG;
 * store: FESC_ERR_NO_KEY if the context holds no key of that element; a
 * seed-expanded key is written in the full layout (a regenerated). */
int fesc_key_load(fesc_ctx* ctx, uint32_t galois_elt, const uint64_t* key, void* stream);
int fesc_key_store(fesc_ctx* ctx, uint32_t galois_elt, uint64_t* key, void* stream);

/* Upload a switching key generated elsewhere (by the client, who holds the
 * secret; Sec. 2.1: the server only receives evaluation keys) from HOST
 * memory.  host_key: uint64[ceil(key_level/alpha)][key_level+alpha][2][N],
 * the layout above over the chain prefix q_0..q_{key_level-1} and the special
 * primes (digit j covers q_{j*alpha}.., as everywhere).  1 <= key_level <= L
 * (else FESC_ERR_LEVEL); a key with key_level < L serves key switches at
 * levels <= key_level only, and any operation that would use it above that
 * level fails with FESC_ERR_LEVEL.  galois_elt as for fesc_key_load.  The
 * host buffer is owned by the caller and read before the call returns (the
 * call synchronises `stream`); the context keeps its own copy, replacing
 * any earlier key of that element. */
int fesc_key_upload(fesc_ctx* ctx, uint32_t galois_elt, const uint64_t* host_key,
                    uint32_t key_level, void* stream);

/* Secret-key encryption from caller-drawn randomness: c1 = a,
 * c0 = -a s + m + e.  s: int8[N]; m: int64[N] plaintext coefficients;
 * a: uint64[l][N] uniform (evaluation form); e: int64[N]. */
int fesc_encrypt_sk(fesc_ctx* ctx, const int8_t* s, const int64_t* m, const uint64_t* a,
                    const int64_t* e, uint64_t* ct, uint32_t level, void* stream);

/* Plaintext [l][N] from signed integer coefficients (reduce, transform). */
int fesc_plain_from_coeffs(fesc_ctx* ctx, const int64_t* m, uint64_t* pt, uint32_t level,
                           void* stream);

/* ------------------------------------------------------------------------
 * Plaintext-matrix x ciphertext projection (paper Appendix "Projection
 * Kernel Breakdown": segment view idx(r, s) = s * unit + r, whole-segment
 * shift Phi^d = rotation by d * unit slots, BSGS with n1 * n2 = C):
 *     c~_{b,p} = sum_{u < n_in} sum_{q < n1} Phi^q(x~_u) * D~[b][p][u][q]
 *     y_b      = sum_{p < n2} Phi^(p n1)(c~_{b,p})
 *     y_b     += conj(y_b)            if real_extract
 *     y_b      = rescale(y_b)         if rescale  (output at level - 1)
 * Baby steps are hoisted (one ModUp per input); giant steps and the
 * conjugation are single key switches.  With real_extract the caller folds
 * the 1/2 of the real-part extraction into the diagonals.
 * complex_pair = 1 (n_out even, real_extract = 0): two real output blocks
 * leave as one ciphertext, output P = y_{2P} + conj(y_{2P+1}) (then rescaled),
 * n_out / 2 outputs in all: 3 key switches per pair for n2 = 2 instead of the
 * 4 of two extracted outputs, and half the rescales.  With paired inputs
 * x~ = x0 + i x1 the diagonal sets 2P and 2P+1 hold alpha and conj(beta) of
 * S + i S' = alpha x~ + beta conj(x~) (fesc_bsgs_diagonal_slots), so that
 * the real and imaginary parts of output P are blocks 2P and 2P+1. 
 * ------------------------------------------------------------------------ */
typedef struct fesc_matvec_desc {
  uint32_t level;        /* level of the inputs (and diagonals) */
  uint32_t n_in;         /* input ciphertexts x~_u */
  uint32_t n_out;        /* diagonal sets y_b (outputs unless complex_pair) */
  uint32_t n1, n2;       /* baby and giant steps */
  uint32_t unit;         /* slots per segment */
  uint32_t real_extract; /* 0 or 1 */
  uint32_t rescale;      /* 0 or 1 */
  uint32_t complex_pair; /* 0 or 1: outputs in pairs, see below */
  uint32_t lazy_moddown; /* 0 or 1: double hoisting, see below */
} fesc_matvec_desc;

/* lazy_moddown = 1 (double hoisting; Bossuat, Mouchet, Troncoso-Pastoriza and
 * Hubaux, Eurocrypt 2021): the baby steps stay in the extended basis Q u P
 * (P Phi^q(c0) + acc, acc' with no ModDown), the pt-MAC runs over the
 * level + alpha rows q_0 .. q_{level-1}, p_0 .. p_{alpha-1} with diagonals
 * encoded there (fesc_encode_plain_ext: every diagonal and bank slot then has
 * level + alpha rows), and each c~_{b,p} takes one ModDown before its giant
 * step.  The results differ from lazy_moddown = 0 only in where ModDown
 * rounds; the plan holds (n_in n1 + n_out n2) extended ciphertexts more. */
typedef struct fesc_matvec_plan fesc_matvec_plan;

/* Plan: `diags` is a host array of n_out*n2*n_in*n1 device pointers to
 * plaintexts ([level][N], evaluation form), indexed [b][p][u][q]; they must
 * stay valid for the plan's lifetime.  Allocates the plan's workspace (the
 * baby-step and partial-sum ciphertexts).  FESC_ERR_NO_KEY if a rotation or
 * conjugation key the schedule needs is not loaded. */
int fesc_matvec_plan_create(fesc_ctx* ctx, const fesc_matvec_desc* desc,
                            const uint64_t* const* diags, fesc_matvec_plan** plan);
void fesc_matvec_plan_destroy(fesc_matvec_plan* plan);

/* in: host array of n_in device ciphertexts [level][2][N]; out: host array of
 * n_out (n_out / 2 with complex_pair) device ciphertexts ([level-1][2][N] with
 * rescale, else [level][2][N]).  Outputs must not alias inputs. */
int fesc_ptct_matvec(fesc_ctx* ctx, fesc_matvec_plan* plan, const uint64_t* const* in,
                     uint64_t* const* out, void* stream);

/* Diagonal bank: the same diagonals in one device buffer laid out for
 * streaming, each residue in 50 bits (every prime is below 2^50).  With
 * O = n_out*n2 outputs (b, p) and T = n_in*n1 terms (u, q), the buffer holds
 * 32-bit words [limb][N/256][T][O + ceil(O/2) + ceil(O/16)][256]: per
 * 256-coefficient tile and term, O planes of the residues' low 32 bits, then
 * ceil(O/2) planes holding bits 32..47 of outputs 2j (low half) and 2j+1
 * (high half), then ceil(O/16) planes holding bits 48..49 of output o at bit
 * 2 (o mod 16).  One workgroup of the plaintext MAC then reads contiguous
 * runs, 6.25 bytes per residue instead of 8 when O is a multiple of 16 (the
 * shared planes are partly empty otherwise: 8 bytes at O = 2, 12 at O = 1).
 * fesc_matvec_bank_words gives its size in uint64 words (level*N*T*(O +
 * ceil(O/2) + ceil(O/16))/2; level+alpha rows with lazy_moddown);
 * fesc_matvec_bank_pack writes plaintext `pt` ([level][N], or
 * [level+alpha][N]; canonical residues, as every encoder here produces) into
 * slot `index` = ((b*n2 + p)*n_in + u)*n1 + q of the bank.  It touches only
 * that diagonal's bits (shared words are updated with atomic AND / OR), so
 * the bank needs no clearing and packs of different slots may run in any
 * order or on different streams.  A plan created from a bank reads it
 * instead of a pointer table (results are identical).  The bank must stay
 * valid for the plan's lifetime. */
int fesc_matvec_bank_words(const fesc_ctx* ctx, const fesc_matvec_desc* desc, size_t* words);
int fesc_matvec_bank_pack(fesc_ctx* ctx, const fesc_matvec_desc* desc, uint64_t* bank,
                          uint32_t index, const uint64_t* pt, void* stream);
/* The same for `count` (at most 65535) consecutive slots first ..
 * first + count - 1 in one launch: slot first + j from plaintext
 * pts + j * pt_stride (uint64 words, at least the plaintext's rows * N when
 * count > 1).  count = 0 does nothing; a slot range past the bank's
 * n_out*n2*n_in*n1 slots is FESC_ERR_ARG before any launch. */
int fesc_matvec_bank_pack_many(fesc_ctx* ctx, const fesc_matvec_desc* desc, uint64_t* bank,
                               uint32_t first, uint32_t count, const uint64_t* pts,
                               size_t pt_stride, void* stream);
int fesc_matvec_plan_create_bank(fesc_ctx* ctx, const fesc_matvec_desc* desc,
                                 const uint64_t* bank, fesc_matvec_plan** plan);

/* Slot vectors of the projection's diagonals on the device (offline
 * preparation; the appendix encodes all plaintext diagonals offline), for
 * fesc_encode_plain and fesc_matvec_bank_pack.  W: device fp64 weight matrix,
 * row-major [d_in][d_out], d_in = n_in * C (2 n_in * C with real_extract or
 * complex_pair: paired inputs), d_out = n_out * C, with C = segs segments of
 * `unit` slots (segs must divide (N/2) / unit; slot j lies in segment
 * (j / unit) mod segs, so a shorter vector repeats); entries outside W read
 * as 0.  z: device [count][N/2] complex slots
 * (interleaved re, im) of the diagonals first .. first + count - 1 in bank
 * order ((b n2 + p) n_in + u) n1 + q.  With t = p n1 + q and
 * diag_t^(g,b)[idx(r, s)] = W[g C + (s + t) mod C, b C + s], each vector is
 * Phi^(-p n1) of:
 *   diag_t^(u,b)                                   (plain),
 *   (diag_t^(2u,b) - i diag_t^(2u+1,b)) / 2        (real_extract),
 *   alpha or conj(beta) of the pair (b = 2P + e):  (complex_pair)
 *     e = 0: ((a + f) + i (d - c)) / 2,  e = 1: ((a - f) - i (d + c)) / 2,
 *     a = diag^(2u,2P), c = diag^(2u+1,2P), d = diag^(2u,2P+1), f = diag^(2u+1,2P+1).
 * FESC_ERR_ARG for a range past the last diagonal, or unit * segs not
 * dividing N/2. */
int fesc_bsgs_diagonal_slots(fesc_ctx* ctx, const fesc_matvec_desc* desc, const double* W,
                             uint32_t d_in, uint32_t d_out, uint32_t segs, uint32_t first,
                             uint32_t count, double* z, void* stream);

/* Phase durations of the plan's last completed run, from HIP events recorded
 * on its stream: baby steps, pt-MAC (one kernel), giant steps + extraction +
 * rescale.  The caller synchronises first; FESC_ERR_HIP if not complete. */
int fesc_matvec_phase_ms(const fesc_matvec_plan* plan, float* baby_ms, float* ptmac_ms,
                         float* tail_ms);

/* ------------------------------------------------------------------------
 * Scan-contract slice of a block of tokens (paper Eq. "hescan-contract-output"
 * and Appendix "Complex-Packed Reduction Accounting").  For each token u and
 * state chunk k (inputs at `level`: state h, broadcast decay a, broadcast
 * output factor C, each [level][2][N], indexed u*chunks + k):
 *     t = RS(relin(RS(relin(a * h)) * C))     (level >= 3; out at level - 2)
 * or, with decay = NULL (the contraction of states the scan already formed,
 * Eq. "hescan-contract-output"),
 *     t = RS(relin(h * C))                    (level >= 2; out at level - 1)
 * each RS(relin(.)) one merged division by P q_{l-1} as in
 * fesc_mul_relin_rescale.
 * Chunks are paired (2l, 2l+1) as chi = t_2l + i t_2l+1 (i = X^(N/2)),
 * reduced over a contiguous d_state axis by rotate-and-add with steps
 * d_state/2, ..., 1 (slot e*d_state then holds the sum over the axis), and
 * split by one conjugation:
 *     out[2l]   = Xi + conj(Xi)        = 2 Sigma(t_2l)
 *     out[2l+1] = -i (Xi - conj(Xi))   = 2 Sigma(t_2l+1)
 * (the factor 2 belongs to the caller's scale bookkeeping).  An odd last
 * chunk is reduced alone.  The products of all (token, chunk) pairs run in
 * groups of 32, every rotation step as one batch over all tokens; each
 * token's result equals that of a one-token call.  h, decay, cfac, out: host
 * arrays of tokens*chunks device pointers; outputs are [lo][2][N] (lo the
 * output level above),
 * distinct, not aliasing inputs (they also serve as the reduction's
 * workspace).  At most 32 tokens when chunks is odd.  Needs the
 * relinearisation key, the rotation keys of the reduction steps and
 * (chunks >= 2) the conjugation key; FESC_ERR_NO_KEY otherwise. */
int fesc_scan_contract(fesc_ctx* ctx, const uint64_t* const* h, const uint64_t* const* decay,
                       const uint64_t* const* cfac, uint32_t chunks, uint32_t tokens,
                       uint32_t d_state, uint64_t* const* out, uint32_t level, void* stream);

/* ------------------------------------------------------------------------
 * Encrypted affine prefix scan (Sec. "Parallel Prefix Scans", paragraph
 * "Affine Prefix Composition", Eq. "compact_affine_compose"; Brent-Kung
 * network of Appendix "Prefix-Network Selection").  `chunks` independent
 * sequences (state chunks) of L token maps F_k(z) = a_k z + s_k: a[c*L + k]
 * and s[c*L + k] are device pointers to [level][2][N] ciphertexts, all at
 * `level` (a: decay broadcast into the chunk's packing; s: additive update).
 * When R follows E the composition is
 *     (RS(relin(a_R a_E)),  RS(relin(a_R s_E)) + s_R)
 * taken at the lower level of the two operands (a higher operand enters
 * through its leading limbs; s_R through its first level - 1 limbs).  The
 * Brent-Kung network (up-sweep over the 2^s-aligned positions; down-sweep
 * from every multiple k of 2^s to k + 2^(s-1); positions past L not computed)
 * runs in place: on return buffer (c, k) holds in its leading *out_level limbs
 * ([out_level][2][N]) the inclusive prefix T_1 o ... o T_k, a = product of the
 * decays and s = the state h_k (the prefix applied to the zero state).
 * out_level = level - D, D the largest composition depth (2m - 2 for
 * L = 2^m >= 4, 1 for L = 2, 0 for L = 1).  Two relinearisations per
 * composition: 2 (2(L - 1) - log2 L) key switches per chunk for L a power of
 * two.  flags FESC_SCAN_STATES_ONLY: only the states are wanted; decay
 * products no later product reads are skipped (about a quarter of all
 * products; the a buffers then hold no defined result).  All 2 L chunks
 * buffers must be distinct.  FESC_ERR_NO_KEY without the relinearisation key;
 * FESC_ERR_LEVEL if a composition would fall below level 2. */
#define FESC_SCAN_STATES_ONLY 1u
int fesc_affine_scan(fesc_ctx* ctx, uint64_t* const* a, uint64_t* const* s, uint32_t L,
                     uint32_t chunks, uint32_t level, uint32_t flags, uint32_t* out_level,
                     void* stream);

/* Output level and number of relinearised products (= key switches) per
 * chunk of fesc_affine_scan with these arguments; no device work. */
int fesc_affine_scan_info(fesc_ctx* ctx, uint32_t L, uint32_t level, uint32_t flags,
                          uint32_t* out_level, uint64_t* key_switches);

/* Host only (no context, no device): the network fesc_affine_scan runs for L
 * positions, one node per composition in execution order, 4 words each:
 * (stage, dst, src, decay) -- position dst takes T_src o T_dst (0-based
 * positions), and decay = 1 if the node forms its decay product (always, unless
 * flags has FESC_SCAN_STATES_ONLY and no later product reads it).  Nodes of
 * one stage are independent.  With nodes = NULL only *count is set; otherwise
 * cap nodes are available and FESC_ERR_ARG is returned (after *count is set)
 * if the network has more.  1 <= L <= 2^20. */
int fesc_affine_scan_network(uint32_t L, uint32_t flags, uint32_t* nodes, size_t cap,
                             size_t* count);

/* The same scan by the two-pass resident block schedule (Sec. "Resident
 * Block Schedule", Eq. "resident-block-schedule"), returning states only.
 * Blocks of `block` tokens (the last may be partial).  Pass 1 keeps the
 * summary (last local prefix) of every block but the last; the same network
 * over the summaries gives the carries G_j = S_{j-1} o ... o S_0; pass 2
 * replays each block's local prefixes P_{j,t} and writes the state of
 * P_{j,t} o G_j, i.e. a_P s_G + s_P (one relinearised product; block 0: s_P).
 * a, s: as for fesc_affine_scan, not modified.  h[c*L + k]: distinct output
 * buffers of [out_level][2][N], not aliasing inputs.  `workspace`: device
 * memory of at least the size fesc_affine_scan_resident_info reports (per
 * chunk one block of tuples and the summaries, at `level`); the info call also
 * gives out_level and the relinearised products per chunk (no device work).
 * Block 0 and the carries are used through their states only, so dead decay
 * products are skipped there as in FESC_SCAN_STATES_ONLY.  Errors as for
 * fesc_affine_scan, and FESC_ERR_ARG for a short workspace. */
int fesc_affine_scan_resident_info(fesc_ctx* ctx, uint32_t L, uint32_t chunks, uint32_t block,
                                   uint32_t level, uint32_t* out_level, size_t* workspace_bytes,
                                   uint64_t* key_switches);
int fesc_affine_scan_resident(fesc_ctx* ctx, const uint64_t* const* a, const uint64_t* const* s,
                              uint32_t L, uint32_t chunks, uint32_t block, uint64_t* const* h,
                              uint32_t level, void* workspace, size_t workspace_bytes,
                              void* stream);

/* Host only (no context, no device): the products fesc_affine_scan issues
 * for `chunks` sequences of L tokens (flags as there), in the format of
 * fesc_affine_scan_resident_program below; a[c L + k] and s[c L + k] are
 * 2^24 + c L + k and 2 * 2^24 + c L + k, and the scan runs in place over
 * them.  chunks * L <= 2^20. */
int fesc_affine_scan_program(uint32_t L, uint32_t chunks, uint32_t flags, uint64_t* words,
                             size_t cap, size_t* count);

/* Host only (no context, no device): the products fesc_affine_scan_resident
 * issues for one chunk of L tokens in blocks of `block`, recorded in issue
 * order with placeholder addresses: 5 words per entry,
 *     (group, x, y, add, out)   out = x * y (+ add; add = 0: none)
 *     (group, src, 0, 0, dst)   a copy
 * where the inputs a[k] and s[k] are 2^24 + k and 2 * 2^24 + k, the outputs
 * h[k] are 3 * 2^24 + k, and workspace slots lie from 4 * 2^24 on.  Entries
 * of one group are one batched call: all their operands are read before any
 * of their outputs is written.  With words = NULL only *count is set;
 * otherwise cap entries are available and FESC_ERR_ARG is returned (after
 * *count is set) if the program has more.  1 <= block <= L <= 2^16. */
int fesc_affine_scan_resident_program(uint32_t L, uint32_t block, uint64_t* words, size_t cap,
                                      size_t* count);

/* ------------------------------------------------------------------------
 * Public slot maps and the HEScan broadcasts (Sec. "CKKS Primitives and Slot
 * Maps": br expands a compact factor into the state packing, br^(kappa)
 * restricts it to chunk kappa; exact maps in Appendix "HEScan Kernel Packing
 * and Correctness", paragraph "Exact State and Slot Maps").
 *
 * A slot map (slots j mod n_slots = N/2, rho(v; r)_j = v_{j+r}) over terms
 * t = p n1 + q < terms (q < n1 baby index, p < n2 = ceil(terms / n1)):
 *     y[j]   = v[j + offset + q stride + p giant_stride]   for j in run(p, q),
 *              run(p, q) = [dst0 + q dst_stride + p dst_giant, ... + width)
 *     y[j]   = 0                                           elsewhere
 *     out[j] = sum_{u < rep_count} y[j - u rep_stride]
 * evaluated homomorphically as
 *     1. rho(v; offset)                           (one key switch; none if 0)
 *     2. sum_t M_t (.) rho(.; q stride + p giant_stride) (M_t = 1 on the run):
 *        the baby steps rho(.; q stride) share one ModUp, the giant steps are
 *        rho(.; p giant_stride); then one rescale
 *     3. log2(rep_count) doublings out += rho(out; -2^s rep_stride).
 * Key switches: [offset != 0] + (n1 - 1) + (n2 - 1) + log2(rep_count); one
 * level (input `level` >= 2, output level - 1).  The runs must be disjoint
 * in the order of t: width <= dst_stride (n1 > 1) and (n1 - 1) dst_stride +
 * width <= dst_giant (n2 > 1), the last run inside the slots.  The error of
 * an output slot grows with the square root of rep_count (each doubling adds
 * the key-switching noise of every slot of the copies it sums). */
typedef struct fesc_slot_map_desc {
  uint32_t level;        /* input level */
  int32_t offset;        /* rotation applied first */
  int32_t stride;        /* rotation per baby step */
  int32_t giant_stride;  /* rotation per giant step */
  uint32_t terms;        /* >= 1 */
  uint32_t n1;           /* baby steps, >= 1 */
  uint32_t dst0, dst_stride, dst_giant, width;  /* runs */
  int32_t rep_stride;
  uint32_t rep_count;    /* power of two, 1 = no replication */
} fesc_slot_map_desc;

/* Shape of the HEScan packing: H heads of width P (E = H P channels
 * e = h P + p), G groups of B and C (heads in G contiguous groups of H / G,
 * group g(h) = floor(h G / H)), state size d_s per channel, c_state channels
 * per chunk (chunk kappa holds (e, i) at slot (e - kappa c_state) d_s + i). */
typedef struct fesc_br_shape {
  uint32_t H, P, G, d_s, c_state;
} fesc_br_shape;

#define FESC_BR_A 0  /* decay a_k, compact at slot k H + h */
#define FESC_BR_X 1  /* input x_k, compact at slot k E + e */
#define FESC_BR_B 2  /* B_k, compact at slot k G d_s + g d_s + i */
#define FESC_BR_C 3  /* C_k, same packing as B_k */

/* Host only: the slot map realising br^(kappa) of token k's factor `kind`
 * from its compact packing, for ring degree N = 2^log_n and input level
 * `level` (giant steps continue the baby steps, giant_stride = n1 stride and
 * dst_giant = n1 dst_stride, unless stated):
 *   x:  offset k E + kappa c, stride 1 - d_s, terms c, runs {t d_s},
 *       replication d_s x 1                   (d_s a power of two);
 *   a:  offset k H + kappa c / P; R = min(P d_s, 512); head p of the chunk
 *       at P d_s / R positions: n1 = P d_s / R, stride -R, dst_stride R,
 *       giant_stride 1 - P d_s, dst_giant P d_s, terms (c / P) n1, width 1;
 *       replication R x 1                      (P | c, P d_s a power of 2);
 *   B, C with chunk kappa inside group g: offset k G d_s + g d_s, one run
 *       [0, d_s), replication c x d_s         (c a power of two);
 *   B, C with chunk kappa over whole groups g0, g0 + 1, ... (Eg = H P / G
 *       channels each): offset k G d_s + g0 d_s, stride d_s - Eg d_s, terms
 *       c / Eg, runs [t Eg d_s, t Eg d_s + d_s), replication Eg x d_s.
 * n1 (x, B, C) = the smallest power of two whose square reaches the term
 * count.  FESC_ERR_ARG for shapes outside these cases, or a token whose
 * compact factor or a chunk that does not fit N/2 slots. */
int fesc_br_desc(uint32_t log_n, const fesc_br_shape* shape, uint32_t kind, uint32_t k,
                 uint32_t kappa, uint32_t level, fesc_slot_map_desc* out);

/* Slot vectors of the masks, rotated for the giant steps: mask m = p n1 + q
 * (m < n1 * n2) is 1 at slot j where j - p giant_stride (mod n_slots) lies
 * in run(p, q), and 0 elsewhere (all zero for m >= terms).  z: device
 * [count][N/2] complex (interleaved re, im) for masks first .. first +
 * count - 1, to be encoded at the scale of q_{level-1} (fesc_encode_plain). */
int fesc_slot_map_mask_slots(fesc_ctx* ctx, const fesc_slot_map_desc* desc, uint32_t first,
                             uint32_t count, double* z, void* stream);

typedef struct fesc_slot_map_plan fesc_slot_map_plan;

/* masks: host array of `terms` device plaintexts [level][N] (the encoded
 * mask slot vectors m < terms); they must stay valid for the plan's lifetime.
 * Allocates the plan's workspace.  FESC_ERR_NO_KEY if a key of the schedule
 * is missing; FESC_ERR_ARG for runs that overlap or leave the slots, or a
 * replication count that is not a power of two. */
int fesc_slot_map_plan_create(fesc_ctx* ctx, const fesc_slot_map_desc* desc,
                              const uint64_t* const* masks, fesc_slot_map_plan** plan);
void fesc_slot_map_plan_destroy(fesc_slot_map_plan* plan);

/* in: device ciphertext [level][2][N]; out: device [level-1][2][N] (may
 * alias in: the input is read before the output is written). */
int fesc_slot_map(fesc_ctx* ctx, fesc_slot_map_plan* plan, const uint64_t* in, uint64_t* out,
                  void* stream);

/* The plan's map over `count` (1 .. 65535) inputs at once, item i with its
 * own first rotation offsets[i] in place of the plan's offset (the rest of
 * the map is the plan's; for br^(kappa) the tokens of one kind and chunk
 * differ only there, Appendix "HEScan Kernel Packing and Correctness").
 * ins[i]: device ciphertext [level][2][N]; outs[i]: device [level-1][2][N]
 * (may alias ins[i]).  Groups of up to 16 items share their key-switch launches:
 * the offset rotations one launch, every doubling one launch with all jobs
 * under one key.  Allocates the plan's batch workspace on first use.
 * FESC_ERR_NO_KEY (before any launch) if an offset's rotation key is
 * missing; the plan must not be used from two streams at once. */
int fesc_slot_map_batch(fesc_ctx* ctx, fesc_slot_map_plan* plan, uint32_t count,
                        const uint64_t* const* ins, const int32_t* offsets,
                        uint64_t* const* outs, void* stream);

/* ------------------------------------------------------------------------
 * Small kernels on the same primitives.
 *
 * HEConv (Sec. "Causal Depthwise Convolution"): causal depthwise convolution
 * over token slots, eta = RS(sum_r M_r (.) rho(q; delta_r)) + b.  q: device
 * ciphertext [level][2][N] (level >= 2); taps (1 .. 16) rotation offsets
 * deltas (host array; rho(v; d)_j = v_{j+d}, so -r brings token k - r to
 * slot k; FESC_CONJ not allowed) and masks (host array of device plaintexts
 * [level][N], tap weights fused with the causal boundary mask, encoded at the
 * scale of q_{level-1}); bias: device plaintext at the output scale with at
 * least level limbs, or NULL.  The rotations share one ModUp.  out: device
 * ciphertext [level-1][2][N], not aliasing q.  FESC_ERR_NO_KEY without a
 * tap's rotation key. */
int fesc_heconv(fesc_ctx* ctx, const uint64_t* q, uint32_t taps, const int32_t* deltas,
                const uint64_t* const* masks, const uint64_t* bias, uint64_t* out,
                uint32_t level, void* stream);

/* Fused post-SSM path (Appendix "Fused Post-SSM Path"), all inputs at `level`
 * (>= 3): y = RS(D (.) x_skip) + m (level - 1), out = y (.) g relinearised
 * and divided by P q_{level-2} in one step (level - 2).  D: device plaintext
 * [level][N] at the scale of q_{level-1}; g at the scale of q_{level-2}; m,
 * x_skip, g: device ciphertexts [level][2][N]; out [level-2][2][N].  Needs the
 * relinearisation key. */
int fesc_post_ssm(fesc_ctx* ctx, const uint64_t* m, const uint64_t* x_skip,
                  const uint64_t* d_skip, const uint64_t* g, uint64_t* out, uint32_t level,
                  void* stream);

/* Plaintext addition out = (c0 + pt, c1) (pt: [level][N], evaluation form);
 * out may alias ct.  With pt a uniform polynomial r_hat this is the server's
 * mask <m> + r_hat of the CKKS-to-MPC conversion (Algorithm "Complex
 * CKKS-to-MPC conversion"); r_hat is drawn by the caller. */
int fesc_add_plain(fesc_ctx* ctx, const uint64_t* ct, const uint64_t* pt, uint64_t* out,
                   uint32_t level, void* stream);

/* Host helper, modulus trimming before conversion (Appendix "Adopted Modulus
 * Trimming"): the smallest l' in 1 .. level whose modulus Q = q[0] ... q[l'-1]
 * has log2 Q >= ell + sigma + 1 and Q / 2 > delta * bmax (exact integer
 * comparisons), or 0 if none; the trimmed ciphertext is the first l' limbs of
 * the buffer.  q: host array of the ciphertext primes. */
int fesc_c2m_level(const uint64_t* q, uint32_t level, uint32_t ell, uint32_t sigma, double delta,
                   double bmax, uint32_t* out_level);

/* Device CKKS encoding (offline plaintext preparation; slot convention and
 * rounding of fesc_encode): `count` slot vectors z ([count][N/2] complex,
 * interleaved re/im fp64, device) at scale `scale` into evaluation-form
 * plaintexts pt ([count][level][N], device): m_k = round half away from zero
 * of (scale / N) Re(zeta^-k Y_k), Y the length-N DFT of the slots placed at
 * the odd exponents 5^j (and their conjugates at -5^j), computed by a two-pass
 * fp64 FFT on the device, then reduced into q_0 .. q_{level-1} and transformed.
 * The coefficients equal fesc_encode's except within the FFTs' rounding of a
 * half-integer (+-1 there).  |scale * z| must stay below 2^62 (not checked on
 * the device).  Uses context scratch; asynchronous on `stream`. */
int fesc_encode_plain(fesc_ctx* ctx, const double* z, uint32_t count, double scale, uint64_t* pt,
                      uint32_t level, void* stream);

/* The same encoding over the extended basis of `level` (q_0 .. q_{level-1},
 * then the special primes p_0 .. p_{alpha-1}): pt ([count][level+alpha][N],
 * device), for the double-hoisted projection (fesc_matvec_desc.lazy_moddown),
 * whose plaintext MAC runs before the ModDown. */
int fesc_encode_plain_ext(fesc_ctx* ctx, const double* z, uint32_t count, double scale,
                          uint64_t* pt, uint32_t level, void* stream);

/* Decoding on the device, the inverse of fesc_encode_plain (Sec. 2.1: slot j is
 * the evaluation at zeta^(5^j mod 2N), zeta = exp(i pi / N)): evaluation-form
 * plaintexts pt[count][level][N] (device, canonical residues) -> slot vectors
 * z[count][N/2] (device, complex as interleaved re/im doubles),
 *     z_j = m(zeta^(5^j)) / scale,
 * m the plaintext's centred integer coefficients in (-Q/2, Q/2], Q the product
 * of the level's primes.  m is reconstructed exactly by a mixed-radix CRT with
 * balanced digits and evaluated in fp64 (a relative error of about level units
 * in the last place; coefficients beyond the double range give infinities),
 * then transformed by an fp64 FFT.  Decoding needs no secret key: a client
 * decodes after decrypting.  pt is left unchanged.  FESC_ERR_LEVEL for a level
 * outside 1..L, FESC_ERR_ARG for a zero or non-finite scale or a null buffer;
 * count 0 does nothing.  Uses the context's scratch. */
int fesc_decode_plain(fesc_ctx* ctx, const uint64_t* pt, uint32_t count, uint32_t level,
                      double scale, double* z, void* stream);

/* Host helper: CKKS encoding of n = N/2 complex slots (re, im host arrays;
 * im may be NULL) at scale Delta into int64 coefficients, rounded half away
 * from zero; slot j is the evaluation at exp(i pi 5^j / N).  FESC_ERR_ARG if
 * a coefficient does not fit in int64. */
int fesc_encode(uint32_t log_n, const double* re, const double* im, double scale,
                int64_t* coeffs);

/* Measurement helper, not part of the method: runs the register-resident
 * arithmetic of the library's inner loops on every compute unit of the
 * context's device with no memory traffic and stores the measured rate in
 * *rate (operations per second).  kind FESC_CALIB_CT: forward NTT
 * butterflies (radix-2 Cooley-Tukey with the transform's lazy reduction);
 * FESC_CALIB_GS: inverse NTT butterflies (Gentleman-Sande); FESC_CALIB_MAC:
 * modular multiply-accumulates as in basis conversion and the key inner
 * product (reduced after every four terms); FESC_CALIB_MODMUL_F64 and
 * FESC_CALIB_MODMUL_U64: the residue product alone in the library's fp64 form
 * (exact product split by one FMA, quotient from the precomputed w / q) and
 * in the 64-bit integer Shoup form (quotient from the high half of
 * x * floor(w 2^64 / q)), the evidence for the fp64 choice;
 * FESC_CALIB_PHILOX: Philox4x64-10 blocks, the generator of seed-expanded
 * keys (rate in blocks per second).  Each thread runs `iters` iterations
 * (1 .. 2^20) of 32 butterflies, 8 products or 2 generator blocks.
 * Synchronises `stream`; uses context scratch; FESC_ERR_ARG for a bad kind
 * or count. */
#define FESC_CALIB_CT 0
#define FESC_CALIB_GS 1
#define FESC_CALIB_MAC 2
#define FESC_CALIB_MODMUL_F64 3
#define FESC_CALIB_MODMUL_U64 4
#define FESC_CALIB_PHILOX 5
int fesc_calib_valu(fesc_ctx* ctx, int kind, uint32_t iters, double* rate, void* stream);

/* Measurement helper, not part of the method: the device's practical HBM
 * ceilings for streaming kernels.  kind FESC_CALIB_HBM_READ: every 16-byte
 * word of a `bytes` buffer read once (non-temporal loads, as the read-once
 * kernels use); FESC_CALIB_HBM_COPY: a `bytes` buffer
 * copied (read plus write).  *rate = bytes moved per second (2 * bytes per
 * copy).  Allocates and frees its buffers (bytes, and bytes or a small
 * output) and synchronises `stream`; FESC_ERR_ARG for an unknown kind or a
 * size outside 1 MiB .. 64 GiB or not a multiple of 16, FESC_ERR_OOM if the
 * buffers do not fit. */
#define FESC_CALIB_HBM_READ 0
#define FESC_CALIB_HBM_COPY 1
int fesc_calib_hbm(fesc_ctx* ctx, int kind, size_t bytes, double* rate, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FESC_H */
