// Kernel launchers of ckks.hip / keyswitch.hip and the host-side operation
// drivers of ops.cpp.
#pragma once

#include <vector>

#include "fesc_internal.hpp"

namespace fesc {

// ---------------------------------------------------------------- ckks.hip
hipError_t k_binary_launch(const Context* c, const uint64_t* a, const uint64_t* b, uint64_t* out,
                           uint32_t rows, uint32_t shift, int op, hipStream_t s);
hipError_t k_mul_plain_launch(const Context* c, const uint64_t* ct, const uint64_t* pt,
                              uint64_t* out, uint32_t level, hipStream_t s);
hipError_t k_add_plain_launch(const Context* c, const uint64_t* ct, const uint64_t* pt,
                              uint64_t* out, uint32_t level, hipStream_t s);
// HEConv taps (at most kMaxConvTaps)
constexpr uint32_t kMaxConvTaps = 16;
struct ConvTable {
  const uint64_t* rot[kMaxConvTaps];   // rotated ciphertexts
  const uint64_t* mask[kMaxConvTaps];  // plaintext masks
  uint32_t taps;
};
hipError_t k_conv_acc_launch(const Context* c, const ConvTable& tab, const uint64_t* bias,
                             uint64_t* acc, uint32_t level, hipStream_t s);
// Complex pairing of real ciphertexts, up to kPairBatch pairs per launch.
// pack (split = false): x[r] = x[r] + X^(N/2) y[r];
// split (split = true): with A = x[r], B = y[r] read first,
//   first[r] = A + B,  second[r] = X^(3N/2) (A - B),
// where {first[r], second[r]} = {x[r], y[r]} (in place, element by element).
constexpr uint32_t kPairBatch = 64;
struct PairTable {
  uint64_t* x[kPairBatch];
  uint64_t* y[kPairBatch];
  uint64_t* first[kPairBatch];
  uint64_t* second[kPairBatch];
};
hipError_t k_pair_launch(const Context* c, const PairTable& tab, uint32_t count, bool split,
                         uint32_t level, hipStream_t s);
hipError_t k_monomial_launch(const Context* c, const uint64_t* in, uint64_t* out,
                             uint32_t level, uint32_t m, hipStream_t s);
hipError_t k_galois_launch(const Context* c, const uint64_t* in, uint64_t* out, uint32_t rows,
                           uint32_t g, hipStream_t s);
hipError_t k_lift_launch(const Context* c, const int64_t* x, const int8_t* x8, uint64_t* out,
                         uint32_t rows, uint32_t prime0, uint32_t split, uint32_t prime1,
                         hipStream_t s);
// Seed of a seed-expanded switching key (seeded = 0: a full key, `a` given).
struct KeySeed {
  uint64_t s0, s1, elt;
  uint32_t dnum, seeded;
};
hipError_t k_keygen_launch(const Context* c, const uint64_t* a, const uint64_t* e_ntt,
                           const uint64_t* s, const uint64_t* s_from, uint64_t* key,
                           const double2* pmod, const KeySeed& sd, hipStream_t st);
// full layout [dnum][L+alpha][2][N] of a compact seed-expanded key
hipError_t k_key_expand_launch(const Context* c, const uint64_t* compact, uint64_t* full,
                               hipStream_t st);
hipError_t k_encrypt_launch(const Context* c, const uint64_t* a, const uint64_t* s,
                            const uint64_t* me, uint64_t* ct, uint32_t level, hipStream_t st);

// Up to kRescaleBatch ciphertexts per batched rescale launch.
constexpr uint32_t kRescaleBatch = 16;
struct RsTable {
  const uint64_t* in[kRescaleBatch];
  uint64_t* out[kRescaleBatch];
  const uint64_t* add[kRescaleBatch];  // added after the division (or null)
};


// ----------------------------------------------------------- keyswitch.hip

// Up to kMaxBatch ModUp sources and key-switch jobs per launch.  Passed by
// value as a kernel argument (under 3 KB).
constexpr uint32_t kMaxBatch = 32;

struct KsTable {
  const uint64_t* src_in[kMaxBatch];  // source s: row i at src_in[s] + i*src_stride[s]
  uint64_t src_stride[kMaxBatch];
  // source s a product (relinearisation): row i is src_in[s] row i times
  // src_y[s] row i (same stride), formed where it is read; null: plain
  const uint64_t* src_y[kMaxBatch];
  // job addend a tensor: with x = add, y = add_y (ciphertexts), the addend
  // components are (x0 y0, x0 y1 + x1 y0); needs fold; null: plain addend
  const uint64_t* add_y[kMaxBatch];
  const uint64_t* key[kMaxBatch];     // job: switching key
  const uint64_t* add[kMaxBatch];     // job: ciphertext added after sigma_g (or null)
  const uint64_t* add2[kMaxBatch];    // job: ciphertext added as is (or null)
  uint64_t* out[kMaxBatch];           // job: output ciphertext
  uint32_t job_src[kMaxBatch];        // job: its ModUp source
  uint32_t galois[kMaxBatch];         // job: Galois element on the digits (0: none)
  uint32_t add_mask[kMaxBatch];       // job: components of `add` used (bit t)
  uint32_t add_galois[kMaxBatch];     // job: permutation of `add` (0: none)
  // jobs sharing a switching key (and Galois element) are consecutive: key
  // group g holds jobs kg_first[g] .. kg_first[g] + kg_count[g] - 1
  uint32_t kg_first[kMaxBatch];
  uint32_t kg_count[kMaxBatch];
  // bit g set: key group g's key is seed-expanded (compact layout, its
  // uniform half regenerated in the inner product)
  uint32_t kg_seeded;
  // 1 when every job's addend uses the job's own Galois element (or there is
  // none): the inner product then stores acc * P^-1 + add on the level rows
  // and the combine only subtracts y * P^-1; 2: extended-basis outputs (the
  // inner product writes acc + P add into out[job], [2][level+alpha][N], and
  // no ModDown follows)
  uint32_t fold;
};

// ntt.hip: transforms of the key-switch pipeline (inverse transforms store
// centred conversion digits; conversions are fused with the first forward pass)
hipError_t launch_ntt_inv_sources(const Context* c, const KsTable& tab, uint32_t nsrc,
                                  uint64_t* cc, uint32_t level, const double2* f, hipStream_t s);
hipError_t launch_ntt_inv_rescale_last(const Context* c, const KsTable& tab, uint32_t nrows,
                                       uint64_t* v, uint32_t last, const double2* ninv,
                                       hipStream_t s);
hipError_t launch_rescale_outer(const Context* c, const uint64_t* v, uint64_t* w, uint32_t groups,
                                uint32_t last, uint32_t rows, const double2* one, hipStream_t s);
hipError_t launch_ntt_fwd_rs_combine(const Context* c, uint64_t* w, uint32_t count, uint32_t last,
                                     uint32_t rows, const RsTable& tab, const double2* qlinv,
                                     hipStream_t s);
hipError_t launch_ntt_inv_digits(const Context* c, const RowSel& rs, uint32_t batch,
                                 uint32_t limbs, const double2* f, hipStream_t s);
hipError_t launch_modup_outer(const Context* c, const LevelTables& T, const uint64_t* cc,
                              uint64_t* ext, uint32_t nsrc, uint32_t level, hipStream_t s);
hipError_t launch_moddown_outer(const Context* c, const LevelTables& T, const uint64_t* acc,
                                uint64_t* y, uint32_t njobs, uint32_t level, hipStream_t s);
hipError_t launch_ntt_fwd_inner_rows(const Context* c, const RowSel& rs, uint32_t batch,
                                     uint32_t limbs, hipStream_t s);
hipError_t launch_moddown_rescale_outer(const Context* c, const LevelTables& T,
                                        const uint64_t* acc, uint64_t* y, uint32_t njobs,
                                        uint32_t level, uint32_t rows, hipStream_t s);
hipError_t launch_ntt_fwd_ks_combine(const Context* c, uint64_t* y, uint32_t njobs,
                                     uint32_t level, uint32_t rows, uint32_t ystride,
                                     const KsTable& tab, const uint64_t* acc,
                                     const double2* pinv, const double2* qlinv, hipStream_t s);
hipError_t k_ip_launch(const Context* c, const KsTable& tab, uint32_t nkeys, const uint64_t* ext,
                       uint64_t* acc, uint32_t level, const double2* pinv, hipStream_t s);

// ------------------------------------------------------------------ ops.cpp
const LevelTables* level_tables(Context* c, uint32_t level, int* err);

// One key switch: polynomial of source `src` switched with `key` under
// Galois element `galois`, combined into `out` (see KsTable).
struct KsJob {
  uint32_t src;
  const uint64_t* key;
  uint32_t galois;
  const uint64_t* add;
  uint32_t add_mask;
  uint32_t add_galois;
  const uint64_t* add2;
  uint64_t* out;
  const uint64_t* add_y = nullptr;  // addend is the tensor (add, add_y): components 0, 1
};
struct KsSource {
  const uint64_t* in;
  size_t stride;
  const uint64_t* y = nullptr;  // source is the product in * y (row by row)
};
static_assert(sizeof(KsTable) < 3072, "key-switch table must stay a small kernel argument");

// Runs any number of key switches at one level: ModUp of every source (at
// most kMaxBatch), then inner product, ModDown and combine of the jobs in
// groups of kMaxBatch, jobs ordered by switching key so that each key is read
// once per group (key-stationary inner product).  Sources must stay
// unmodified until all jobs have read them; a job's output must not alias a
// source or addend of another job.  rescale_rows > 0: ModDown is merged with
// the rescale (one division by P q_{level-1}, every addend folded) and the
// outputs are the first rescale_rows (<= level - 1) limbs at level - 1.
// given: use this scratch (its capacity and regions) instead of the
// context's, so that nothing is allocated; null: the context's scratch.
struct Scratch;
// ext_out: the jobs' outputs stay in the extended basis (out = P sigma_g(add)
// + acc over every row, [2][level+alpha][N]; addends must use the job's own
// Galois element, plain only): double hoisting's baby steps.
int key_switch_batch(Context* c, uint32_t level, const std::vector<KsSource>& srcs,
                     const std::vector<KsJob>& jobs, hipStream_t s, uint32_t rescale_rows = 0,
                     const Scratch* given = nullptr, bool ext_out = false);
// ModDown of `count` extended-basis ciphertexts stored contiguously,
// ext[count][2][level+alpha][N], into outs[i] ([level][2][N]); the special-
// prime rows of ext are overwritten (they become the conversion's digits).
int op_moddown_many(Context* c, uint32_t count, uint64_t* ext, uint64_t* const* outs,
                    uint32_t level, hipStream_t s);

int op_rotate_many(Context* c, const uint64_t* in, uint32_t count, const int32_t* steps,
                   uint64_t* const* outs, uint32_t level, hipStream_t s);
int op_rotate_batch(Context* c, uint32_t count, const uint64_t* const* ins,
                    const int32_t* steps, uint64_t* const* outs, const uint64_t* const* add2,
                    uint32_t level, hipStream_t s, const Scratch* given = nullptr);
// noalloc.cpp: the statically allocated scratch of the device (set up by the
// context's creation) and the rotation batch that runs in it.
int static_scratch_init(Context* c);
size_t static_scratch_bytes();
size_t rotate_scratch_words(const Context* c, uint32_t level);
int op_rotate_batch_static(Context* c, uint32_t count, const uint64_t* const* ins,
                           const int32_t* steps, uint64_t* const* outs, uint32_t level,
                           hipStream_t s);
int op_rescale(Context* c, const uint64_t* in, uint64_t* out, uint32_t level, hipStream_t s);
// Switching key of `galois` from the secret s (int8 coefficients) and the
// error e ([dnum][N]); seed null: uniform half `a` given ([dnum][L+alpha][N]),
// full layout; seed (two host words): `a` regenerated from it, compact layout.
int op_keygen(Context* c, uint32_t galois, const int8_t* sk, const uint64_t* a, const int64_t* e,
              const uint64_t* seed, hipStream_t s);
// Words of a key in the full layout [dnum][L+alpha][2][N] and in the compact
// seed-expanded layout (header + [dnum][L+alpha][N]).
size_t full_key_words(const Context* c);
size_t seeded_key_words(const Context* c);
// The key buffer of `galois` with room for `words` words (the present one
// reused if large enough, else replaced); its prefix-level and seed records
// are cleared.
int key_buffer(Context* c, uint32_t galois, size_t words, uint64_t** out);
// Relinearised products out_i = a_i * b_i (batched); out_i may alias a_i or b_i.
int op_mul_relin_many(Context* c, uint32_t count, const uint64_t* const* as,
                      const uint64_t* const* bs, uint64_t* const* outs, uint32_t level,
                      hipStream_t s);
// Rescale of `count` ciphertexts (batched launches); out[i] may alias in[i].
int op_rescale_many(Context* c, uint32_t count, const uint64_t* const* ins, uint64_t* const* outs,
                    uint32_t level, hipStream_t s);
// out_i = RS(in_i) + add_i (adds null, or add_i null: no addend), only the
// first out_rows limbs (1 <= out_rows <= level - 1) written.  out_i may alias
// in_i or add_i.
int op_rescale_add_many(Context* c, uint32_t count, const uint64_t* const* ins,
                        uint64_t* const* outs, const uint64_t* const* adds, uint32_t level,
                        uint32_t out_rows, hipStream_t s);
// Products out_i = relin(x_i * y_i) / (P q_{level-1}) + add_i (ModDown merged
// with the rescale) at `level`, first out_rows limbs written.  Runs in groups
// of the scratch capacity (an even number), one key switch per group: every
// operand of a group is read before any output of the group is written, so an
// output may alias an input of a product in its own group (add_i only its own
// product's); it must not alias an input of a product in a later group.
int op_prod_rescale_many(Context* c, uint32_t count, const uint64_t* const* xs,
                         const uint64_t* const* ys, uint64_t* const* outs,
                         const uint64_t* const* adds, uint32_t level, uint32_t out_rows,
                         hipStream_t s);
// Scratch capacity (products per group of op_prod_rescale_many).
uint32_t prod_group(Context* c, int* err);
uint32_t galois_of_step(const Context* c, int32_t step);

}  // namespace fesc
