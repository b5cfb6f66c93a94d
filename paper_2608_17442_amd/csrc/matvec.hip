// Plaintext-matrix x ciphertext projection (BSGS diagonal method on the
// segment view of the slots; paper Appendix "Projection Kernel Breakdown").
//
//   c~_{b,p} = sum_u sum_q Phi^q(x~_u) * D~_{b,u,p,q}        (pt-MAC)
//   y_b      = sum_p Phi^(p n1)(c~_{b,p});  y_b += conj(y_b);  rescale
//
// Phi^delta is one rotation by delta * unit slots.  Baby steps Phi^q(x~_u)
// share one ModUp per input (hoisted); giant steps and the conjugation are
// ordinary key switches.  Double hoisting (lazy_moddown; Bossuat et al.,
// Eurocrypt 2021) also leaves the baby steps in the extended basis Q u P
// (P Phi^q(c0) + acc, no ModDown), runs the pt-MAC there with diagonals
// encoded over Q u P, and takes one ModDown per c~_{b,p}.
//
// The pt-MAC streams every plaintext diagonal once.  A thread owns one
// coefficient of one limb and accumulates G outputs (b, p) at a time, so each
// baby-step value it loads is reused G times; the diagonals are read with
// coalesced loads and nothing else is written until the final sums.  Every
// prime is below 2^50, so a diagonal bank stores each residue in 50 bits
// (6.25 bytes instead of 8) as three word planes: the low 32 bits, bits
// 32..47 (two outputs per word) and bits 48..49 (16 outputs per word).
#include <string>
#include <vector>

#include "fesc_internal.hpp"
#include "ops.hpp"

struct fesc_matvec_plan {
  fesc_matvec_desc d;
  std::vector<const uint64_t*> diag;  // host copy of the table [n_out][n2][n_in][n1]
  const uint64_t** d_diag = nullptr;  // device copy
  uint64_t* work = nullptr;           // baby [n_in][n1], c~ [n_out][n2], extraction [n_out] cts
  // double hoisting: baby steps and c~ over the extended basis,
  // [n_in n1 + n_out n2][2][level+alpha][N]
  uint64_t* ext_work = nullptr;
  const uint64_t** d_baby = nullptr;  // device table of baby pointers (pt-MAC inputs)
  uint64_t** d_ct = nullptr;          // device table of c~ pointers (pt-MAC outputs)
  size_t ct_words = 0;
  const uint32_t* bank = nullptr;     // diagonal bank (instead of the table), or null
  int64_t giant = 0;                  // rotation per giant step (n1 unit unless given)
  hipEvent_t ev[4] = {};               // phase marks of the last run
  // several independent vectors at once (ptct_matvec_many): per vector baby
  // [n1] and c~ [n2] cts, with device tables of their pointers; mcap vectors
  uint64_t* mwork = nullptr;
  const uint64_t** d_mbaby = nullptr;
  uint64_t** d_mct = nullptr;
  uint32_t mcap = 0;
};

namespace fesc {

int op_rotate_many(Context* c, const uint64_t* in, uint32_t count, const int32_t* steps,
                   uint64_t* const* outs, uint32_t level, hipStream_t s);
int op_rescale(Context* c, const uint64_t* in, uint64_t* out, uint32_t level, hipStream_t s);
int op_rescale_many(Context* c, uint32_t count, const uint64_t* const* ins, uint64_t* const* outs,
                    uint32_t level, hipStream_t s);
uint32_t galois_of_step(const Context* c, int32_t step);

namespace {

constexpr int kThreads = 256;  // also the coefficient tile of the diagonal bank
constexpr int kGroup = 16;     // outputs accumulated per thread
static_assert(kGroup % 16 == 0, "an output group covers whole top-bit words");

// Diagonal bank.  For each (limb i, tile of kThreads coefficients, term t) a
// record of bank_record_words(n_outputs) 32-bit words per coefficient, laid
// out as planes of kThreads words (coefficient-minor, so every plane load is
// coalesced):
//   plane o                          bits 0..31 of output o's residue
//   plane n_outputs + o/2            bits 32..47 of outputs 2j, 2j+1 (low, high half)
//   plane n_outputs + H + o/16       bits 48..49 of output o at bit 2 (o mod 16)
// with H = ceil(n_outputs / 2).  Records are ordered [limb][tile][term]: a
// workgroup reads its G outputs' planes of a term as three contiguous runs, and
// the output groups of one tile (kept on one XCD, adjacent in time) sweep one
// contiguous terms-long region together.
__host__ __device__ __forceinline__ uint32_t bank_hi_planes(uint32_t n_outputs) {
  return (n_outputs + 1) / 2;
}
__host__ __device__ __forceinline__ uint32_t bank_record_words(uint32_t n_outputs) {
  return n_outputs + bank_hi_planes(n_outputs) + (n_outputs + 15) / 16;
}
// first word of record (i, tile, t)
__host__ __device__ __forceinline__ size_t bank_record(uint32_t i, uint32_t tile, uint32_t t,
                                                       uint32_t n, uint32_t n_outputs,
                                                       uint32_t terms) {
  const size_t tiles = n / kThreads;
  return (((size_t)i * tiles + tile) * terms + t) * bank_record_words(n_outputs) * kThreads;
}

// Residue from its three bank fields: an exact fp64 integer below 2^50.
__device__ __forceinline__ double bank_value(uint32_t lo, uint32_t hi_word, uint32_t hi_shift,
                                             uint32_t top_word, uint32_t top_shift) {
  const uint32_t hi = ((hi_word >> hi_shift) & 0xFFFFu) | (((top_word >> top_shift) & 3u) << 16);
  return __hiloint2double((int)(hi | 0x43300000u), (int)lo) - kTwo52;
}

// BANK: diagonals from the diagonal bank; otherwise from the table of plaintexts.
// Ciphertext rows: component c of limb i at i * row_stride + c * comp_stride
// ([limbs][2][N]: 2N and N; extended basis [2][limbs][N]: N and limbs N);
// limb i uses prime i below `split`, prime1 + (i - split) from there.
struct PtLayout {
  uint32_t row_stride, comp_stride, split, prime1;
};

// Device memory seen through a pointer read from a table: the cast tells the
// compiler the address is global, so it emits global (not flat) loads and
// stores, whose completions it can count in order; flat loads would make it
// drain every outstanding load before the first use of each one.
typedef __attribute__((address_space(1))) const uint64_t gcu64;
typedef __attribute__((address_space(1))) uint64_t gu64;

template <int G, bool BANK>
__global__ __launch_bounds__(kThreads) void k_ptmac(const uint64_t* const* __restrict__ baby,
                                                    const uint64_t* const* __restrict__ diag,
                                                    const uint32_t* __restrict__ bank,
                                                    uint64_t* const* __restrict__ outs,
                                                    uint32_t n_outputs, uint32_t terms,
                                                    uint32_t n, uint32_t limbs,
                                                    const PrimeK* __restrict__ pk, PtLayout lay) {
  // 1-D grid over (coefficient tile, limb, output group).  Workgroups are
  // dealt to the 8 XCDs round-robin; the decode keeps all output groups of one
  // tile on the same XCD and adjacent in time, so the tile's baby-step values
  // (read once per group) come from that XCD's L2 instead of HBM.
  const uint32_t tiles = n / kThreads, n_groups = (n_outputs + G - 1) / G;
  const uint32_t total_tiles = tiles * limbs;
  uint32_t tile_lin, grp;
  if ((total_tiles & 7u) == 0) {
    const uint32_t L = blockIdx.x, xcd = L & 7u, slot = L >> 3;
    grp = slot % n_groups;
    tile_lin = (slot / n_groups) * 8u + xcd;
  } else {
    grp = blockIdx.x % n_groups;
    tile_lin = blockIdx.x / n_groups;
  }
  const uint32_t i = tile_lin / tiles, tile = tile_lin % tiles;
  const uint32_t k = tile * kThreads + threadIdx.x;
  const uint32_t o0 = grp * G;
  if (i >= limbs) return;
  const PrimeK P = pk[i < lay.split ? i : lay.prime1 + (i - lay.split)];
  const uint32_t g_end = min((uint32_t)G, n_outputs - o0);
  double a0[G], a1[G];
#pragma unroll
  for (int g = 0; g < G; ++g) a0[g] = a1[g] = 0.0;
  const size_t pi = (size_t)i * n + k, c0 = (size_t)i * lay.row_stride + k,
               c1 = c0 + lay.comp_stride;
  // Outputs past the end of a partial group re-read the group's last valid
  // diagonal (results discarded at the store), which keeps the loop body free
  // of branches so the loads of a term are issued together.
  uint32_t og[G];
#pragma unroll
  for (int g = 0; g < G; ++g) og[g] = min((uint32_t)g, g_end - 1);
  // bank: this thread's words of record (i, tile, 0); the planes of the group
  const uint32_t* bk =
      BANK ? bank + bank_record(i, tile, 0, n, n_outputs, terms) + threadIdx.x : nullptr;
  const size_t rec_stride = (size_t)bank_record_words(n_outputs) * kThreads;
  const uint32_t hi_plane = n_outputs, top_plane = n_outputs + bank_hi_planes(n_outputs);
  for (uint32_t t = 0; t < terms; ++t) {
    const gcu64* bp = (const gcu64*)baby[t];
    const double x0 = u2d(bp[c0]), x1 = u2d(bp[c1]);
    double w[G];
    if (BANK) {
      // every bank word streams past once (non-temporal loads), so that the
      // bank does not evict the baby-step values the tile's other output
      // groups re-read
      const uint32_t* rec = bk + (size_t)t * rec_stride;
      uint32_t lo[G], hw[G / 2], tw[G / 16];
#pragma unroll
      for (int g = 0; g < G; ++g)
        lo[g] = __builtin_nontemporal_load(rec + (size_t)(o0 + og[g]) * kThreads);
#pragma unroll
      for (int j = 0; j < G / 2; ++j)
        hw[j] = __builtin_nontemporal_load(rec + (size_t)(hi_plane + ((o0 + og[2 * j]) >> 1)) *
                                                     kThreads);
#pragma unroll
      for (int m = 0; m < G / 16; ++m)
        tw[m] = __builtin_nontemporal_load(rec + (size_t)(top_plane + ((o0 + og[16 * m]) >> 4)) *
                                                     kThreads);
      // o0 is a multiple of 16: output o0 + og[g] sits at half og[g] & 1 of its
      // hi word and at bit 2 (og[g] & 15) of its top word
#pragma unroll
      for (int g = 0; g < G; ++g)
        w[g] = bank_value(lo[g], hw[g / 2], 16u * (og[g] & 1u), tw[g / 16], 2u * (og[g] & 15u));
    } else {
#pragma unroll
      for (int g = 0; g < G; ++g)
        w[g] = u2d(((const gcu64*)diag[(size_t)(o0 + og[g]) * terms + t])[pi]);
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      a0[g] += mm_var(x0, w[g], P.q, P.qinv);
      a1[g] += mm_var(x1, w[g], P.q, P.qinv);
    }
    if ((t & 3) == 3) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        a0[g] = red_bal(a0[g], P.q, P.qinv);
        a1[g] = red_bal(a1[g], P.q, P.qinv);
      }
    }
  }
#pragma unroll
  for (int g = 0; g < G; ++g) {
    if ((uint32_t)g < g_end) {
      gu64* o = (gu64*)outs[o0 + g];
      o[c0] = to_res(a0[g], P.q, P.qinv);
      o[c1] = to_res(a1[g], P.q, P.qinv);
    }
  }
}

// bank fields of diagonal (o, t) <- plaintext limb i, coefficients of the tile.
// The hi and top words are shared with other outputs: each diagonal clears and
// sets only its own bits with atomic AND / OR, so packs of different diagonals
// may run in any order or concurrently.
// Diagonal `first + blockIdx.z` from plaintext pts + blockIdx.z * pt_stride.
__global__ __launch_bounds__(kThreads) void k_bank_pack(const uint64_t* __restrict__ pts,
                                                        size_t pt_stride,
                                                        uint32_t* __restrict__ bank,
                                                        uint32_t first, uint32_t n,
                                                        uint32_t n_outputs, uint32_t terms) {
  const uint32_t i = blockIdx.y, tile = blockIdx.x, index = first + blockIdx.z;
  const uint32_t o = index / terms, t = index % terms;
  const uint64_t* pt = pts + (size_t)blockIdx.z * pt_stride;
  const uint64_t v = pt[(size_t)i * n + (size_t)tile * kThreads + threadIdx.x];
  uint32_t* rec = bank + bank_record(i, tile, t, n, n_outputs, terms) + threadIdx.x;
  rec[(size_t)o * kThreads] = (uint32_t)v;
  uint32_t* hw = rec + (size_t)(n_outputs + o / 2) * kThreads;
  const uint32_t hs = 16u * (o & 1u);
  atomicAnd(hw, ~(0xFFFFu << hs));
  atomicOr(hw, (uint32_t)((v >> 32) & 0xFFFFu) << hs);
  uint32_t* tw = rec + (size_t)(n_outputs + bank_hi_planes(n_outputs) + o / 16) * kThreads;
  const uint32_t ts = 2u * (o & 15u);
  atomicAnd(tw, ~(3u << ts));
  atomicOr(tw, (uint32_t)((v >> 48) & 3u) << ts);
}

// Identity baby step over the extended basis: x[t][i] = P c_t[i] on the
// level rows (c = ct [level][2][N]), 0 on the special-prime rows.
__global__ __launch_bounds__(kThreads) void k_ext_identity(const uint64_t* __restrict__ ct,
                                                           uint64_t* __restrict__ x, uint32_t n,
                                                           uint32_t level, uint32_t E,
                                                           const double2* __restrict__ pmod,
                                                           const PrimeK* __restrict__ pk) {
  const uint32_t row = blockIdx.y, t = blockIdx.z;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  if (k >= n) return;
  uint64_t v = 0;
  if (row < level) {
    const PrimeK P = pk[row];
    const double2 f = pmod[row];
    v = to_res(mm_shoup(u2d(ct[((size_t)2 * row + t) * n + k]), f.x, f.y, P.q), P.q, P.qinv);
  }
  x[((size_t)t * E + row) * n + k] = v;
}

// Slot vectors of the diagonals first .. first + count - 1 (bank order) of a
// projection: z[k][j] for slot j, the vector Phi^(-p n1) of the diagonal's
// combination (plain / real_extract / complex_pair), from W [d_in][d_out].
// Slot j reads segment s = ((j - p n1 unit) mod n_slots) / unit mod C of the
// unshifted vector.  Grid: (n_slots / kThreads, count).
struct SlotDesc {
  uint32_t n_in, n1, n2, unit, C, n_slots, d_in, d_out, first, mode;  // mode 0/1/2
};
__device__ __forceinline__ double wdiag(const double* W, const SlotDesc& S, uint32_t g,
                                        uint32_t b, uint32_t t, uint32_t s) {
  const uint32_t row = g * S.C + (s + t) % S.C, col = b * S.C + s;
  return (row < S.d_in && col < S.d_out) ? W[(size_t)row * S.d_out + col] : 0.0;
}
__global__ __launch_bounds__(kThreads) void k_bsgs_slots(const double* __restrict__ W,
                                                         SlotDesc S, double2* __restrict__ z) {
  const uint32_t j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= S.n_slots) return;
  const uint32_t idx = S.first + blockIdx.y;
  const uint32_t q = idx % S.n1, u = (idx / S.n1) % S.n_in, p = (idx / (S.n1 * S.n_in)) % S.n2,
                 b = idx / (S.n1 * S.n_in * S.n2);
  const uint32_t t = p * S.n1 + q;
  const uint32_t shift = (uint32_t)(((uint64_t)p * S.n1 * S.unit) % S.n_slots);
  const uint32_t s = ((j + S.n_slots - shift) % S.n_slots / S.unit) % S.C;
  double re, im;
  if (S.mode == 0) {
    re = wdiag(W, S, u, b, t, s);
    im = 0.0;
  } else if (S.mode == 1) {
    re = 0.5 * wdiag(W, S, 2 * u, b, t, s);
    im = 0.5 * -wdiag(W, S, 2 * u + 1, b, t, s);
  } else {
    const uint32_t P = b / 2;
    const double a = wdiag(W, S, 2 * u, 2 * P, t, s), c = wdiag(W, S, 2 * u + 1, 2 * P, t, s);
    const double d = wdiag(W, S, 2 * u, 2 * P + 1, t, s);
    const double f = wdiag(W, S, 2 * u + 1, 2 * P + 1, t, s);
    if (b % 2 == 0) {
      re = 0.5 * (a + f);
      im = 0.5 * (d - c);
    } else {
      re = 0.5 * (a - f);
      im = -(0.5 * (d + c));
    }
  }
  z[(size_t)blockIdx.y * S.n_slots + j] = double2{re, im};
}

#define HIPCK(expr)                                   \
  do {                                                \
    hipError_t e_ = (expr);                           \
    if (e_ != hipSuccess) return hip_check(e_, #expr); \
  } while (0)

}  // namespace

int check_desc(const Context* c, const fesc_matvec_desc* d) {
  if (!d) return fail(FESC_ERR_ARG, "null descriptor");
  if (d->level < 1 || d->level > c->L) return fail(FESC_ERR_LEVEL, "matvec level out of range");
  if (d->rescale && d->level < 2) return fail(FESC_ERR_LEVEL, "rescale needs level >= 2");
  if (!d->n_in || !d->n_out || !d->n1 || !d->n2 || !d->unit)
    return fail(FESC_ERR_ARG, "matvec sizes must be positive");
  if (d->real_extract > 1 || d->rescale > 1 || d->complex_pair > 1 || d->lazy_moddown > 1)
    return fail(FESC_ERR_ARG, "matvec flags must be 0 or 1");
  if (d->complex_pair && (d->real_extract || d->n_out % 2))
    return fail(FESC_ERR_ARG, "complex_pair needs an even n_out and real_extract = 0");
  return FESC_OK;
}

static uint32_t matvec_outputs(const fesc_matvec_desc& d) {
  return d.complex_pair ? d.n_out / 2 : d.n_out;
}

// Rows of each diagonal: the level's primes, plus the special primes when the
// pt-MAC runs over the extended basis.
static uint32_t diag_rows(const Context* c, const fesc_matvec_desc& d) {
  return d.level + (d.lazy_moddown ? c->alpha : 0);
}

// Every Galois key the schedule needs must be present (checked when a plan is
// made and again before a run launches anything: a key may have been replaced
// since, and a failed replacement leaves none).
static int check_plan_keys(const Context* c, const fesc_matvec_desc& d, int64_t giant) {
  std::vector<int64_t> steps;
  for (uint32_t q = 1; q < d.n1; ++q) steps.push_back((int64_t)q * d.unit);
  for (uint32_t p = 1; p < d.n2; ++p) steps.push_back((int64_t)p * giant);
  for (int64_t st : steps) {
    const uint32_t g = galois_of_step(c, (int32_t)(st % (c->n / 2)));
    if (g != 1 && !c->keys.count(g))
      return fail(FESC_ERR_NO_KEY, "matvec needs the key of rotation " + std::to_string(st));
  }
  if ((d.real_extract || d.complex_pair) && !c->keys.count(2 * c->n - 1))
    return fail(FESC_ERR_NO_KEY, "matvec real extraction needs the conjugation key");
  return FESC_OK;
}

// giant_unit: the rotation of one giant step, INT64_MIN for n1 * unit (the
// projection); the slot maps give their own.
int matvec_plan_create(Context* c, const fesc_matvec_desc* d, const uint64_t* const* diags,
                       const uint64_t* bank, fesc_matvec_plan** out, int64_t giant_unit) {
  if (!out || (!diags && !bank)) return fail(FESC_ERR_ARG, "null argument");
  *out = nullptr;
  int rc = check_desc(c, d);
  if (rc) return rc;
  const size_t n_diag = (size_t)d->n_out * d->n2 * d->n_in * d->n1;
  if (!bank)
    for (size_t t = 0; t < n_diag; ++t)
      if (!diags[t]) return fail(FESC_ERR_ARG, "null diagonal " + std::to_string(t));
  const int64_t giant = giant_unit == INT64_MIN ? (int64_t)d->n1 * d->unit : giant_unit;
  if ((rc = check_plan_keys(c, *d, giant))) return rc;

  fesc_matvec_plan* p = new fesc_matvec_plan();
  p->d = *d;
  p->giant = giant;
  p->bank = reinterpret_cast<const uint32_t*>(bank);
  if (!bank) p->diag.assign(diags, diags + n_diag);
  p->ct_words = (size_t)2 * d->level * c->n;
  const size_t n_baby = (size_t)d->n_in * d->n1, n_ct = (size_t)d->n_out * d->n2;
  std::vector<const uint64_t*> baby(n_baby);
  std::vector<uint64_t*> cts(n_ct);
  const size_t ext_words = (size_t)2 * diag_rows(c, *d) * c->n;
  bool ok = hipMalloc(&p->work, (n_baby + n_ct + d->n_out) * p->ct_words * 8) == hipSuccess &&
            (!d->lazy_moddown ||
             hipMalloc(&p->ext_work, (n_baby + n_ct) * ext_words * 8) == hipSuccess) &&
            (bank || hipMalloc(&p->d_diag, n_diag * sizeof(void*)) == hipSuccess) &&
            hipMalloc(&p->d_baby, n_baby * sizeof(void*)) == hipSuccess &&
            hipMalloc(&p->d_ct, n_ct * sizeof(void*)) == hipSuccess;
  if (ok) {
    // the pt-MAC's operands: the ciphertext regions, or the extended ones
    for (size_t t = 0; t < n_baby; ++t)
      baby[t] = d->lazy_moddown ? p->ext_work + t * ext_words : p->work + t * p->ct_words;
    for (size_t t = 0; t < n_ct; ++t)
      cts[t] = d->lazy_moddown ? p->ext_work + (n_baby + t) * ext_words
                               : p->work + (n_baby + t) * p->ct_words;
    ok = (bank || hipMemcpy(p->d_diag, p->diag.data(), n_diag * sizeof(void*),
                            hipMemcpyHostToDevice) == hipSuccess) &&
         hipMemcpy(p->d_baby, baby.data(), n_baby * sizeof(void*), hipMemcpyHostToDevice) ==
             hipSuccess &&
         hipMemcpy(p->d_ct, cts.data(), n_ct * sizeof(void*), hipMemcpyHostToDevice) == hipSuccess;
  }
  if (ok)
    for (auto& e : p->ev) ok = ok && hipEventCreate(&e) == hipSuccess;
  if (!ok) {
    for (auto& e : p->ev)
      if (e) (void)hipEventDestroy(e);
    (void)hipFree(p->work);
    (void)hipFree(p->ext_work);
    (void)hipFree(p->d_diag);
    (void)hipFree(p->d_baby);
    (void)hipFree(p->d_ct);
    delete p;
    return fail(FESC_ERR_OOM, "matvec workspace or event allocation failed");
  }
  *out = p;
  return FESC_OK;
}

void matvec_plan_destroy(fesc_matvec_plan* p) {
  if (!p) return;
  (void)hipDeviceSynchronize();
  (void)hipFree(p->work);
  (void)hipFree(p->ext_work);
  (void)hipFree(p->d_diag);
  (void)hipFree(p->d_baby);
  (void)hipFree(p->d_ct);
  (void)hipFree(p->mwork);
  (void)hipFree(p->d_mbaby);
  (void)hipFree(p->d_mct);
  for (auto& e : p->ev)
    if (e) (void)hipEventDestroy(e);
  delete p;
}

int ptct_matvec(Context* c, fesc_matvec_plan* p, const uint64_t* const* in,
                uint64_t* const* out, hipStream_t s) {
  const fesc_matvec_desc& d = p->d;
  const uint32_t level = d.level;
  const size_t W = p->ct_words, n_baby = (size_t)d.n_in * d.n1;
  uint64_t* baby = p->work;
  uint64_t* ct = p->work + n_baby * W;
  uint64_t* tmp = ct + (size_t)d.n_out * d.n2 * W;
  const size_t n = c->n;
  int err;
  const bool lazy = d.lazy_moddown;
  const uint32_t rows = diag_rows(c, d);
  const size_t ext_words = (size_t)2 * rows * n;
  if ((err = check_plan_keys(c, d, p->giant))) return err;
  const LevelTables* T = nullptr;
  if (lazy && !(T = level_tables(c, level, &err))) return err;
  HIPCK(hipEventRecord(p->ev[0], s));
  // baby steps: one ModUp per input, all (u, q) key switches batched; with
  // double hoisting their outputs stay in the extended basis
  std::vector<KsSource> srcs;
  std::vector<KsJob> jobs;
  for (uint32_t u = 0; u < d.n_in; ++u) {
    for (uint32_t q = 0; q < d.n1; ++q) {
      const size_t t = (size_t)u * d.n1 + q;
      uint64_t* o = lazy ? p->ext_work + t * ext_words : baby + t * W;
      const uint32_t g = galois_of_step(c, (int32_t)(((int64_t)q * d.unit) % (c->n / 2)));
      if (g == 1) {
        if (lazy)
          hipLaunchKernelGGL(k_ext_identity, dim3(c->n / kThreads, rows, 2), dim3(kThreads), 0,
                             s, in[u], o, c->n, level, rows, T->pmod, c->d_pk);
        else
          HIPCK(hipMemcpyAsync(o, in[u], W * 8, hipMemcpyDeviceToDevice, s));
        HIPCK(hipGetLastError());
        continue;
      }
      jobs.push_back(KsJob{(uint32_t)srcs.size(), c->keys.find(g)->second, g, in[u], 1u, g,
                           nullptr, o});
    }
    srcs.push_back(KsSource{in[u] + n, 2 * n});
    if (srcs.size() == kMaxBatch || u + 1 == d.n_in) {
      if ((err = key_switch_batch(c, level, srcs, jobs, s, 0, nullptr, lazy))) return err;
      srcs.clear();
      jobs.clear();
    }
  }
  HIPCK(hipEventRecord(p->ev[1], s));
  // pt-MAC over all (b, p)
  const uint32_t n_outputs = d.n_out * d.n2;
  const PtLayout lay = lazy ? PtLayout{(uint32_t)n, rows * (uint32_t)n, level, c->L}
                            : PtLayout{2 * (uint32_t)n, (uint32_t)n, level, c->L};
  dim3 grid((c->n / kThreads) * rows * ((n_outputs + kGroup - 1) / kGroup));
  if (p->bank)
    hipLaunchKernelGGL((k_ptmac<kGroup, true>), grid, dim3(kThreads), 0, s, p->d_baby,
                       (const uint64_t* const*)nullptr, p->bank, p->d_ct, n_outputs,
                       (uint32_t)n_baby, c->n, rows, c->d_pk, lay);
  else
    hipLaunchKernelGGL((k_ptmac<kGroup, false>), grid, dim3(kThreads), 0, s, p->d_baby,
                       p->d_diag, (const uint32_t*)nullptr, p->d_ct, n_outputs,
                       (uint32_t)n_baby, c->n, rows, c->d_pk, lay);
  HIPCK(hipGetLastError());
  if (lazy) {
    // one ModDown per c~_{b,p}, into the ciphertext regions
    std::vector<uint64_t*> cts(n_outputs);
    for (uint32_t t = 0; t < n_outputs; ++t) cts[t] = ct + (size_t)t * W;
    if ((err = op_moddown_many(c, n_outputs, p->ext_work + n_baby * ext_words, cts.data(), level,
                               s)))
      return err;
  }
  HIPCK(hipEventRecord(p->ev[2], s));
  // giant steps: y_b = sum_p Phi^(p n1)(c~_{b,p}).  One giant step: one batch
  // over b with the sum folded into the key switch's combine.  More: every
  // rotation of every (b, p >= 1) in one batch, in place, then the sums (the
  // same residues: the rotations do not depend on the partial sums, and the
  // additions are exact mod q)
  std::vector<const uint64_t*> gin(d.n_out);
  std::vector<uint64_t*> gout(d.n_out);
  std::vector<int32_t> gst(d.n_out);
  if (d.n2 == 2) {
    for (uint32_t b = 0; b < d.n_out; ++b) {
      gin[b] = ct + ((size_t)b * d.n2 + 1) * W;
      gout[b] = ct + (size_t)b * d.n2 * W;
      gst[b] = (int32_t)(p->giant % (c->n / 2));
    }
    if ((err = op_rotate_batch(c, d.n_out, gin.data(), gst.data(), gout.data(),
                               (const uint64_t* const*)gout.data(), level, s)))
      return err;
  } else if (d.n2 > 2) {
    std::vector<const uint64_t*> rin;
    std::vector<uint64_t*> rout;
    std::vector<int32_t> rst;
    for (uint32_t b = 0; b < d.n_out; ++b)
      for (uint32_t g = 1; g < d.n2; ++g) {
        uint64_t* cg = ct + ((size_t)b * d.n2 + g) * W;
        rin.push_back(cg);
        rout.push_back(cg);
        rst.push_back((int32_t)(((int64_t)g * p->giant) % (c->n / 2)));
      }
    // in place: each job's c0 addend is read by the inner product and its c1
    // by the ModUp, both before the combine writes the job's output (rotation
    // jobs fold their addend, so the combine reads neither)
    if ((err = op_rotate_batch(c, (uint32_t)rin.size(), rin.data(), rst.data(), rout.data(),
                               nullptr, level, s)))
      return err;
    for (uint32_t b = 0; b < d.n_out; ++b) {
      uint64_t* y = ct + (size_t)b * d.n2 * W;
      for (uint32_t g = 1; g < d.n2; ++g)
        HIPCK(k_binary_launch(c, y, y + (size_t)g * W, y, 2 * level, 1, 0, s));
    }
  }
  // real extraction: t_b = conj(y_b) + y_b, one batch
  std::vector<uint64_t*> res(d.n_out);
  for (uint32_t b = 0; b < d.n_out; ++b) res[b] = ct + (size_t)b * d.n2 * W;
  if (d.real_extract) {
    for (uint32_t b = 0; b < d.n_out; ++b) {
      gin[b] = res[b];
      gout[b] = tmp + (size_t)b * W;
      gst[b] = INT32_MIN;
    }
    if ((err = op_rotate_batch(c, d.n_out, gin.data(), gst.data(), gout.data(), gin.data(),
                               level, s)))
      return err;
    for (uint32_t b = 0; b < d.n_out; ++b) res[b] = gout[b];
  }
  if (d.complex_pair) {
    // output P = y_2P + conj(y_2P+1), one batch of conjugations
    const uint32_t np_ = d.n_out / 2;
    std::vector<const uint64_t*> even(np_);
    for (uint32_t P = 0; P < np_; ++P) {
      gin[P] = res[2 * P + 1];
      even[P] = res[2 * P];
      gout[P] = tmp + (size_t)P * W;
      gst[P] = INT32_MIN;
    }
    if ((err = op_rotate_batch(c, np_, gin.data(), gst.data(), gout.data(), even.data(), level,
                               s)))
      return err;
    for (uint32_t P = 0; P < np_; ++P) res[P] = gout[P];
  }
  const uint32_t n_res = matvec_outputs(d);
  if (d.rescale) {
    if ((err = op_rescale_many(c, n_res, res.data(), out, level, s))) return err;
  } else {
    for (uint32_t b = 0; b < n_res; ++b)
      HIPCK(hipMemcpyAsync(out[b], res[b], W * 8, hipMemcpyDeviceToDevice, s));
  }
  HIPCK(hipEventRecord(p->ev[3], s));
  return FESC_OK;
}

// The plan's projection of `count` independent vectors (plans with one input
// and one output block, no extraction, no double hoisting): vector v's
// ciphertext in[v] -> out[v], the same residues as ptct_matvec on each.  Up
// to kMaxBatch vectors at a time share the launches: one ModUp launch for all
// of them and their baby steps batched with jobs of one rotation under one
// key, one pt-MAC per vector, every giant-step rotation in one batch, one
// batched rescale.
int ptct_matvec_many(Context* c, fesc_matvec_plan* p, uint32_t count, const uint64_t* const* in,
                     uint64_t* const* out, hipStream_t s) {
  const fesc_matvec_desc& d = p->d;
  if (d.n_in != 1 || d.n_out != 1 || d.lazy_moddown || d.real_extract || d.complex_pair)
    return fail(FESC_ERR_ARG, "batched projection: one input and one output block, "
                              "no extraction, no double hoisting");
  if (!count) return FESC_OK;
  const uint32_t level = d.level, n1 = d.n1, n2 = d.n2;
  const size_t W = p->ct_words, n = c->n, per = (size_t)n1 + n2;
  int err;
  if ((err = check_plan_keys(c, d, p->giant))) return err;
  const uint32_t want = std::min<uint32_t>(count, kMaxBatch);
  if (p->mcap < want) {
    (void)hipStreamSynchronize(s);  // earlier calls may still use the old workspace
    (void)hipFree(p->mwork);
    (void)hipFree(p->d_mbaby);
    (void)hipFree(p->d_mct);
    p->mwork = nullptr;
    p->d_mbaby = nullptr;
    p->d_mct = nullptr;
    p->mcap = 0;
    std::vector<const uint64_t*> baby((size_t)want * n1);
    std::vector<uint64_t*> cts((size_t)want * n2);
    bool ok = hipMalloc(&p->mwork, want * per * W * 8) == hipSuccess &&
              hipMalloc(&p->d_mbaby, baby.size() * sizeof(void*)) == hipSuccess &&
              hipMalloc(&p->d_mct, cts.size() * sizeof(void*)) == hipSuccess;
    if (ok) {
      for (size_t v = 0; v < want; ++v) {
        for (size_t q = 0; q < n1; ++q) baby[v * n1 + q] = p->mwork + (v * per + q) * W;
        for (size_t g = 0; g < n2; ++g) cts[v * n2 + g] = p->mwork + (v * per + n1 + g) * W;
      }
      ok = hipMemcpy(p->d_mbaby, baby.data(), baby.size() * sizeof(void*),
                     hipMemcpyHostToDevice) == hipSuccess &&
           hipMemcpy(p->d_mct, cts.data(), cts.size() * sizeof(void*), hipMemcpyHostToDevice) ==
               hipSuccess;
    }
    if (!ok) {
      (void)hipFree(p->mwork);
      (void)hipFree(p->d_mbaby);
      (void)hipFree(p->d_mct);
      p->mwork = nullptr;
      p->d_mbaby = nullptr;
      p->d_mct = nullptr;
      return fail(FESC_ERR_OOM, "batched projection workspace");
    }
    p->mcap = want;
  }
  auto baby_of = [&](uint32_t v, uint32_t q) { return p->mwork + ((size_t)v * per + q) * W; };
  auto ct_of = [&](uint32_t v, uint32_t g) { return p->mwork + ((size_t)v * per + n1 + g) * W; };
  for (uint32_t b0 = 0; b0 < count; b0 += p->mcap) {
    const uint32_t nb = std::min(p->mcap, count - b0);
    // baby steps
    std::vector<KsSource> srcs;
    std::vector<KsJob> jobs;
    for (uint32_t v = 0; v < nb; ++v) {
      const uint64_t* x = in[b0 + v];
      for (uint32_t q = 0; q < n1; ++q) {
        const uint32_t g = galois_of_step(c, (int32_t)(((int64_t)q * d.unit) % (c->n / 2)));
        if (g == 1) {
          HIPCK(hipMemcpyAsync(baby_of(v, q), x, W * 8, hipMemcpyDeviceToDevice, s));
          continue;
        }
        jobs.push_back(KsJob{v, c->keys.find(g)->second, g, x, 1u, g, nullptr, baby_of(v, q)});
      }
      srcs.push_back(KsSource{x + n, 2 * n});
    }
    if ((err = key_switch_batch(c, level, srcs, jobs, s, 0, nullptr, false))) return err;
    // pt-MAC per vector
    const uint32_t rows = diag_rows(c, d);
    const PtLayout lay{2 * (uint32_t)n, (uint32_t)n, level, c->L};
    const dim3 grid((c->n / kThreads) * rows * ((n2 + kGroup - 1) / kGroup));
    for (uint32_t v = 0; v < nb; ++v) {
      if (p->bank)
        hipLaunchKernelGGL((k_ptmac<kGroup, true>), grid, dim3(kThreads), 0, s,
                           p->d_mbaby + (size_t)v * n1, (const uint64_t* const*)nullptr, p->bank,
                           p->d_mct + (size_t)v * n2, n2, n1, c->n, rows, c->d_pk, lay);
      else
        hipLaunchKernelGGL((k_ptmac<kGroup, false>), grid, dim3(kThreads), 0, s,
                           p->d_mbaby + (size_t)v * n1, p->d_diag, (const uint32_t*)nullptr,
                           p->d_mct + (size_t)v * n2, n2, n1, c->n, rows, c->d_pk, lay);
      HIPCK(hipGetLastError());
    }
    // giant steps (as in ptct_matvec)
    std::vector<const uint64_t*> gin;
    std::vector<uint64_t*> gout;
    std::vector<int32_t> gst;
    if (n2 == 2) {
      for (uint32_t v = 0; v < nb; ++v) {
        gin.push_back(ct_of(v, 1));
        gout.push_back(ct_of(v, 0));
        gst.push_back((int32_t)(p->giant % (c->n / 2)));
      }
      if ((err = op_rotate_batch(c, nb, gin.data(), gst.data(), gout.data(),
                                 (const uint64_t* const*)gout.data(), level, s)))
        return err;
    } else if (n2 > 2) {
      for (uint32_t v = 0; v < nb; ++v)
        for (uint32_t g = 1; g < n2; ++g) {
          gin.push_back(ct_of(v, g));
          gout.push_back(ct_of(v, g));
          gst.push_back((int32_t)(((int64_t)g * p->giant) % (c->n / 2)));
        }
      // in place, as in ptct_matvec
      if ((err = op_rotate_batch(c, (uint32_t)gin.size(), gin.data(), gst.data(), gout.data(),
                                 nullptr, level, s)))
        return err;
      for (uint32_t v = 0; v < nb; ++v)
        for (uint32_t g = 1; g < n2; ++g)
          HIPCK(k_binary_launch(c, ct_of(v, 0), ct_of(v, g), ct_of(v, 0), 2 * level, 1, 0, s));
    }
    std::vector<uint64_t*> res(nb);
    for (uint32_t v = 0; v < nb; ++v) res[v] = ct_of(v, 0);
    if (d.rescale) {
      if ((err = op_rescale_many(c, nb, res.data(), out + b0, level, s))) return err;
    } else {
      for (uint32_t v = 0; v < nb; ++v)
        HIPCK(hipMemcpyAsync(out[b0 + v], res[v], W * 8, hipMemcpyDeviceToDevice, s));
    }
  }
  return FESC_OK;
}

}  // namespace fesc

extern "C" {

int fesc_matvec_plan_create(fesc_ctx* ctx, const fesc_matvec_desc* desc,
                            const uint64_t* const* diags, fesc_matvec_plan** plan) {
  if (!ctx) return fesc::fail(FESC_ERR_ARG, "null context");
  if (!diags) return fesc::fail(FESC_ERR_ARG, "null diagonal table");
  return fesc::matvec_plan_create(ctx, desc, diags, nullptr, plan, INT64_MIN);
}

int fesc_matvec_bank_words(const fesc_ctx* ctx, const fesc_matvec_desc* desc, size_t* words) {
  if (!ctx || !words) return fesc::fail(FESC_ERR_ARG, "null argument");
  int rc = fesc::check_desc(ctx, desc);
  if (rc) return rc;
  // 32-bit words: rows * N * terms * record words, an even count (N is even)
  const uint32_t outputs = desc->n_out * desc->n2;
  *words = (size_t)desc->n_in * desc->n1 * fesc::bank_record_words(outputs) *
           fesc::diag_rows(ctx, *desc) * ctx->n / 2;
  return FESC_OK;
}

int fesc_matvec_bank_pack_many(fesc_ctx* ctx, const fesc_matvec_desc* desc, uint64_t* bank,
                               uint32_t first, uint32_t count, const uint64_t* pts,
                               size_t pt_stride, void* stream) {
  if (!ctx || !bank) return fesc::fail(FESC_ERR_ARG, "null argument");
  int rc = fesc::check_desc(ctx, desc);
  if (rc) return rc;
  const uint32_t terms = desc->n_in * desc->n1, outputs = desc->n_out * desc->n2;
  const uint32_t rows = fesc::diag_rows(ctx, *desc);
  if (count == 0) return FESC_OK;
  if (!pts) return fesc::fail(FESC_ERR_ARG, "null plaintexts");
  if (count > 65535) return fesc::fail(FESC_ERR_ARG, "at most 65535 diagonals per call");
  if ((uint64_t)first + count > (uint64_t)terms * outputs)
    return fesc::fail(FESC_ERR_ARG, "diagonal index out of range");
  if (count > 1 && pt_stride < (size_t)rows * ctx->n)
    return fesc::fail(FESC_ERR_ARG, "plaintext stride below rows * N");
  hipLaunchKernelGGL(fesc::k_bank_pack, dim3(ctx->n / fesc::kThreads, rows, count),
                     dim3(fesc::kThreads), 0, reinterpret_cast<hipStream_t>(stream), pts,
                     pt_stride, reinterpret_cast<uint32_t*>(bank), first, ctx->n, outputs,
                     terms);
  return fesc::hip_check(hipGetLastError(), "bank_pack");
}

int fesc_matvec_bank_pack(fesc_ctx* ctx, const fesc_matvec_desc* desc, uint64_t* bank,
                          uint32_t index, const uint64_t* pt, void* stream) {
  return fesc_matvec_bank_pack_many(ctx, desc, bank, index, 1, pt, 0, stream);
}

int fesc_bsgs_diagonal_slots(fesc_ctx* ctx, const fesc_matvec_desc* desc, const double* W,
                             uint32_t d_in, uint32_t d_out, uint32_t segs, uint32_t first,
                             uint32_t count, double* z, void* stream) {
  if (!ctx || !W || !z) return fesc::fail(FESC_ERR_ARG, "null argument");
  int rc = fesc::check_desc(ctx, desc);
  if (rc) return rc;
  const uint32_t n_slots = ctx->n / 2;
  if (!segs || n_slots % desc->unit || (n_slots / desc->unit) % segs)
    return fesc::fail(FESC_ERR_ARG, "unit * segs must divide N/2");
  const uint64_t total = (uint64_t)desc->n_out * desc->n2 * desc->n_in * desc->n1;
  if ((uint64_t)first + count > total) return fesc::fail(FESC_ERR_ARG, "diagonal range");
  if (count == 0) return FESC_OK;
  if (count > 65535) return fesc::fail(FESC_ERR_ARG, "at most 65535 diagonals per call");
  const fesc::SlotDesc S{desc->n_in, desc->n1, desc->n2, desc->unit, segs,
                         n_slots, d_in, d_out, first,
                         desc->complex_pair ? 2u : (desc->real_extract ? 1u : 0u)};
  hipLaunchKernelGGL(fesc::k_bsgs_slots, dim3((n_slots + fesc::kThreads - 1) / fesc::kThreads,
                                              count),
                     dim3(fesc::kThreads), 0, reinterpret_cast<hipStream_t>(stream), W, S,
                     reinterpret_cast<double2*>(z));
  return fesc::hip_check(hipGetLastError(), "bsgs_diagonal_slots");
}

int fesc_matvec_plan_create_bank(fesc_ctx* ctx, const fesc_matvec_desc* desc,
                                 const uint64_t* bank, fesc_matvec_plan** plan) {
  if (!ctx) return fesc::fail(FESC_ERR_ARG, "null context");
  if (!bank) return fesc::fail(FESC_ERR_ARG, "null bank");
  return fesc::matvec_plan_create(ctx, desc, nullptr, bank, plan, INT64_MIN);
}

void fesc_matvec_plan_destroy(fesc_matvec_plan* plan) { fesc::matvec_plan_destroy(plan); }

int fesc_ptct_matvec(fesc_ctx* ctx, fesc_matvec_plan* plan, const uint64_t* const* in,
                     uint64_t* const* out, void* stream) {
  if (!ctx || !plan || !in || !out) return fesc::fail(FESC_ERR_ARG, "null argument");
  for (uint32_t u = 0; u < plan->d.n_in; ++u)
    if (!in[u]) return fesc::fail(FESC_ERR_ARG, "null input");
  for (uint32_t b = 0; b < fesc::matvec_outputs(plan->d); ++b)
    if (!out[b]) return fesc::fail(FESC_ERR_ARG, "null output");
  return fesc::ptct_matvec(ctx, plan, in, out, reinterpret_cast<hipStream_t>(stream));
}

int fesc_matvec_phase_ms(const fesc_matvec_plan* plan, float* baby_ms, float* ptmac_ms,
                         float* tail_ms) {
  if (!plan || !baby_ms || !ptmac_ms || !tail_ms) return fesc::fail(FESC_ERR_ARG, "null argument");
  float* dst[3] = {baby_ms, ptmac_ms, tail_ms};
  for (int i = 0; i < 3; ++i) {
    hipError_t e = hipEventElapsedTime(dst[i], plan->ev[i], plan->ev[i + 1]);
    if (e != hipSuccess) return fesc::hip_check(e, "matvec phase timing");
  }
  return FESC_OK;
}

}  // extern "C"
