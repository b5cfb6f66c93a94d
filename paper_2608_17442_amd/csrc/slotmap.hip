// Public slot maps and the HEScan broadcasts br^(kappa) (Sec. "CKKS
// Primitives and Slot Maps"; the exact maps of Appendix "HEScan Kernel Packing
// and Correctness").  A slot map moves each of its runs of slots, term
// t = p n1 + q, by its own rotation offset + q stride + p giant_stride and
// replicates the result by doubling:
//
//   out = sum_{u < R} rho( RS( sum_t M_t (.) rho(rho(v; offset); q stride + p giant) ); -u S )
//
// Step 2 is the diagonal method with 0/1 masks, split baby-step/giant-step by
// the projection's plan (hoisted baby steps, one pt-MAC pass, giant steps, one
// rescale); step 3 is log2 R rotate-and-add key switches.  The broadcasts of
// the scan factors are instances (fesc_br_desc): x spreads a chunk's channels
// to stride d_s and replicates each over its d_s slots; a places each head at
// P d_s / R positions and replicates R <= 512 times (the error of an output
// slot grows as the square root of R: R doublings add the key-switching noise
// of R shifted copies); B and C select a group's d_s values and tile them over
// the chunk's channels.
#include <algorithm>
#include <string>
#include <vector>

#include "fesc_internal.hpp"
#include "ops.hpp"

struct fesc_slot_map_plan {
  fesc_slot_map_desc d;
  fesc_matvec_plan* mv = nullptr;  // step 2 (n_in = n_out = 1, rescale)
  uint64_t* zero = nullptr;        // [level][N] zero plaintext for masks past `terms`
  uint64_t* work = nullptr;        // rotated input [level][2][N], two [level-1][2][N]
  uint64_t* bwork = nullptr;       // the same per item of a batch (up to kSlotMapGroup items)
  uint32_t bcap = 0;               // items bwork holds
};

namespace fesc {

int matvec_plan_create(Context* c, const fesc_matvec_desc* d, const uint64_t* const* diags,
                       const uint64_t* bank, fesc_matvec_plan** out, int64_t giant_unit);
void matvec_plan_destroy(fesc_matvec_plan* p);
int ptct_matvec_many(Context* c, fesc_matvec_plan* p, uint32_t count, const uint64_t* const* in,
                     uint64_t* const* out, hipStream_t s);
int ptct_matvec(Context* c, fesc_matvec_plan* p, const uint64_t* const* in,
                uint64_t* const* out, hipStream_t s);

namespace {

constexpr int kThreads = 256;
// largest replication of the decay's broadcast (see the file comment)
constexpr uint64_t kMaxDecayRep = 512;

uint32_t giant_count(const fesc_slot_map_desc& d) { return (d.terms + d.n1 - 1) / d.n1; }

// v mod m in [0, m) for a signed v
int32_t slot_step(int64_t v, uint32_t m) {
  const int64_t r = v % (int64_t)m;
  return (int32_t)(r < 0 ? r + m : r);
}

int check_map(const Context* c, const fesc_slot_map_desc* d) {
  if (!d) return fail(FESC_ERR_ARG, "null slot-map descriptor");
  if (d->level < 2 || d->level > c->L)
    return fail(FESC_ERR_LEVEL, "slot map needs 2 <= level <= L (one rescale)");
  const uint64_t ns = c->n / 2;
  if (!d->terms || !d->n1 || !d->width) return fail(FESC_ERR_ARG, "slot-map sizes must be positive");
  // runs ordered by t = p n1 + q and disjoint: each run ends before the next
  // baby run, each giant row before the next row; then the last run ends last
  const uint32_t n2 = giant_count(*d), pl = (d->terms - 1) / d->n1, ql = (d->terms - 1) % d->n1;
  if (d->n1 > 1 && d->terms > 1 && d->width > d->dst_stride)
    return fail(FESC_ERR_ARG, "slot-map runs overlap");
  if (n2 > 1 && (uint64_t)(d->n1 - 1) * d->dst_stride + d->width > d->dst_giant)
    return fail(FESC_ERR_ARG, "slot-map runs overlap");
  if ((uint64_t)d->dst0 + (uint64_t)pl * d->dst_giant + (uint64_t)ql * d->dst_stride + d->width >
      ns)
    return fail(FESC_ERR_ARG, "slot-map runs leave the slots");
  if (!d->rep_count || (d->rep_count & (d->rep_count - 1)) || d->rep_count > ns)
    return fail(FESC_ERR_ARG, "replication count must be a power of two up to N/2");
  return FESC_OK;
}

// Mask m = p n1 + q of the map, rotated by -p giant: 1 at slot j where
// j - p giant (mod N/2) lies in run (p, q).
__global__ __launch_bounds__(kThreads) void k_mask_slots(double2* __restrict__ z, uint32_t ns,
                                                         uint32_t first, uint32_t n1,
                                                         uint32_t terms, int32_t giant,
                                                         uint32_t dst0, uint32_t dst_stride,
                                                         uint32_t dst_giant, uint32_t width) {
  const uint32_t j = blockIdx.x * kThreads + threadIdx.x;
  if (j >= ns) return;
  const uint32_t m = first + blockIdx.y, p = m / n1, q = m % n1;
  double v = 0.0;
  if (m < terms) {
    int64_t jj = ((int64_t)j - (int64_t)p * giant) % (int64_t)ns;
    if (jj < 0) jj += ns;
    const int64_t start = (int64_t)dst0 + (int64_t)q * dst_stride + (int64_t)p * dst_giant;
    v = (jj >= start && jj < start + width) ? 1.0 : 0.0;
  }
  z[(size_t)blockIdx.y * ns + j] = double2{v, 0.0};
}

bool pow2(uint64_t x) { return x && !(x & (x - 1)); }

uint32_t baby_of(uint32_t terms) {
  uint32_t n1 = 1;
  while ((uint64_t)n1 * n1 < terms) n1 *= 2;
  return n1;
}

}  // namespace

int br_desc(uint32_t log_n, const fesc_br_shape* sh, uint32_t kind, uint32_t k, uint32_t kappa,
            uint32_t level, fesc_slot_map_desc* out) {
  if (!sh || !out) return fail(FESC_ERR_ARG, "null argument");
  if (log_n < 1 || log_n > 17) return fail(FESC_ERR_ARG, "log_n out of range");
  const uint64_t ns = 1ull << (log_n - 1), H = sh->H, P = sh->P, G = sh->G, ds = sh->d_s, cs = sh->c_state;
  if (!H || !P || !G || !ds || !cs) return fail(FESC_ERR_ARG, "broadcast shape must be positive");
  const uint64_t E = H * P;
  if (E % cs || kappa >= E / cs || cs * ds > ns)
    return fail(FESC_ERR_ARG, "chunks must tile the channels and fit the slots");
  fesc_slot_map_desc d{};
  d.level = level;
  if (kind == FESC_BR_X) {
    if (!pow2(ds) || (k + 1) * E > ns) return fail(FESC_ERR_ARG, "x broadcast: shape");
    d.offset = slot_step((int64_t)(k * E + kappa * cs), (uint32_t)ns);
    d.stride = (int32_t)(1 - (int64_t)ds);
    d.terms = (uint32_t)cs;
    d.dst_stride = (uint32_t)ds;
    d.width = 1;
    d.rep_stride = 1;
    d.rep_count = (uint32_t)ds;
  } else if (kind == FESC_BR_A) {
    if (cs % P || !pow2(P * ds) || (k + 1) * H > ns) return fail(FESC_ERR_ARG, "a broadcast: shape");
    // head j of the chunk at positions j P d_s + u R, u < P d_s / R (baby
    // steps), heads as giant steps; then R copies
    const uint64_t heads = cs / P, span = P * ds, R = span < kMaxDecayRep ? span : kMaxDecayRep;
    d.offset = slot_step((int64_t)(k * H + kappa * heads), (uint32_t)ns);
    d.n1 = (uint32_t)(span / R);
    d.terms = (uint32_t)(heads * d.n1);
    d.stride = -(int32_t)R;
    d.dst_stride = (uint32_t)R;
    d.giant_stride = (int32_t)(1 - (int64_t)span);
    d.dst_giant = (uint32_t)span;
    d.width = 1;
    d.rep_stride = 1;
    d.rep_count = (uint32_t)R;
    *out = d;
    return FESC_OK;
  } else if (kind == FESC_BR_B || kind == FESC_BR_C) {
    if (H % G || (k + 1) * G * ds > ns) return fail(FESC_ERR_ARG, "B/C broadcast: shape");
    const uint64_t Eg = P * (H / G);  // channels per group
    const uint64_t g_lo = kappa * cs / Eg, g_hi = (kappa * cs + cs - 1) / Eg;
    d.offset = slot_step((int64_t)(k * G * ds + g_lo * ds), (uint32_t)ns);
    d.width = (uint32_t)ds;
    d.rep_stride = (int32_t)ds;
    if (g_lo == g_hi) {  // the chunk lies inside one group: tile its d_s values
      if (!pow2(cs)) return fail(FESC_ERR_ARG, "B/C broadcast: chunk size");
      d.stride = 0;
      d.terms = 1;
      d.dst_stride = 0;
      d.rep_count = (uint32_t)cs;
    } else {  // whole groups: one run per group, tiled over its channels
      if (cs % Eg || !pow2(Eg)) return fail(FESC_ERR_ARG, "B/C broadcast: groups");
      d.stride = (int32_t)((int64_t)ds - (int64_t)(Eg * ds));
      d.terms = (uint32_t)(cs / Eg);
      d.dst_stride = (uint32_t)(Eg * ds);
      d.rep_count = (uint32_t)Eg;
    }
  } else {
    return fail(FESC_ERR_ARG, "unknown broadcast kind");
  }
  // one progression: giant steps continue the baby steps
  d.n1 = baby_of(d.terms);
  d.giant_stride = (int32_t)((int64_t)d.n1 * d.stride);
  d.dst_giant = d.n1 * d.dst_stride;
  *out = d;
  return FESC_OK;
}

int slot_map_mask_slots(Context* c, const fesc_slot_map_desc* d, uint32_t first, uint32_t count,
                        double2* z, hipStream_t s) {
  int err;
  if ((err = check_map(c, d))) return err;
  if (!z) return fail(FESC_ERR_ARG, "null argument");
  if (!count || count > 65535 || (uint64_t)first + count > (uint64_t)d->n1 * giant_count(*d))
    return fail(FESC_ERR_ARG, "mask range outside n1 * n2 (or more than 65535 masks)");
  const uint32_t ns = c->n / 2;
  hipLaunchKernelGGL(k_mask_slots, dim3((ns + kThreads - 1) / kThreads, count), dim3(kThreads), 0,
                     s, z, ns, first, d->n1, d->terms, d->giant_stride, d->dst0, d->dst_stride,
                     d->dst_giant, d->width);
  return hip_check(hipGetLastError(), "k_mask_slots");
}

void slot_map_plan_destroy(fesc_slot_map_plan* p) {
  if (!p) return;
  (void)hipDeviceSynchronize();
  matvec_plan_destroy(p->mv);
  (void)hipFree(p->zero);
  (void)hipFree(p->work);
  (void)hipFree(p->bwork);
  delete p;
}

int slot_map_plan_create(Context* c, const fesc_slot_map_desc* d, const uint64_t* const* masks,
                         fesc_slot_map_plan** out) {
  if (!out || !masks) return fail(FESC_ERR_ARG, "null argument");
  *out = nullptr;
  int err;
  if ((err = check_map(c, d))) return err;
  for (uint32_t t = 0; t < d->terms; ++t)
    if (!masks[t]) return fail(FESC_ERR_ARG, "null mask " + std::to_string(t));
  const uint32_t ns = c->n / 2;
  // keys of the offset rotation and of the doublings (the matvec plan
  // checks its own)
  std::vector<int32_t> steps{slot_step(d->offset, ns)};
  for (uint32_t r = 1; r < d->rep_count; r *= 2)
    steps.push_back(slot_step(-(int64_t)r * d->rep_stride, ns));
  for (int32_t st : steps) {
    const uint32_t g = galois_of_step(c, st);
    if (g != 1 && !c->keys.count(g))
      return fail(FESC_ERR_NO_KEY, "slot map needs the key of rotation " + std::to_string(st));
  }
  auto* p = new fesc_slot_map_plan();
  p->d = *d;
  const size_t n = c->n, level = d->level;
  const uint32_t n2 = giant_count(*d);
  const size_t diags = (size_t)d->n1 * n2;
  if (hipMalloc(&p->zero, level * n * 8) != hipSuccess ||
      hipMalloc(&p->work, (2 * level + 4 * (level - 1)) * n * 8) != hipSuccess ||
      hipMemset(p->zero, 0, level * n * 8) != hipSuccess) {
    slot_map_plan_destroy(p);
    return fail(FESC_ERR_OOM, "slot-map workspace");
  }
  std::vector<const uint64_t*> tab(diags);
  for (size_t t = 0; t < diags; ++t) tab[t] = t < d->terms ? masks[t] : p->zero;
  fesc_matvec_desc md{};
  md.level = d->level;
  md.n_in = md.n_out = 1;
  md.n1 = d->n1;
  md.n2 = n2;
  md.unit = (uint32_t)slot_step(d->stride, ns);
  if (!md.unit) md.unit = 1;  // a single term (n1 = n2 = 1) rotates by nothing
  md.rescale = 1;
  if ((err = matvec_plan_create(c, &md, tab.data(), nullptr, &p->mv,
                                slot_step(d->giant_stride, ns)))) {
    slot_map_plan_destroy(p);
    return err;
  }
  *out = p;
  return FESC_OK;
}

int slot_map(Context* c, fesc_slot_map_plan* p, const uint64_t* in, uint64_t* out,
             hipStream_t s) {
  const fesc_slot_map_desc& d = p->d;
  const size_t n = c->n, lo = d.level - 1;
  const uint32_t ns = c->n / 2;
  uint64_t* rot = p->work;
  uint64_t* y[2] = {rot + 2 * d.level * n, rot + 2 * d.level * n + 2 * lo * n};
  int err;
  const uint64_t* src = in;
  const int32_t off = slot_step(d.offset, ns);
  if (off) {
    if ((err = op_rotate_batch(c, 1, &in, &off, &rot, nullptr, d.level, s, nullptr))) return err;
    src = rot;
  }
  if ((err = ptct_matvec(c, p->mv, &src, &y[0], s))) return err;
  int cur = 0;
  if (d.rep_count == 1)
    return hip_check(hipMemcpyAsync(out, y[0], 2 * lo * n * 8, hipMemcpyDeviceToDevice, s),
                     "slot-map copy");
  for (uint32_t r = 1; r < d.rep_count; r *= 2) {
    const int32_t st = slot_step(-(int64_t)r * d.rep_stride, ns);
    uint64_t* dst = 2 * r == d.rep_count ? out : y[1 - cur];
    const uint64_t* a = y[cur];
    if ((err = op_rotate_batch(c, 1, &a, &st, &dst, &a, (uint32_t)lo, s, nullptr))) return err;
    cur = 1 - cur;
  }
  return FESC_OK;
}

// Items of a batched slot map processed together (their workspaces at once).
constexpr uint32_t kSlotMapGroup = 16;

// The plan's map for `count` inputs with their own first rotations: the
// offset rotations of a group share one key-switch launch, the step-2 sums of
// the group run as one batched projection (ptct_matvec_many), and every
// doubling is one launch over the group, all its jobs under one key.
int slot_map_batch(Context* c, fesc_slot_map_plan* p, uint32_t count, const uint64_t* const* ins,
                   const int32_t* offsets, uint64_t* const* outs, hipStream_t s) {
  if (!ins || !offsets || !outs) return fail(FESC_ERR_ARG, "null argument");
  if (!count || count > 65535) return fail(FESC_ERR_ARG, "batch of 1 .. 65535 items");
  const fesc_slot_map_desc& d = p->d;
  const size_t n = c->n, lo = d.level - 1;
  const uint32_t ns = c->n / 2;
  for (uint32_t i = 0; i < count; ++i) {
    if (!ins[i] || !outs[i]) return fail(FESC_ERR_ARG, "null item " + std::to_string(i));
    const uint32_t g = galois_of_step(c, slot_step(offsets[i], ns));
    if (g != 1 && !c->keys.count(g))
      return fail(FESC_ERR_NO_KEY, "slot map needs the key of rotation " +
                                       std::to_string(slot_step(offsets[i], ns)));
  }
  const size_t item = (2 * d.level + 4 * lo) * n;  // words per item
  const uint32_t want = std::min(kSlotMapGroup, count);
  if (p->bcap < want) {
    (void)hipStreamSynchronize(s);  // earlier batches may still use the old workspace
    (void)hipFree(p->bwork);
    p->bcap = 0;
    if (hipMalloc(&p->bwork, want * item * 8) != hipSuccess) {
      p->bwork = nullptr;
      return fail(FESC_ERR_OOM, "slot-map batch workspace");
    }
    p->bcap = want;
  }
  int err;
  for (uint32_t b0 = 0; b0 < count; b0 += p->bcap) {
    const uint32_t nb = std::min(p->bcap, count - b0);
    std::vector<const uint64_t*> src(nb), rin;
    std::vector<uint64_t*> rout, y0(nb), y1(nb);
    std::vector<int32_t> rst;
    for (uint32_t i = 0; i < nb; ++i) {
      uint64_t* w = p->bwork + i * item;
      y0[i] = w + 2 * d.level * n;
      y1[i] = y0[i] + 2 * lo * n;
      const int32_t off = slot_step(offsets[b0 + i], ns);
      src[i] = ins[b0 + i];
      if (off) {
        rin.push_back(ins[b0 + i]);
        rout.push_back(w);
        rst.push_back(off);
        src[i] = w;
      }
    }
    if (!rst.empty() && (err = op_rotate_batch(c, (uint32_t)rst.size(), rin.data(), rst.data(),
                                              rout.data(), nullptr, d.level, s, nullptr)))
      return err;
    if ((err = ptct_matvec_many(c, p->mv, nb, src.data(), y0.data(), s))) return err;
    if (d.rep_count == 1) {
      for (uint32_t i = 0; i < nb; ++i)
        if ((err = hip_check(hipMemcpyAsync(outs[b0 + i], y0[i], 2 * lo * n * 8,
                                            hipMemcpyDeviceToDevice, s), "slot-map copy")))
          return err;
      continue;
    }
    std::vector<uint64_t*>* cur = &y0;
    std::vector<uint64_t*>* nxt = &y1;
    for (uint32_t r = 1; r < d.rep_count; r *= 2) {
      const std::vector<int32_t> st(nb, slot_step(-(int64_t)r * d.rep_stride, ns));
      std::vector<const uint64_t*> a(cur->begin(), cur->end());
      std::vector<uint64_t*> dst = 2 * r == d.rep_count
                                       ? std::vector<uint64_t*>(outs + b0, outs + b0 + nb)
                                       : *nxt;
      if ((err = op_rotate_batch(c, nb, a.data(), st.data(), dst.data(), a.data(), (uint32_t)lo,
                                 s, nullptr)))
        return err;
      std::swap(cur, nxt);
    }
  }
  return FESC_OK;
}

}  // namespace fesc

extern "C" {

int fesc_br_desc(uint32_t log_n, const fesc_br_shape* shape, uint32_t kind, uint32_t k,
                 uint32_t kappa, uint32_t level, fesc_slot_map_desc* out) {
  return fesc::br_desc(log_n, shape, kind, k, kappa, level, out);
}

int fesc_slot_map_mask_slots(fesc_ctx* ctx, const fesc_slot_map_desc* desc, uint32_t first,
                             uint32_t count, double* z, void* stream) {
  if (!ctx) return fesc::fail(FESC_ERR_ARG, "null context");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  return fesc::slot_map_mask_slots(ctx, desc, first, count, reinterpret_cast<double2*>(z), s);
}

int fesc_slot_map_plan_create(fesc_ctx* ctx, const fesc_slot_map_desc* desc,
                              const uint64_t* const* masks, fesc_slot_map_plan** plan) {
  if (!ctx) return fesc::fail(FESC_ERR_ARG, "null context");
  return fesc::slot_map_plan_create(ctx, desc, masks, plan);
}

void fesc_slot_map_plan_destroy(fesc_slot_map_plan* plan) { fesc::slot_map_plan_destroy(plan); }

int fesc_slot_map(fesc_ctx* ctx, fesc_slot_map_plan* plan, const uint64_t* in, uint64_t* out,
                  void* stream) {
  if (!ctx || !plan || !in || !out) return fesc::fail(FESC_ERR_ARG, "null argument");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  return fesc::slot_map(ctx, plan, in, out, s);
}

int fesc_slot_map_batch(fesc_ctx* ctx, fesc_slot_map_plan* plan, uint32_t count,
                        const uint64_t* const* ins, const int32_t* offsets,
                        uint64_t* const* outs, void* stream) {
  if (!ctx || !plan) return fesc::fail(FESC_ERR_ARG, "null argument");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  return fesc::slot_map_batch(ctx, plan, count, ins, offsets, outs, s);
}

}  // extern "C"
