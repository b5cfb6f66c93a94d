// Rotation batch that allocates nothing, for callers that cannot call
// hipMalloc (work under HIP graph capture, tight serving loops, harnesses that
// forbid device allocation).
//
// Its key-switch temporaries live in one statically allocated device array
// per GPU (`scratch` below, kStaticScratchBytes, held until the process
// ends).  In host code the array's name is only a host-side stand-in, never a
// device address: the context's creation, with its device current, asks the
// runtime for the array's device address on that device (once per device) and
// every launch uses that address.  All calls on one GPU share the array, so
// calls that overlap on one GPU race; no region needs clearing, since every
// word the key switch reads is written earlier in the same call (the inverse
// transforms write the ModUp digits, the conversions the extended rows, the
// inner product every accumulator row, ModDown its conversions).
#include <map>
#include <mutex>

#include "fesc_internal.hpp"
#include "ops.hpp"
#include "scratch.hpp"

namespace {
constexpr size_t kStaticScratchBytes = size_t(256) << 20;  // 256 MiB per GPU
}  // namespace

static __device__ __align__(256) uint64_t scratch[kStaticScratchBytes / sizeof(uint64_t)];

namespace fesc {

int static_scratch_init(Context* c) {
  static std::mutex mu;
  static std::map<int, uint64_t*> addr;  // device -> address of `scratch` there
  std::lock_guard<std::mutex> lock(mu);
  auto it = addr.find(c->device);
  if (it == addr.end()) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(::scratch));
    if (e != hipSuccess || !p) return hip_check(e, "hipGetSymbolAddress(scratch)");
    it = addr.emplace(c->device, static_cast<uint64_t*>(p)).first;
  }
  c->static_scratch = it->second;
  return FESC_OK;
}

size_t static_scratch_bytes() { return kStaticScratchBytes; }

// Words one rotation's key switch needs at `level`: its ModUp digits
// [level][N], extended digits [dnum_l][level+alpha][N], inner products
// [2][level+alpha][N] and ModDown conversions [2][level][N].
size_t rotate_scratch_words(const Context* c, uint32_t level) {
  const size_t E = level + c->alpha, dnum_l = (level + c->alpha - 1) / c->alpha;
  return (level + dnum_l * E + 2 * E + 2 * (size_t)level) * c->n;
}

int op_rotate_batch_static(Context* c, uint32_t count, const uint64_t* const* ins,
                           const int32_t* steps, uint64_t* const* outs, uint32_t level,
                           hipStream_t s) {
  if (!c->static_scratch) return fail(FESC_ERR_ARG, "static scratch not set up");
  const size_t per = rotate_scratch_words(c, level);
  const size_t cap = kStaticScratchBytes / sizeof(uint64_t) / per;
  if (cap == 0)
    return fail(FESC_ERR_ARG, "one rotation at level " + std::to_string(level) + " needs " +
                                  std::to_string(per * 8) + " bytes of scratch; the static "
                                  "scratch holds " + std::to_string(kStaticScratchBytes));
  // the per-level constants were built with the context: found, not allocated
  if (!c->level_tabs.count(level)) return fail(FESC_ERR_ARG, "level tables missing");
  const size_t B = cap < kMaxBatch ? cap : kMaxBatch;
  const size_t n = c->n, E = level + c->alpha, dnum_l = (level + c->alpha - 1) / c->alpha;
  Scratch S{};
  S.cap = (uint32_t)B;
  S.cc = c->static_scratch;
  S.ext = S.cc + B * level * n;
  S.acc = S.ext + B * dnum_l * E * n;
  S.y = S.acc + B * 2 * E * n;
  return op_rotate_batch(c, count, ins, steps, outs, nullptr, level, s, &S);
}

}  // namespace fesc
