// Negacyclic NTT / inverse NTT over word-sized primes, batched over rows.
//
// Definition (the forward transform's output order is bit-reversed):
//     A[j] = sum_k a_k psi^((2 brv(j) + 1) k)  mod q,
// psi the smallest primitive 2N-th root of unity mod q.  The transform is the
// radix-2 Cooley-Tukey network whose butterfly on the pair (j, j + t) uses the
// twiddle psi^brv((N + j) / 2t); the inverse is the Gentleman-Sande network
// with psi^-1 and a final scaling by N^-1.
//
// gfx950 mapping.  N = N1 * 256 with N1 = 2^(log N - 8) in [16, 256].  Two
// passes, each over independent sub-transforms held entirely on chip:
//   outer pass: the first log N1 stages couple only indices that agree mod
//               256, i.e. N1-point "columns" at stride 256;
//   inner pass: the last 8 stages couple only indices inside a contiguous
//               256-element block.
// Every sub-transform is split over 16-value register tiles: a thread runs
// four radix-2 stages on its 16 values (a radix-16 step), the tiles are
// transposed through LDS, and the thread runs the remaining stages.  Between
// the passes the row holds the signed fp64 intermediate in place of the
// uint64 residues (same 8 bytes per value), so no conversion or full
// reduction is spent on it.
#include "fesc_internal.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;
constexpr int kPadRow = 17;  // LDS: one pad word per 16 values

__device__ __forceinline__ uint32_t pad16(uint32_t k) { return k + (k >> 4); }

template <int H>
struct Log2H { static constexpr int v = H == 8 ? 3 : H == 4 ? 2 : H == 2 ? 1 : 0; };

// One forward stage on the 16-value tile x: pairs (r, r + H), r & H == 0.
// Value r sits at global index jb + (r << js_log).
template <int H>
__device__ __forceinline__ void ct_stage(double (&x)[16], const double2* __restrict__ tw,
                                         uint32_t n, uint32_t jb, uint32_t js_log, double q,
                                         double qinv) {
  const uint32_t sh = Log2H<H>::v + js_log + 1;
#pragma unroll
  for (int g = 0; g < 16; g += 2 * H) {
    const double2 w = tw[(n + jb + ((uint32_t)g << js_log)) >> sh];
#pragma unroll
    for (int r = g; r < g + H; ++r) {
      double u = red_bal(x[r], q, qinv);
      double v = mm_shoup(x[r + H], w.x, w.y, q);
      x[r] = u + v;
      x[r + H] = u - v;
    }
  }
}

template <int H>
__device__ __forceinline__ void gs_stage(double (&x)[16], const double2* __restrict__ tw,
                                         uint32_t n, uint32_t jb, uint32_t js_log, double q,
                                         double qinv) {
  const uint32_t sh = Log2H<H>::v + js_log + 1;
#pragma unroll
  for (int g = 0; g < 16; g += 2 * H) {
    const double2 w = tw[(n + jb + ((uint32_t)g << js_log)) >> sh];
#pragma unroll
    for (int r = g; r < g + H; ++r) {
      double u = x[r], v = x[r + H];
      x[r] = red_bal(u + v, q, qinv);
      x[r + H] = mm_shoup(u - v, w.x, w.y, q);
    }
  }
}

// Forward stages with register distances 2^(nst-1), ..., 1.
template <int NST>
__device__ __forceinline__ void ct_tail(double (&x)[16], const double2* tw, uint32_t n,
                                        uint32_t jb, uint32_t js_log, double q, double qinv) {
  if constexpr (NST >= 4) ct_stage<8>(x, tw, n, jb, js_log, q, qinv);
  if constexpr (NST >= 3) ct_stage<4>(x, tw, n, jb, js_log, q, qinv);
  if constexpr (NST >= 2) ct_stage<2>(x, tw, n, jb, js_log, q, qinv);
  if constexpr (NST >= 1) ct_stage<1>(x, tw, n, jb, js_log, q, qinv);
}

// Inverse stages with register distances 1, ..., 2^(nst-1).
template <int NST>
__device__ __forceinline__ void gs_head(double (&x)[16], const double2* tw, uint32_t n,
                                        uint32_t jb, uint32_t js_log, double q, double qinv) {
  if constexpr (NST >= 1) gs_stage<1>(x, tw, n, jb, js_log, q, qinv);
  if constexpr (NST >= 2) gs_stage<2>(x, tw, n, jb, js_log, q, qinv);
  if constexpr (NST >= 3) gs_stage<4>(x, tw, n, jb, js_log, q, qinv);
  if constexpr (NST >= 4) gs_stage<8>(x, tw, n, jb, js_log, q, qinv);
}

}  // namespace

// Row selection of a batched transform launch.  blockIdx.y = batch index b,
// blockIdx.z = limb index i (the batch varies fastest between workgroups, so
// the twiddle table of one prime stays resident in L2 across the batch).
// Limb i < split uses prime prime0 + i, limb i >= split prime1 + (i - split).
// If skip_alpha != 0, limbs [d*skip_alpha, min((d+1)*skip_alpha, skip_limit))
// of batch element b, d = b mod skip_mod, are left untouched (the own-digit
// rows of digit d in a batch of ModUp outputs).
__device__ __forceinline__ uint64_t* RowSel::row() const {
  return base + (size_t)blockIdx.y * batch_stride + (size_t)blockIdx.z * limb_stride;
}
__device__ __forceinline__ uint32_t RowSel::prime() const {
  const uint32_t i = blockIdx.z;
  return i < split ? prime0 + i : prime1 + (i - split);
}
__device__ __forceinline__ bool RowSel::skip() const {
  if (!skip_alpha) return false;
  const uint32_t lo = (blockIdx.y % skip_mod) * skip_alpha;
  const uint32_t hi = min(lo + skip_alpha, skip_limit);
  return blockIdx.z >= lo && blockIdx.z < hi;
}

namespace {

// ---------------------------------------------------------------- forward

// Outer pass, M = 2^LOGM point columns at stride 256.  TPS threads per column,
// SPW columns per workgroup.  Reads uint64 residues, writes fp64.
template <int LOGM>
__global__ __launch_bounds__(kThreads) void k_fwd_outer(RowSel rs, uint32_t log_n,
                                                        const PrimeK* __restrict__ pk,
                                                        const double2* __restrict__ twf) {
  constexpr int TPS = (1 << LOGM) / 16;
  constexpr int SPW = kThreads / TPS;
  __shared__ double lds[SPW * TPS * 16 + SPW * TPS];
  if (rs.skip()) return;
  const uint32_t n = 1u << log_n;
  const uint32_t prime = rs.prime();
  const double q = pk[prime].q, qinv = pk[prime].qinv;
  const double2* tw = twf + (size_t)prime * n;
  uint64_t* row = rs.row();
  const uint32_t tid = threadIdx.x, sp = tid % SPW, k0 = tid / SPW;
  const uint32_t c = blockIdx.x * SPW + sp;
  double x[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = u2d(row[c + 256u * (k0 + TPS * r)]);
  // first four stages: value r is at global index c + 256 * (k0 + TPS * r)
  ct_tail<4>(x, tw, n, c + 256u * k0, 8 + (LOGM - 4), q, qinv);
  double* rowd = reinterpret_cast<double*>(row);
  if constexpr (LOGM > 4) {
    double* my = lds + sp * (TPS * kPadRow);
#pragma unroll
    for (int r = 0; r < 16; ++r) my[pad16(k0 + TPS * r)] = x[r];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = my[pad16(16 * k0 + r)];
    ct_tail<LOGM - 4>(x, tw, n, c + 256u * 16u * k0, 8, q, qinv);
#pragma unroll
    for (int r = 0; r < 16; ++r) rowd[c + 256u * (16 * k0 + r)] = x[r];
  } else {
#pragma unroll
    for (int r = 0; r < 16; ++r) rowd[c + 256u * r] = x[r];
  }
}

// Inner-pass twiddles.  For half-distance t = 2^lt inside block `blk` the
// butterfly group r (< 128/t) uses psi_rev[N/2t + blk*128/t + r]; the two
// parts of that index have disjoint bits, so the twiddle factors as
//     F_lt * psi_rev[r],   F_lt = psi_rev[N/2t + blk*128/t],
// i.e. eight per-block values and the first 128 table entries (kept in LDS).
// Each twiddle costs one modular product instead of a global load.
__device__ __forceinline__ double2 tw_prod(double F, const double2* small, uint32_t r, double q,
                                           double qinv) {
  const double2 c = small[r];
  const double w = mm_shoup(F, c.x, c.y, q);  // |w| < q
  return double2{w, w * qinv};
}

// Forward stage with register distance H on a tile whose group g has twiddle
// index r = rbase + g / 2H.
template <int H, bool RB0>
__device__ __forceinline__ void ct_stage_f(double (&x)[16], double F, const double2* small,
                                           uint32_t rbase, double q, double qinv) {
#pragma unroll
  for (int g = 0; g < 16; g += 2 * H) {
    const double2 w = (RB0 && g == 0) ? double2{F, F * qinv}
                                      : tw_prod(F, small, rbase + g / (2 * H), q, qinv);
#pragma unroll
    for (int r = g; r < g + H; ++r) {
      double u = red_bal(x[r], q, qinv);
      double v = mm_shoup(x[r + H], w.x, w.y, q);
      x[r] = u + v;
      x[r + H] = u - v;
    }
  }
}

template <int H, bool RB0>
__device__ __forceinline__ void gs_stage_f(double (&x)[16], double F, const double2* small,
                                           uint32_t rbase, double q, double qinv) {
#pragma unroll
  for (int g = 0; g < 16; g += 2 * H) {
    const double2 w = (RB0 && g == 0) ? double2{F, F * qinv}
                                      : tw_prod(F, small, rbase + g / (2 * H), q, qinv);
#pragma unroll
    for (int r = g; r < g + H; ++r) {
      double u = x[r], v = x[r + H];
      x[r] = red_bal(u + v, q, qinv);
      x[r + H] = mm_shoup(u - v, w.x, w.y, q);
    }
  }
}

// Inner pass: 256-point blocks, 16 threads per block, 16 blocks per workgroup.
// Reads fp64 (outer-pass output), writes canonical uint64 residues.
__global__ __launch_bounds__(kThreads) void k_fwd_inner(RowSel rs, uint32_t log_n,
                                                        const PrimeK* __restrict__ pk,
                                                        const double2* __restrict__ twf) {
  __shared__ double lds[16 * 16 * kPadRow];
  __shared__ double2 small[128];
  if (rs.skip()) return;
  const uint32_t n = 1u << log_n;
  const uint32_t prime = rs.prime();
  const double q = pk[prime].q, qinv = pk[prime].qinv;
  const double2* tw = twf + (size_t)prime * n;
  uint64_t* row = rs.row();
  const uint32_t tid = threadIdx.x, sp = tid >> 4, s0 = tid & 15;
  const uint32_t base = (blockIdx.x * 16 + sp) * 256;
  if (tid < 128) small[tid] = tw[tid];
  double F[8];
#pragma unroll
  for (int lt = 0; lt < 8; ++lt) F[lt] = tw[(n + base) >> (lt + 1)].x;
  const double* src = reinterpret_cast<const double*>(row) + base;
  double x[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = src[s0 + 16 * r];
  __syncthreads();
  // t = 128, 64, 32, 16: value r at s0 + 16r, group index g / 2H
  ct_stage_f<8, true>(x, F[7], small, 0, q, qinv);
  ct_stage_f<4, true>(x, F[6], small, 0, q, qinv);
  ct_stage_f<2, true>(x, F[5], small, 0, q, qinv);
  ct_stage_f<1, true>(x, F[4], small, 0, q, qinv);
  double* my = lds + sp * (16 * kPadRow);
#pragma unroll
  for (int r = 0; r < 16; ++r) my[pad16(s0 + 16 * r)] = x[r];
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = my[pad16(16 * s0 + r)];
  // t = 8, 4, 2, 1: value r at 16 s0 + r, group index 8 s0 / H + g / 2H
  ct_stage_f<8, false>(x, F[3], small, s0, q, qinv);
  ct_stage_f<4, false>(x, F[2], small, 2 * s0, q, qinv);
  ct_stage_f<2, false>(x, F[1], small, 4 * s0, q, qinv);
  ct_stage_f<1, false>(x, F[0], small, 8 * s0, q, qinv);
  ulonglong2* dst = reinterpret_cast<ulonglong2*>(row + base + 16 * s0);
#pragma unroll
  for (int r = 0; r < 16; r += 2) {
    ulonglong2 v;
    v.x = d2u(red_full(x[r], q, qinv));
    v.y = d2u(red_full(x[r + 1], q, qinv));
    dst[r / 2] = v;
  }
}

// ---------------------------------------------------------------- inverse

// Inner pass first: reads uint64 residues, writes fp64.
__global__ __launch_bounds__(kThreads) void k_inv_inner(RowSel rs, uint32_t log_n,
                                                        const PrimeK* __restrict__ pk,
                                                        const double2* __restrict__ twi) {
  __shared__ double lds[16 * 16 * kPadRow];
  __shared__ double2 small[128];
  if (rs.skip()) return;
  const uint32_t n = 1u << log_n;
  const uint32_t prime = rs.prime();
  const double q = pk[prime].q, qinv = pk[prime].qinv;
  const double2* tw = twi + (size_t)prime * n;
  uint64_t* row = rs.row();
  const uint32_t tid = threadIdx.x, sp = tid >> 4, s0 = tid & 15;
  const uint32_t base = (blockIdx.x * 16 + sp) * 256;
  if (tid < 128) small[tid] = tw[tid];
  double F[8];
#pragma unroll
  for (int lt = 0; lt < 8; ++lt) F[lt] = tw[(n + base) >> (lt + 1)].x;
  const ulonglong2* src = reinterpret_cast<const ulonglong2*>(row + base + 16 * s0);
  double x[16];
#pragma unroll
  for (int r = 0; r < 16; r += 2) {
    ulonglong2 v = src[r / 2];
    x[r] = u2d(v.x);
    x[r + 1] = u2d(v.y);
  }
  __syncthreads();
  // t = 1, 2, 4, 8 on 16 consecutive values
  gs_stage_f<1, false>(x, F[0], small, 8 * s0, q, qinv);
  gs_stage_f<2, false>(x, F[1], small, 4 * s0, q, qinv);
  gs_stage_f<4, false>(x, F[2], small, 2 * s0, q, qinv);
  gs_stage_f<8, false>(x, F[3], small, s0, q, qinv);
  double* my = lds + sp * (16 * kPadRow);
#pragma unroll
  for (int r = 0; r < 16; ++r) my[pad16(16 * s0 + r)] = x[r];
  __syncthreads();
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = my[pad16(s0 + 16 * r)];
  // t = 16, 32, 64, 128 on values s0 + 16 r
  gs_stage_f<1, true>(x, F[4], small, 0, q, qinv);
  gs_stage_f<2, true>(x, F[5], small, 0, q, qinv);
  gs_stage_f<4, true>(x, F[6], small, 0, q, qinv);
  gs_stage_f<8, true>(x, F[7], small, 0, q, qinv);
  double* dst = reinterpret_cast<double*>(row) + base;
#pragma unroll
  for (int r = 0; r < 16; ++r) dst[s0 + 16 * r] = x[r];
}

// Outer pass last: reads fp64, scales by N^-1, writes canonical uint64.
template <int LOGM>
__global__ __launch_bounds__(kThreads) void k_inv_outer(RowSel rs, uint32_t log_n,
                                                        const PrimeK* __restrict__ pk,
                                                        const double2* __restrict__ twi) {
  constexpr int TPS = (1 << LOGM) / 16;
  constexpr int SPW = kThreads / TPS;
  __shared__ double lds[SPW * TPS * 16 + SPW * TPS];
  if (rs.skip()) return;
  const uint32_t n = 1u << log_n;
  const uint32_t prime = rs.prime();
  const PrimeK P = pk[prime];
  const double2* tw = twi + (size_t)prime * n;
  uint64_t* row = rs.row();
  const double* rowd = reinterpret_cast<const double*>(row);
  const uint32_t tid = threadIdx.x, sp = tid % SPW, k0 = tid / SPW;
  const uint32_t c = blockIdx.x * SPW + sp;
  double x[16];
  if constexpr (LOGM > 4) {
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = rowd[c + 256u * (16 * k0 + r)];
    gs_head<LOGM - 4>(x, tw, n, c + 256u * 16u * k0, 8, P.q, P.qinv);
    double* my = lds + sp * (TPS * kPadRow);
#pragma unroll
    for (int r = 0; r < 16; ++r) my[pad16(16 * k0 + r)] = x[r];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = my[pad16(k0 + TPS * r)];
  } else {
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] = rowd[c + 256u * r];
  }
  gs_head<4>(x, tw, n, c + 256u * k0, 8 + (LOGM - 4), P.q, P.qinv);
#pragma unroll
  for (int r = 0; r < 16; ++r)
    row[c + 256u * (k0 + TPS * r)] =
        d2u(red_full(mm_shoup(x[r], P.ninv, P.ninvp, P.q), P.q, P.qinv));
}

template <int LOGM>
void launch_outer(bool inverse, dim3 grid, hipStream_t s, RowSel rs, uint32_t log_n,
                  const PrimeK* pk, const double2* tw) {
  grid.x = (1u << LOGM) / 16;  // 256 / SPW
  if (inverse)
    hipLaunchKernelGGL(k_inv_outer<LOGM>, grid, dim3(kThreads), 0, s, rs, log_n, pk, tw);
  else
    hipLaunchKernelGGL(k_fwd_outer<LOGM>, grid, dim3(kThreads), 0, s, rs, log_n, pk, tw);
}

}  // namespace

// Both passes of one batch chunk.
static hipError_t launch_chunk(const Context* c, const RowSel& rs, uint32_t batch, uint32_t limbs,
                               bool inverse, hipStream_t s) {
  const uint32_t log_n = c->log_n;
  const double2* tw = inverse ? c->d_tw_inv : c->d_tw_fwd;
  dim3 inner(c->n / 4096, batch, limbs);
  dim3 outer(1, batch, limbs);
  if (inverse)
    hipLaunchKernelGGL(k_inv_inner, inner, dim3(kThreads), 0, s, rs, log_n, c->d_pk, tw);
  switch (log_n) {
    case 12: launch_outer<4>(inverse, outer, s, rs, log_n, c->d_pk, tw); break;
    case 13: launch_outer<5>(inverse, outer, s, rs, log_n, c->d_pk, tw); break;
    case 14: launch_outer<6>(inverse, outer, s, rs, log_n, c->d_pk, tw); break;
    case 15: launch_outer<7>(inverse, outer, s, rs, log_n, c->d_pk, tw); break;
    case 16: launch_outer<8>(inverse, outer, s, rs, log_n, c->d_pk, tw); break;
    default: return hipErrorInvalidValue;
  }
  if (!inverse)
    hipLaunchKernelGGL(k_fwd_inner, inner, dim3(kThreads), 0, s, rs, log_n, c->d_pk, tw);
  return hipGetLastError();
}

// (Splitting a large batch into cache-sized chunks, so that the second pass
// would read the first pass's output back from the 256 MB Infinity Cache,
// measured slower on MI355X than one launch per pass over the whole batch.)
hipError_t launch_ntt_rows(const Context* c, const RowSel& rs, uint32_t batch, uint32_t limbs,
                           bool inverse, hipStream_t s) {
  return launch_chunk(c, rs, batch, limbs, inverse, s);
}

hipError_t launch_ntt(const Context* c, uint64_t* d, uint32_t batch, size_t batch_stride,
                      uint32_t limbs, size_t limb_stride, uint32_t prime0, bool inverse,
                      hipStream_t s) {
  RowSel rs{d, batch_stride, limb_stride, prime0, limbs, 0, 0, 0};
  return launch_ntt_rows(c, rs, batch, limbs, inverse, s);
}

}  // namespace fesc
