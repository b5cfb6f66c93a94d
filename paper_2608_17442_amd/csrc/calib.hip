// VALU calibration: the register-resident arithmetic of the NTT stages and of
// the modular multiply-accumulate sums (basis conversion, key inner product),
// run on every compute unit with no memory traffic.  The measured rates are
// the compute roof against which the transforms and key switching are
// reported; they are not part of the method.
#include <cmath>

#include "butterfly.hpp"
#include "fesc_internal.hpp"
#include "seedkey.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;

// The 15 twiddles of one radix-16 step (1 + 2 + 4 + 8 groups), uniform.
struct Tw15 {
  double2 w[15];
};
template <int OFF>
struct TwArg {
  const Tw15* t;
  __device__ __forceinline__ double2 operator()(int gi) const { return t->w[OFF + gi]; }
};

// One radix-16 step (four radix-2 stages, 32 butterflies per thread) per
// iteration, forward (CT) or inverse (GS), with the kernels' lazy reduction
// pattern.
template <bool INV>
__global__ __launch_bounds__(kThreads) void k_calib_bfly(Tw15 tw, double q, double qinv,
                                                         uint32_t iters, double* out) {
  const uint32_t t = blockIdx.x * kThreads + threadIdx.x;
  double x[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = (double)((t * 16u + r) % 1000003u);
  for (uint32_t i = 0; i < iters; ++i) {
    if constexpr (INV) {
      gs_st<1, true>(x, TwArg<7>{&tw}, q, qinv);
      gs_st<2, false>(x, TwArg<3>{&tw}, q, qinv);
      gs_st<4, true>(x, TwArg<1>{&tw}, q, qinv);
      gs_st<8, false>(x, TwArg<0>{&tw}, q, qinv);
    } else {
      ct_st<8, true>(x, TwArg<0>{&tw}, q, qinv);
      ct_st<4, false>(x, TwArg<1>{&tw}, q, qinv);
      ct_st<2, true>(x, TwArg<3>{&tw}, q, qinv);
      ct_st<1, false>(x, TwArg<7>{&tw}, q, qinv);
    }
  }
  double s = 0.0;
#pragma unroll
  for (int r = 0; r < 16; ++r) s += x[r];
  out[t] = s;
}

// Eight independent sums of products x_j * y_j mod q (per-lane operands),
// reduced after every four terms as the basis-conversion and inner-product
// kernels do: 8 MACs per thread per iteration.
__global__ __launch_bounds__(kThreads) void k_calib_mac(double q, double qinv, uint32_t iters,
                                                        double* out) {
  const uint32_t t = blockIdx.x * kThreads + threadIdx.x;
  double x[8], y[8], acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    x[j] = (double)((t * 8u + j) % 1000003u);
    y[j] = (double)((t * 131u + 7u * j) % 999983u);
    acc[j] = 0.0;
  }
  for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] += mm_var(x[j], y[j], q, qinv);
    if ((i & 3) == 3) {
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = red_bal(acc[j], q, qinv);
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = acc[j];  // carry a dependency into the next term
  }
  double s = 0.0;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += acc[j];
  out[t] = s;
}

// The residue product alone, in the two forms considered for the VALU:
// eight independent chains x <- x w mod q per thread and iteration.
//   fp64 (the library's): h = x w, l = fma(x, w, -h), c = rint(x w'),
//     x = fma(-c, q, h) + l  (w' = w / q in fp64);
//   u64 (Shoup's integer form): c = hi64(x w'), x = x w - c q  (mod 2^64,
//     w' = floor(w 2^64 / q); the result stays below 2q).
__global__ __launch_bounds__(kThreads) void k_calib_modmul_f64(double q, double w, double wp,
                                                               uint32_t iters, double* out) {
  const uint32_t t = blockIdx.x * kThreads + threadIdx.x;
  double x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = (double)((t * 8u + j) % 1000003u);
  for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = mm_shoup(x[j], w, wp, q);
  }
  double s = 0.0;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += x[j];
  out[t] = s;
}

__global__ __launch_bounds__(kThreads) void k_calib_modmul_u64(uint64_t q, uint64_t w,
                                                               uint64_t wp, uint32_t iters,
                                                               double* out) {
  const uint32_t t = blockIdx.x * kThreads + threadIdx.x;
  uint64_t x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = (uint64_t)((t * 8u + j) % 1000003u);
  for (uint32_t i = 0; i < iters; ++i) {
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = x[j] * w - __umul64hi(x[j], wp) * q;
  }
  uint64_t s = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += x[j];
  out[t] = (double)(s & 0xFFFFFFFFull);
}

// The generator of seed-expanded keys: two independent chains of
// Philox4x64-10 blocks per thread, each block's output the next counter.
__global__ __launch_bounds__(kThreads) void k_calib_philox(uint64_t k0, uint64_t k1,
                                                           uint32_t iters, double* out) {
  const uint32_t t = blockIdx.x * kThreads + threadIdx.x;
  uint64_t x[4] = {t, 1, 2, 3}, y[4] = {t, 5, 6, 7};
  for (uint32_t i = 0; i < iters; ++i) {
    philox4x64_10(x, k0, k1);
    philox4x64_10(y, k1, k0);
  }
  out[t] = (double)((x[0] ^ x[1] ^ x[2] ^ x[3] ^ y[0] ^ y[1] ^ y[2] ^ y[3]) & 0xFFFFFFFFull);
}

// Streaming HBM ceilings: every 16-byte word of `src` read once (grid-
// stride; an XOR per thread keeps the loads live), or copied to `dst`.
__global__ __launch_bounds__(kThreads) void k_calib_read(const ulonglong2* __restrict__ src,
                                                         size_t words2, uint64_t* __restrict__ out) {
  const size_t t = (size_t)blockIdx.x * kThreads + threadIdx.x, nt = (size_t)gridDim.x * kThreads;
  uint64_t x = 0;
  typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));
  for (size_t i = t; i < words2; i += nt) {
    // streaming (non-temporal) loads, as the read-once kernels use
    const u64x2 v = __builtin_nontemporal_load(reinterpret_cast<const u64x2*>(src) + i);
    x ^= v.x ^ v.y;
  }
  out[t] = x;
}

__global__ __launch_bounds__(kThreads) void k_calib_copy(const ulonglong2* __restrict__ src,
                                                         ulonglong2* __restrict__ dst,
                                                         size_t words2) {
  const size_t t = (size_t)blockIdx.x * kThreads + threadIdx.x, nt = (size_t)gridDim.x * kThreads;
  for (size_t i = t; i < words2; i += nt) dst[i] = src[i];
}

}  // namespace

int calib_hbm(Context* c, int kind, size_t bytes, double* rate, hipStream_t s) {
  if ((kind != FESC_CALIB_HBM_READ && kind != FESC_CALIB_HBM_COPY) || bytes < ((size_t)1 << 20) ||
      bytes > ((size_t)64 << 30) || bytes % 16)
    return fail(FESC_ERR_ARG, "bad HBM calibration arguments");
  int cus = 0;
  if (int rc = hip_check(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount,
                                               c->device), "hipDeviceGetAttribute"))
    return rc;
  // grids from a sweep on MI355X: 8 workgroups per CU for reads, 64 for copies
  const uint32_t blocks = (uint32_t)cus * (kind == FESC_CALIB_HBM_READ ? 8 : 64);
  void *src = nullptr, *dst = nullptr;
  const size_t out_bytes = (size_t)blocks * kThreads * 8;
  if (hipMalloc(&src, bytes) != hipSuccess ||
      hipMalloc(&dst, kind == FESC_CALIB_HBM_COPY ? bytes : out_bytes) != hipSuccess) {
    (void)hipFree(src);
    return fail(FESC_ERR_OOM, "HBM calibration buffers");
  }
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = hip_check(hipMemsetAsync(src, 1, bytes, s), "hipMemsetAsync");
  if (!rc) rc = hip_check(hipEventCreate(&e0), "hipEventCreate");
  if (!rc) rc = hip_check(hipEventCreate(&e1), "hipEventCreate");
  const size_t w2 = bytes / 16;
  auto launch = [&]() {
    if (kind == FESC_CALIB_HBM_READ)
      hipLaunchKernelGGL(k_calib_read, dim3(blocks), dim3(kThreads), 0, s,
                         static_cast<const ulonglong2*>(src), w2, static_cast<uint64_t*>(dst));
    else
      hipLaunchKernelGGL(k_calib_copy, dim3(blocks), dim3(kThreads), 0, s,
                         static_cast<const ulonglong2*>(src), static_cast<ulonglong2*>(dst), w2);
  };
  float ms = 0.f;
  if (!rc) {
    launch();  // warm-up
    rc = hip_check(hipGetLastError(), "HBM calibration launch");
  }
  if (!rc) rc = hip_check(hipEventRecord(e0, s), "hipEventRecord");
  if (!rc) {
    launch();
    rc = hip_check(hipGetLastError(), "HBM calibration launch");
  }
  if (!rc) rc = hip_check(hipEventRecord(e1, s), "hipEventRecord");
  if (!rc) rc = hip_check(hipEventSynchronize(e1), "hipEventSynchronize");
  if (!rc) rc = hip_check(hipEventElapsedTime(&ms, e0, e1), "hipEventElapsedTime");
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  (void)hipStreamSynchronize(s);
  (void)hipFree(src);
  (void)hipFree(dst);
  if (rc) return rc;
  *rate = (double)bytes * (kind == FESC_CALIB_HBM_COPY ? 2.0 : 1.0) / (ms * 1e-3);
  return FESC_OK;
}

int calib_valu(Context* c, int kind, uint32_t iters, double* rate, hipStream_t s) {
  if (kind < FESC_CALIB_CT || kind > FESC_CALIB_PHILOX || iters == 0 || iters > (1u << 20))
    return fail(FESC_ERR_ARG, "bad calibration arguments");
  int cus = 0;
  if (int rc = hip_check(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount,
                                               c->device), "hipDeviceGetAttribute"))
    return rc;
  const uint32_t blocks = (uint32_t)cus * 8;
  int err;
  double* out = static_cast<double*>(scratch_get(c, sizeof(double) * blocks * kThreads, &err));
  if (!out) return err;
  const double q = (double)c->primes[0], qinv = 1.0 / q;
  Tw15 tw;
  for (int i = 0; i < 15; ++i) {
    const double w = std::floor(q / (3.0 + i));
    tw.w[i] = double2{w, w / q};
  }
  hipEvent_t e0, e1;
  if (int rc = hip_check(hipEventCreate(&e0), "hipEventCreate")) return rc;
  if (int rc = hip_check(hipEventCreate(&e1), "hipEventCreate")) {
    (void)hipEventDestroy(e0);
    return rc;
  }
  // the product's operands for the modmul probes: w < q, w' its Shoup constant
  const uint64_t qu = c->primes[0], wu = qu / 3 + 12345;
  const uint64_t wpu = (uint64_t)(((unsigned __int128)wu << 64) / qu);
  auto launch = [&]() {
    if (kind == FESC_CALIB_PHILOX)
      hipLaunchKernelGGL(k_calib_philox, dim3(blocks), dim3(kThreads), 0, s,
                         0x0123456789ABCDEFull, 0xFEDCBA9876543210ull, iters, out);
    else if (kind == FESC_CALIB_MODMUL_F64)
      hipLaunchKernelGGL(k_calib_modmul_f64, dim3(blocks), dim3(kThreads), 0, s, q, (double)wu,
                         (double)wu / q, iters, out);
    else if (kind == FESC_CALIB_MODMUL_U64)
      hipLaunchKernelGGL(k_calib_modmul_u64, dim3(blocks), dim3(kThreads), 0, s, qu, wu, wpu,
                         iters, out);
    else if (kind == FESC_CALIB_CT)
      hipLaunchKernelGGL(k_calib_bfly<false>, dim3(blocks), dim3(kThreads), 0, s, tw, q, qinv,
                         iters, out);
    else if (kind == FESC_CALIB_GS)
      hipLaunchKernelGGL(k_calib_bfly<true>, dim3(blocks), dim3(kThreads), 0, s, tw, q, qinv,
                         iters, out);
    else
      hipLaunchKernelGGL(k_calib_mac, dim3(blocks), dim3(kThreads), 0, s, q, qinv, iters, out);
  };
  launch();  // warm-up
  int rc = hip_check(hipGetLastError(), "calibration launch");
  if (!rc) rc = hip_check(hipEventRecord(e0, s), "hipEventRecord");
  if (!rc) launch();
  if (!rc) rc = hip_check(hipGetLastError(), "calibration launch");
  if (!rc) rc = hip_check(hipEventRecord(e1, s), "hipEventRecord");
  if (!rc) rc = hip_check(hipEventSynchronize(e1), "hipEventSynchronize");
  float ms = 0.f;
  if (!rc) rc = hip_check(hipEventElapsedTime(&ms, e0, e1), "hipEventElapsedTime");
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (rc) return rc;
  const double per_thread =
      (kind == FESC_CALIB_CT || kind == FESC_CALIB_GS) ? 32.0 * iters
      : kind == FESC_CALIB_PHILOX                      ? 2.0 * iters
                                                       : 8.0 * iters;
  *rate = (double)blocks * kThreads * per_thread / (ms * 1e-3);
  return FESC_OK;
}

}  // namespace fesc
