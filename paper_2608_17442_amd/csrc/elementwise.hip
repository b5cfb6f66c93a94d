// Limb-wise modular kernels: Hadamard multiply-accumulate and the ciphertext
// elementwise operations.  Each thread owns two adjacent coefficients of one
// row (one 16-byte load per operand), rows map to blockIdx.y.
#include "fesc_internal.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void k_mac(const uint64_t* __restrict__ a,
                                                  const uint64_t* __restrict__ b,
                                                  uint64_t* __restrict__ out, uint32_t pairs,
                                                  size_t pair_stride, uint32_t n,
                                                  uint32_t prime0,
                                                  const PrimeK* __restrict__ pk) {
  const uint32_t limb = blockIdx.y;
  const uint32_t k = (blockIdx.x * kThreads + threadIdx.x) * 2;
  if (k >= n) return;
  const double q = pk[prime0 + limb].q, qinv = pk[prime0 + limb].qinv;
  const size_t off = (size_t)limb * n + k;
  double acc0 = 0.0, acc1 = 0.0;
#pragma unroll 4
  for (uint32_t j = 0; j < pairs; ++j) {
    const ulonglong2 va = *reinterpret_cast<const ulonglong2*>(a + j * pair_stride + off);
    const ulonglong2 vb = *reinterpret_cast<const ulonglong2*>(b + j * pair_stride + off);
    acc0 = red_bal(acc0 + mm_var(u2d(va.x), u2d(vb.x), q, qinv), q, qinv);
    acc1 = red_bal(acc1 + mm_var(u2d(va.y), u2d(vb.y), q, qinv), q, qinv);
  }
  ulonglong2 r;
  r.x = to_res(acc0, q, qinv);
  r.y = to_res(acc1, q, qinv);
  *reinterpret_cast<ulonglong2*>(out + off) = r;
}

}  // namespace

hipError_t launch_mac(const Context* c, const uint64_t* a, const uint64_t* b, uint64_t* out,
                      uint32_t pairs, size_t pair_stride, uint32_t limbs, uint32_t prime0,
                      hipStream_t s) {
  dim3 grid((c->n / 2 + kThreads - 1) / kThreads, limbs);
  hipLaunchKernelGGL(k_mac, grid, dim3(kThreads), 0, s, a, b, out, pairs, pair_stride, c->n,
                     prime0, c->d_pk);
  return hipGetLastError();
}

}  // namespace fesc
