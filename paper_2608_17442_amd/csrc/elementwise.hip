// Limb-wise modular kernels: Hadamard multiply-accumulate and the ciphertext
// elementwise operations.  Each thread owns two adjacent coefficients of one
// row (one 16-byte load per operand), rows map to blockIdx.y.
#include "fesc_internal.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;

typedef unsigned long long u64x2 __attribute__((ext_vector_type(2)));

// V coefficients per thread, as V/2 16-byte loads per operand and pair; load
// i of thread t covers coefficients 2(i kThreads + t) and the next, so each load
// instruction of a wave reads one contiguous 1 KiB run.

template <int V>
__global__ __launch_bounds__(kThreads) void k_mac(const uint64_t* __restrict__ a,
                                                  const uint64_t* __restrict__ b,
                                                  uint64_t* __restrict__ out, uint32_t pairs,
                                                  size_t pair_stride, uint32_t n,
                                                  uint32_t prime0,
                                                  const PrimeK* __restrict__ pk) {
  const uint32_t limb = blockIdx.y;
  const uint32_t k = blockIdx.x * kThreads * V + 2 * threadIdx.x;
  if (k >= n) return;
  const double q = pk[prime0 + limb].q, qinv = pk[prime0 + limb].qinv;
  const size_t off = (size_t)limb * n + k;
  double acc[V];
#pragma unroll
  for (int v = 0; v < V; ++v) acc[v] = 0.0;
#pragma unroll 4
  for (uint32_t j = 0; j < pairs; ++j) {
    // every operand is read once: streaming (non-temporal) loads
    const u64x2* pa = reinterpret_cast<const u64x2*>(a + j * pair_stride + off);
    const u64x2* pb = reinterpret_cast<const u64x2*>(b + j * pair_stride + off);
#pragma unroll
    for (int v = 0; v < V; v += 2) {
      const u64x2 va = __builtin_nontemporal_load(pa + v / 2 * kThreads);
      const u64x2 vb = __builtin_nontemporal_load(pb + v / 2 * kThreads);
      acc[v] = red_bal(acc[v] + mm_var(u2d(va.x), u2d(vb.x), q, qinv), q, qinv);
      acc[v + 1] = red_bal(acc[v + 1] + mm_var(u2d(va.y), u2d(vb.y), q, qinv), q, qinv);
    }
  }
  ulonglong2* po = reinterpret_cast<ulonglong2*>(out + off);
#pragma unroll
  for (int v = 0; v < V; v += 2) {
    ulonglong2 r;
    r.x = to_res(acc[v], q, qinv);
    r.y = to_res(acc[v + 1], q, qinv);
    po[v / 2 * kThreads] = r;
  }
}

}  // namespace

hipError_t launch_mac(const Context* c, const uint64_t* a, const uint64_t* b, uint64_t* out,
                      uint32_t pairs, size_t pair_stride, uint32_t limbs, uint32_t prime0,
                      hipStream_t s) {
  // eight coefficients per thread: the launch fits on the device in one round
  // (768 workgroups at 24 limbs x 2^16) with four 16-byte loads per operand
  // and pair in flight; two per thread ran in 1.5 rounds at 4.9 TB/s, eight
  // stream at 5.8 TB/s.  N >= 4096 is a multiple of 8 x 256.
  constexpr int V = 8;
  dim3 grid((c->n / V + kThreads - 1) / kThreads, limbs);
  hipLaunchKernelGGL(k_mac<V>, grid, dim3(kThreads), 0, s, a, b, out, pairs, pair_stride, c->n,
                     prime0, c->d_pk);
  return hipGetLastError();
}

}  // namespace fesc
