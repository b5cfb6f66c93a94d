// CKKS encoding on the device: slot vectors -> evaluation-form plaintexts
// (offline plaintext preparation: the projection's diagonals, masks).
//
// Slot j is the evaluation at zeta^(5^j mod 2N), zeta = exp(i pi / N).  With
// y[(e_j - 1)/2] = z_j and y[N - 1 - (e_j - 1)/2] = conj(z_j), e_j = 5^j mod 2N,
// the real plaintext coefficients are
//     m_k = round(Delta / N * Re(zeta^-k Y_k)),   Y = DFT_N(y)   (e^{-2 pi i/N}),
// rounded half away from zero, as the host encoder computes them.  The DFT runs
// in fp64 in two passes over N = M * 4096 (n = 4096 n1 + n2, k = k1 + M k2):
//   pass 1 (columns n2): gather y through the inverse slot table, M-point DFT
//     over n1, twiddle w_N^(n2 k1) -> X[k1][n2];
//   pass 2 (rows k1): 4096-point decimation-in-frequency DFT over n2 in three
//     radix-16 register steps with padded-LDS transposes; the epilogue applies
//     the twist zeta^-k, scales and rounds, storing m in the transform's
//     digit-reversed order;
// then a lift to the RNS limbs (reading m through the bit reversal) and the
// forward NTT of every limb.  Every twiddle is an entry of one table
// T[k] = exp(-i pi k / N), k < 2N.
#include <cmath>

#include "fesc_internal.hpp"
#include "ops.hpp"

namespace fesc {

namespace {

constexpr int kThreads = 256;
constexpr int kRow = 4096;
constexpr int kLdsC = 4096 + 256;  // padded layout of the NTT's inner pass

// padded LDS address of element e = 256 a + 16 c + b: 272 a + 17 c + b
__device__ __forceinline__ uint32_t lds_e(uint32_t e) {
  return 272u * (e >> 8) + 17u * ((e >> 4) & 15u) + (e & 15u);
}

__device__ __forceinline__ double2 cmul(double2 a, double2 b) {
  return double2{a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x};
}

// Pass 1: column n2 = blockIdx.x * 256 + t of plaintext blockIdx.y.
template <int M>
__global__ __launch_bounds__(kThreads) void k_enc_outer(const double2* __restrict__ z,
                                                        const int32_t* __restrict__ inv,
                                                        const double2* __restrict__ T,
                                                        double2* __restrict__ X, uint32_t n) {
  const uint32_t n2 = blockIdx.x * kThreads + threadIdx.x;
  const uint32_t b = blockIdx.y;
  const double2* zb = z + (size_t)b * (n / 2);
  double2 y[M];
#pragma unroll
  for (int n1 = 0; n1 < M; ++n1) {
    const int32_t s = inv[(uint32_t)n1 * kRow + n2];
    const double2 v = zb[s >= 0 ? s : ~s];
    y[n1] = s >= 0 ? v : double2{v.x, -v.y};
  }
  double2* Xb = X + (size_t)b * n;
#pragma unroll
  for (int k1 = 0; k1 < M; ++k1) {
    double2 acc{0.0, 0.0};
#pragma unroll
    for (int n1 = 0; n1 < M; ++n1) {
      // w_M^(n1 k1) = T[(2N / M) (n1 k1 mod M)]
      const double2 w = T[(size_t)(2 * n / M) * ((n1 * k1) % M)];
      const double2 p = cmul(y[n1], w);
      acc.x += p.x;
      acc.y += p.y;
    }
    // twiddle w_N^(n2 k1) = T[2 n2 k1 mod 2N]
    const double2 w = T[(2ull * n2 * k1) % (2ull * n)];
    Xb[(size_t)k1 * kRow + n2] = cmul(acc, w);
  }
}

// One radix-2 DIF stage on register pairs (r, r + H): x_r <- x_r + x_{r+H},
// x_{r+H} <- (x_r - x_{r+H}) T[idx(r)].
template <int H, class IDX>
__device__ __forceinline__ void dif_st(double2 (&x)[16], const double2* __restrict__ T, IDX idx) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    if (r & H) continue;
    const double2 u = x[r], v = x[r + H];
    x[r] = double2{u.x + v.x, u.y + v.y};
    x[r + H] = cmul(double2{u.x - v.x, u.y - v.y}, T[idx(r)]);
  }
}

__device__ __forceinline__ int64_t round_half_away(double v) {
  return (int64_t)(v >= 0.0 ? floor(v + 0.5) : ceil(v - 0.5));
}

// Pass 2: row k1 = blockIdx.x of plaintext blockIdx.y.  Element e of the row
// (its n2) starts at thread e % 256, register e / 256.  A DIF stage of half
// size h pairs e with e + h and multiplies the difference by
// w_{2h}^(e mod h) = T[(e mod h) N / h].
__global__ __launch_bounds__(kThreads) void k_enc_inner(const double2* __restrict__ X,
                                                        const double2* __restrict__ T,
                                                        int64_t* __restrict__ mt, uint32_t n,
                                                        uint32_t M, double scale) {
  __shared__ double lre[kLdsC], lim[kLdsC];
  const uint32_t t = threadIdx.x, k1 = blockIdx.x, b = blockIdx.y;
  const double2* row = X + (size_t)b * n + (size_t)k1 * kRow;
  double2 x[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = row[t + 256 * r];
  // bits 11..8 in registers: h = 256 H, e mod h = t + 256 (r mod H)
  dif_st<8>(x, T, [&](int r) { return (size_t)(t + 256 * (r % 8)) * (n / 2048); });
  dif_st<4>(x, T, [&](int r) { return (size_t)(t + 256 * (r % 4)) * (n / 1024); });
  dif_st<2>(x, T, [&](int r) { return (size_t)(t + 256 * (r % 2)) * (n / 512); });
  dif_st<1>(x, T, [&](int) { return (size_t)t * (n / 256); });
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const uint32_t a = lds_e(t + 256 * r);
    lre[a] = x[r].x;
    lim[a] = x[r].y;
  }
  __syncthreads();
  // bits 7..4: thread t = 16 a + bb holds e = 256 a + 16 r + bb;
  // h = 16 H, e mod h = 16 (r mod H) + bb
  const uint32_t aa = t >> 4, bb = t & 15;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const uint32_t a = lds_e(256 * aa + 16 * r + bb);
    x[r] = double2{lre[a], lim[a]};
  }
  dif_st<8>(x, T, [&](int r) { return (size_t)(16 * (r % 8) + bb) * (n / 128); });
  dif_st<4>(x, T, [&](int r) { return (size_t)(16 * (r % 4) + bb) * (n / 64); });
  dif_st<2>(x, T, [&](int r) { return (size_t)(16 * (r % 2) + bb) * (n / 32); });
  dif_st<1>(x, T, [&](int) { return (size_t)bb * (n / 16); });
  __syncthreads();  // every thread has read its words of the first transpose
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const uint32_t a = lds_e(256 * aa + 16 * r + bb);
    lre[a] = x[r].x;
    lim[a] = x[r].y;
  }
  __syncthreads();
  // bits 3..0: thread t holds e = 16 t + r; h = H, e mod h = r mod H
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const uint32_t a = lds_e(16 * t + r);
    x[r] = double2{lre[a], lim[a]};
  }
  dif_st<8>(x, T, [&](int r) { return (size_t)(r % 8) * (n / 8); });
  dif_st<4>(x, T, [&](int r) { return (size_t)(r % 4) * (n / 4); });
  dif_st<2>(x, T, [&](int r) { return (size_t)(r % 2) * (n / 2); });
  dif_st<1>(x, T, [&](int) { return (size_t)0; });
  // position e holds Y'[bitrev12(e)]: frequency k = k1 + M k2
  const double f = scale / (double)n;
  int64_t* out = mt + (size_t)b * n + (size_t)k1 * kRow;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const uint32_t e = 16 * t + r;
    const uint32_t k2 = __builtin_bitreverse32(e) >> 20;
    const uint32_t k = k1 + M * k2;
    const double2 w = T[k];
    out[e] = round_half_away((x[r].x * w.x - x[r].y * w.y) * f);
  }
}

// Lift: coefficient k (m at row k % M, position bitrev12(k / M)) of plaintext
// blockIdx.z reduced into row i = blockIdx.y of pt[b][rows][N]; row i uses
// prime i below `split`, prime1 + (i - split) from there (the special primes
// of an extended-basis plaintext).
__global__ __launch_bounds__(kThreads) void k_enc_lift(const int64_t* __restrict__ mt,
                                                       uint64_t* __restrict__ pt, uint32_t n,
                                                       uint32_t M, uint32_t level,
                                                       uint32_t split, uint32_t prime1,
                                                       const PrimeK* __restrict__ pk) {
  const uint32_t i = blockIdx.y, b = blockIdx.z;
  const uint32_t k = blockIdx.x * kThreads + threadIdx.x;
  const PrimeK P = pk[i < split ? i : prime1 + (i - split)];
  const uint32_t k1 = k % M, k2 = k / M;
  const int64_t v = mt[(size_t)b * n + (size_t)k1 * kRow + (__builtin_bitreverse32(k2) >> 20)];
  // exact for |v| < 2^63: hi * 2^32 + lo, each part reduced
  const double hi = (double)(int32_t)(v >> 32);
  const double lo = (double)(uint32_t)(v & 0xffffffffu);
  const double two32 = red_full(4294967296.0, P.q, P.qinv);
  const double r = mm_var(red_full(hi, P.q, P.qinv), two32, P.q, P.qinv) + lo;
  pt[((size_t)b * level + i) * n + k] = to_res(r, P.q, P.qinv);
}

}  // namespace

// Encodes `count` slot vectors z[count][N/2] (complex, device) at scale
// `scale` into evaluation-form plaintexts pt[count][rows][N], 32 per round
// through the scratch ciphertext region (X and m of each plaintext in one
// ciphertext slot: 3N words <= 2 L N); rows = level, or level + alpha over
// the extended basis q_0 .. q_{level-1}, p_0 .. p_{alpha-1} (ext).
int op_encode_plain(Context* c, const double2* z, uint32_t count, double scale, uint64_t* pt,
                    uint32_t level, uint64_t* slots, uint32_t nslots, hipStream_t s, bool ext) {
  const uint32_t n = c->n, M = n / kRow;
  const uint32_t rows = ext ? level + c->alpha : level;
  const size_t W = (size_t)2 * c->L * n;
  for (uint32_t b0 = 0; b0 < count; b0 += nslots) {
    const uint32_t m = std::min(nslots, count - b0);
    double2* X = reinterpret_cast<double2*>(slots);   // [m][N] complex
    int64_t* mt = reinterpret_cast<int64_t*>(slots + (size_t)2 * n * m);  // [m][N]
    if ((size_t)3 * n * m > W * nslots) return fail(FESC_ERR_ARG, "encode scratch too small");
    const dim3 g1(kRow / kThreads, m);
    const double2* zb = z + (size_t)b0 * (n / 2);
    switch (M) {
      case 1: k_enc_outer<1><<<g1, kThreads, 0, s>>>(zb, c->d_enc_inv, c->d_enc_tw, X, n); break;
      case 2: k_enc_outer<2><<<g1, kThreads, 0, s>>>(zb, c->d_enc_inv, c->d_enc_tw, X, n); break;
      case 4: k_enc_outer<4><<<g1, kThreads, 0, s>>>(zb, c->d_enc_inv, c->d_enc_tw, X, n); break;
      case 8: k_enc_outer<8><<<g1, kThreads, 0, s>>>(zb, c->d_enc_inv, c->d_enc_tw, X, n); break;
      case 16: k_enc_outer<16><<<g1, kThreads, 0, s>>>(zb, c->d_enc_inv, c->d_enc_tw, X, n); break;
      default: return fail(FESC_ERR_ARG, "ring degree outside 2^12 .. 2^16");
    }
    if (int rc = hip_check(hipGetLastError(), "k_enc_outer")) return rc;
    k_enc_inner<<<dim3(M, m), kThreads, 0, s>>>(X, c->d_enc_tw, mt, n, M, scale);
    if (int rc = hip_check(hipGetLastError(), "k_enc_inner")) return rc;
    uint64_t* pb = pt + (size_t)b0 * rows * n;
    k_enc_lift<<<dim3(n / kThreads, rows, m), kThreads, 0, s>>>(mt, pb, n, M, rows, level, c->L,
                                                               c->d_pk);
    if (int rc = hip_check(hipGetLastError(), "k_enc_lift")) return rc;
    const RowSel rs{pb, (size_t)rows * n, (size_t)n, 0, level, c->L, 0, 0, 0};
    if (int rc = hip_check(launch_ntt_rows(c, rs, m, rows, false, s), "encode NTT")) return rc;
  }
  return FESC_OK;
}

}  // namespace fesc
