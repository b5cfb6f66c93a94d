// Radix-2 butterfly stages on 16-value register tiles, shared by the NTT
// kernels and the VALU calibration kernel.
#pragma once

#include "fesc_internal.hpp"

namespace fesc {

// Radix-2 stages on a 16-value register tile, pairs (r, r + H) with r & H == 0.
// tw(gi) gives the twiddle {w, w/q} of group gi = r / 2H.
//
// Twiddles are stored balanced, |w| <= q/2, so the Shoup product of
// |x| <= X q lands within (0.5 + X/8) q for q < 2^50 (its quotient estimate is
// off by at most |x w/q| 2^-52).  Butterflies therefore reduce lazily:
//   forward (CT): only every other stage (RED) reduces the pass-through
//     operand u; a reducing stage maps the bound X to 1 + X/8, a lazy one to
//     0.5 + 1.125 X, so from any input below 2.6 q values stay below 2.6 q;
//   inverse (GS): only every other stage reduces the sum u + v; the
//     difference goes through a Shoup product, so a (reducing, lazy) pair maps
//     X to 1 + X/2 and inputs below 2 q stay below 2 q.
// Both are far inside the 2^53 range of exact fp64 integers.
template <int H, bool RED, class TW>
__device__ __forceinline__ void ct_st(double (&x)[16], TW tw, double q, double qinv) {
#pragma unroll
  for (int g = 0; g < 16; g += 2 * H) {
    const double2 w = tw(g / (2 * H));
#pragma unroll
    for (int r = g; r < g + H; ++r) {
      const double u = RED ? red_bal(x[r], q, qinv) : x[r];
      const double v = mm_shoup(x[r + H], w.x, w.y, q);
      x[r] = u + v;
      x[r + H] = u - v;
    }
  }
}

template <int H, bool RED, class TW>
__device__ __forceinline__ void gs_st(double (&x)[16], TW tw, double q, double qinv) {
#pragma unroll
  for (int g = 0; g < 16; g += 2 * H) {
    const double2 w = tw(g / (2 * H));
#pragma unroll
    for (int r = g; r < g + H; ++r) {
      const double u = x[r], v = x[r + H];
      x[r] = RED ? red_bal(u + v, q, qinv) : u + v;
      x[r + H] = mm_shoup(u - v, w.x, w.y, q);
    }
  }
}

}  // namespace fesc
