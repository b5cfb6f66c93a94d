// Scratch layout of a context (ops.cpp): every operation takes its device
// temporaries from one allocation per context, sized for the top level.
#pragma once

#include <cstdint>

#include "fesc_internal.hpp"

namespace fesc {

// One scratch layout, sized for the top level and a batch capacity B (1, or
// kMaxBatch once a batched key switch is requested), shared by every
// operation of the context.
struct Scratch {
  uint32_t cap;
  uint64_t* cin;  // [L][2][N]          private copy of an aliased input
  uint64_t* cc;   // [B][L][N]          centred ModUp digits of the switched polynomials (fp64)
  uint64_t* ext;  // [B][dnum][L+a][N]  ModUp outputs (evaluation form)
  uint64_t* acc;  // [B][2][L+a][N]     key inner products
  uint64_t* y;    // [B][2][L][N]       ModDown conversions (first-pass fp64)
  uint64_t* d2;   // [L][N]             one polynomial (encryption: the secret)
  uint64_t* v;    // [2][N]             rescale: last limb
  uint64_t* w;    // [2][L][N]          rescale: lifted last limb
  uint64_t* cts;  // [B][L][2][N]       batched composite operations: ciphertexts
};

// Carve the layout out of the context's scratch allocation (grown, after a
// device synchronisation, when too small).  batch > 1 asks for the batched
// capacity kMaxBatch; once allocated the larger capacity is kept.
int scratch(Context* c, Scratch* s, uint32_t batch = 1);

}  // namespace fesc
