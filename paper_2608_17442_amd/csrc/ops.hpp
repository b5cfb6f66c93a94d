// Kernel launchers of ckks.hip / keyswitch.hip and the host-side operation
// drivers of ops.cpp.
#pragma once

#include "fesc_internal.hpp"

namespace fesc {

// ---------------------------------------------------------------- ckks.hip
hipError_t k_binary_launch(const Context* c, const uint64_t* a, const uint64_t* b, uint64_t* out,
                           uint32_t rows, uint32_t shift, int op, hipStream_t s);
hipError_t k_mul_plain_launch(const Context* c, const uint64_t* ct, const uint64_t* pt,
                              uint64_t* out, uint32_t level, hipStream_t s);
hipError_t k_tensor_launch(const Context* c, const uint64_t* a, const uint64_t* b,
                           uint64_t* d01, uint64_t* d2, uint32_t level, hipStream_t s);
hipError_t k_monomial_launch(const Context* c, const uint64_t* in, uint64_t* out,
                             uint32_t level, uint32_t m, hipStream_t s);
hipError_t k_galois_launch(const Context* c, const uint64_t* in, uint64_t* out, uint32_t rows,
                           uint32_t g, hipStream_t s);
hipError_t k_lift_launch(const Context* c, const int64_t* x, const int8_t* x8, uint64_t* out,
                         uint32_t rows, uint32_t prime0, uint32_t split, uint32_t prime1,
                         hipStream_t s);
hipError_t k_keygen_launch(const Context* c, const uint64_t* a, const uint64_t* e_ntt,
                           const uint64_t* s, const uint64_t* s_from, uint64_t* key,
                           const double2* pmod, hipStream_t st);
hipError_t k_encrypt_launch(const Context* c, const uint64_t* a, const uint64_t* s,
                            const uint64_t* me, uint64_t* ct, uint32_t level, hipStream_t st);
hipError_t k_rescale_lift_launch(const Context* c, const uint64_t* v, uint64_t* w,
                                 uint32_t level, hipStream_t s);
hipError_t k_rescale_combine_launch(const Context* c, const uint64_t* in, const uint64_t* w,
                                    uint64_t* out, uint32_t level, const double2* qlinv,
                                    hipStream_t s);

// ----------------------------------------------------------- keyswitch.hip

// Scratch buffers of one key switch at `level` (all uint64, device).
struct KsBuffers {
  uint64_t* cc;   // [level][N]                 coefficient form of the input
  uint64_t* ext;  // [dnum][level+alpha][N]     ModUp output, evaluation form
  uint64_t* acc;  // [2][level+alpha][N]        inner products
  uint64_t* y;    // [2][level][N]              ModDown conversion
};

hipError_t k_modup_launch(const Context* c, const LevelTables& T, const uint64_t* cc,
                          uint64_t* ext, uint32_t level, hipStream_t s);
hipError_t k_ip_launch(const Context* c, const uint64_t* ext, const uint64_t* in,
                       size_t in_stride, const uint64_t* key, uint64_t* acc, uint32_t level,
                       uint32_t galois, hipStream_t s);
hipError_t k_moddown_bconv_launch(const Context* c, const LevelTables& T, const uint64_t* acc,
                                  uint64_t* y, uint32_t level, hipStream_t s);
hipError_t k_ks_combine_launch(const Context* c, const LevelTables& T, const uint64_t* acc,
                               const uint64_t* y, const uint64_t* add, uint32_t add_mask,
                               uint32_t add_galois, uint64_t* out, uint32_t level,
                               hipStream_t s);

// ------------------------------------------------------------------ ops.cpp
const LevelTables* level_tables(Context* c, uint32_t level, int* err);

}  // namespace fesc
