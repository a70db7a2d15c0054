// bf16x6.h -- exact three-way bf16 split of fp32 values for the matrix cores.
//
// a = hi + mid + lo with each part a bf16 (round to nearest): hi takes the top 8
// significant bits, mid the next 8 of the exact residual a - hi, lo the exact rest
// (<= 8 bits), so the split loses nothing.  A product a b is then the sum of the nine
// part products, each exact in fp32; the six of order <= 2 (hi.hi, hi.mid, mid.hi,
// hi.lo, mid.mid, lo.hi) keep the result at fp32 accuracy (the three dropped ones are
// below 2^-24 |a b|).
#pragma once

#include "internal.h"

namespace gcn {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// Two round-to-nearest bf16 values packed in one dword (a in the low half).
__device__ __forceinline__ uint32_t pk_bf16(float a, float b) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  const f2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, b2));
}

// Exact three-way split of a pair: a = hi + mid + lo (each part a bf16), packed per part.
__device__ __forceinline__ void split_pair(float a, float b, uint32_t& hi, uint32_t& mid, uint32_t& lo) {
  hi = pk_bf16(a, b);
  const float ra = a - __uint_as_float(hi << 16), rb = b - __uint_as_float(hi & 0xffff0000u);
  mid = pk_bf16(ra, rb);
  lo = pk_bf16(ra - __uint_as_float(mid << 16), rb - __uint_as_float(mid & 0xffff0000u));
}

}  // namespace
}  // namespace gcn
