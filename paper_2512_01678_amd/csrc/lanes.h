// lanes.h -- cross-lane reductions over aligned groups of a wavefront.
#pragma once

#include <cstdint>

namespace gcn {
namespace {

// Lane move inside a 16-lane row (DPP): CTRL 0xB1 takes lane i ^ 1, 0x4E lane i ^ 2,
// 0x141 the mirror in the half-row (7 - i), 0x140 the mirror in the row (15 - i).
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

// All-reduce over aligned groups of LANES lanes, every lane ending with the same bits
// (each step combines a lane with a partner that holds the mirror-image partial, and
// the operation is commutative).  Inside a 16-lane row the partners are reached by DPP
// moves rather than through LDS; wider groups add cross-row shuffles.  Every lane of a
// group must be active.
template <int LANES, class Op>
__device__ __forceinline__ float group_reduce(float v, Op op) {
  if constexpr (LANES >= 2) v = op(v, dpp_mov<0xB1>(v));
  if constexpr (LANES >= 4) v = op(v, dpp_mov<0x4E>(v));
  if constexpr (LANES >= 8) v = op(v, dpp_mov<0x141>(v));
  if constexpr (LANES >= 16) v = op(v, dpp_mov<0x140>(v));
  if constexpr (LANES >= 32) v = op(v, __shfl_xor(v, 16, 64));
  if constexpr (LANES >= 64) v = op(v, __shfl_xor(v, 32, 64));
  return v;
}
// OR over aligned groups of LANES lanes (bitmask words), every lane ending with the word.
template <int LANES>
__device__ __forceinline__ uint32_t group_or(uint32_t v) {
  if constexpr (LANES >= 2) v |= dpp_mov<0xB1>(v);
  if constexpr (LANES >= 4) v |= dpp_mov<0x4E>(v);
  if constexpr (LANES >= 8) v |= dpp_mov<0x141>(v);
  if constexpr (LANES >= 16) v |= dpp_mov<0x140>(v);
  if constexpr (LANES >= 32) v |= (uint32_t)__shfl_xor((int)v, 16, 64);
  if constexpr (LANES >= 64) v |= (uint32_t)__shfl_xor((int)v, 32, 64);
  return v;
}

}  // namespace
}  // namespace gcn
