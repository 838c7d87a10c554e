// Wavefront-wide (64-lane) scans and reductions on the vector ALU's DPP
// cross-lane paths: shifts within each 16-lane row, then the broadcasts of
// lane 15 (to rows 1 and 3) and lane 31 (to rows 2 and 3).  Six full-rate
// moves per 32-bit value, no LDS traffic and no loop over active lanes (the
// form a compiler gives an atomic on one LDS address).  Every lane of the
// wavefront must be active at the call.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mori {
namespace wave {

constexpr int ROW_SHR = 0x110;      // row_shr:n is ROW_SHR + n
constexpr int ROW_BCAST15 = 0x142;  // lane 15 of a row to every lane of the next row
constexpr int ROW_BCAST31 = 0x143;  // lane 31 to every lane of rows 2 and 3

// v of the lane CTRL names; 0 where there is none or the row is masked off
template <int CTRL, int ROW_MASK>
__device__ inline uint32_t shift(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROW_MASK, 0xF, true);
}
template <int CTRL, int ROW_MASK>
__device__ inline uint64_t shift(uint64_t v) {
  const uint32_t lo = shift<CTRL, ROW_MASK>((uint32_t)v);
  const uint32_t hi = shift<CTRL, ROW_MASK>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive scan over lanes 0..lane under op, whose identity is 0.
template <typename T, typename Op>
__device__ inline T incl(T v, Op op) {
  v = op(v, shift<ROW_SHR + 1, 0xF>(v));
  v = op(v, shift<ROW_SHR + 2, 0xF>(v));
  v = op(v, shift<ROW_SHR + 4, 0xF>(v));
  v = op(v, shift<ROW_SHR + 8, 0xF>(v));  // inclusive within each row of 16
  v = op(v, shift<ROW_BCAST15, 0xA>(v));  // rows 1 and 3 take the row before
  v = op(v, shift<ROW_BCAST31, 0xC>(v));  // rows 2 and 3 take rows 0-1
  return v;
}

struct Add {
  template <typename T>
  __device__ T operator()(T a, T b) const { return a + b; }
};
struct Or {
  template <typename T>
  __device__ T operator()(T a, T b) const { return a | b; }
};

template <typename T>
__device__ inline T incl_add(T v) { return incl(v, Add()); }

__device__ inline uint32_t lane63(uint32_t v) { return (uint32_t)__builtin_amdgcn_readlane((int)v, 63); }
__device__ inline uint64_t lane63(uint64_t v) {
  return ((uint64_t)lane63((uint32_t)(v >> 32)) << 32) | lane63((uint32_t)v);
}

// Totals over the wavefront, the same (wave-uniform) value in every lane.
template <typename T>
__device__ inline T sum(T v) { return lane63(incl(v, Add())); }
template <typename T>
__device__ inline T all_or(T v) { return lane63(incl(v, Or())); }
template <typename T>
__device__ inline T all_and(T v) { return ~all_or<T>(~v); }

// The lanes whose low BITS-bit digit differs from this lane's: one ballot per
// bit, each lane's bit sign-extended to a whole mask serving both as the
// ballot's input and as the XOR that turns the ballot into "bit differs".
template <int BITS>
__device__ inline uint64_t digit_differs(uint32_t d) {
  uint32_t lo = 0, hi = 0;  // the mask's halves: lanes 0-31 and 32-63
#pragma unroll
  for (int b = 0; b < BITS; ++b) {
    const uint32_t m = (uint32_t)((int32_t)(d << (31 - b)) >> 31);  // all ones where this lane's bit b is set
    const uint64_t bal = __ballot(m != 0);
    lo |= (uint32_t)bal ^ m;
    hi |= (uint32_t)(bal >> 32) ^ m;
  }
  return ((uint64_t)hi << 32) | lo;
}

}  // namespace wave
}  // namespace mori
