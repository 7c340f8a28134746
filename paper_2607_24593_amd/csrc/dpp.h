// Cross-lane steps of a wave over DPP (data-parallel primitives): the value
// comes from another lane in the same VALU instruction, with no LDS round trip
// (a shuffle ladder costs one ds_bpermute and a wait per step).
//   xor1 / xor2 : quad permutations (1,0,3,2) and (2,3,0,1)
//   xor4        : the half-row mirror (i -> 7 - i in each 8 lanes), then the
//                 quad reversal (3,2,1,0): i -> i ^ 4
//   xor8        : the row mirror (i -> 15 - i in each 16 lanes), then the
//                 half-row mirror: i -> i ^ 8
// Each lane receives exactly the value a shuffle by the same xor would bring,
// so sums taken over these steps keep their bits.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace pivot {

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, true);
}
__device__ __forceinline__ uint32_t lane_xor1(uint32_t x) { return dpp_u<0xB1>(x); }
__device__ __forceinline__ uint32_t lane_xor2(uint32_t x) { return dpp_u<0x4E>(x); }
__device__ __forceinline__ uint32_t lane_xor4(uint32_t x) { return dpp_u<0x1B>(dpp_u<0x141>(x)); }
__device__ __forceinline__ uint32_t lane_xor8(uint32_t x) { return dpp_u<0x141>(dpp_u<0x140>(x)); }
__device__ __forceinline__ float lane_xor1(float x) { return __uint_as_float(lane_xor1(__float_as_uint(x))); }
__device__ __forceinline__ float lane_xor2(float x) { return __uint_as_float(lane_xor2(__float_as_uint(x))); }
__device__ __forceinline__ float lane_xor4(float x) { return __uint_as_float(lane_xor4(__float_as_uint(x))); }
__device__ __forceinline__ float lane_xor8(float x) { return __uint_as_float(lane_xor8(__float_as_uint(x))); }

// A reduction over the 64 lanes with an associative, commutative op (min,
// max, and, or), its result in every lane: butterflies inside each row of 16,
// then the four rows' results read once each.
template <class T, class Op>
__device__ __forceinline__ T wave_reduce(T x, Op op) {
  x = op(x, lane_xor1(x));
  x = op(x, lane_xor2(x));
  x = op(x, lane_xor4(x));
  x = op(x, lane_xor8(x));
  auto at = [&](int l) {
    if constexpr (sizeof(T) == 4 && !__is_same(T, float))
      return (T)__builtin_amdgcn_readlane((int)x, l);
    else
      return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
  };
  return op(op(at(15), at(31)), op(at(47), at(63)));
}

// The same reduction left in lane 63 only, without scalar registers: an
// inclusive scan by row shifts and row broadcasts, lanes without a source
// keeping the op's identity `id`.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t dpp_keep(uint32_t x, uint32_t id) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)id, (int)x, CTRL, ROW_MASK, 0xF, false);
}
template <class Op>
__device__ __forceinline__ uint32_t wave_total_at63(uint32_t x, uint32_t id, Op op) {
  x = op(x, dpp_keep<0x111, 0xF>(x, id));  // row_shr:1
  x = op(x, dpp_keep<0x112, 0xF>(x, id));  // row_shr:2
  x = op(x, dpp_keep<0x114, 0xF>(x, id));  // row_shr:4
  x = op(x, dpp_keep<0x118, 0xF>(x, id));  // row_shr:8
  x = op(x, dpp_keep<0x142, 0xA>(x, id));  // row_bcast:15 -> rows 1, 3
  x = op(x, dpp_keep<0x143, 0xC>(x, id));  // row_bcast:31 -> rows 2, 3
  return x;
}

}  // namespace pivot
