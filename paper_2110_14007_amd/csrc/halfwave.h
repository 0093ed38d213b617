// Cross-lane moves and bitonic networks inside the two 32-lane halves of a
// wave64 (CDNA4 DPP / permlane forms; lane semantics verified on gfx950).
//
// Partner for "lane xor s" within a half:
//   s = 1, 2      DPP quad_perm
//   s = 4         row_half_mirror (xor 7) then quad reverse (xor 3)
//   s = 8         row_mirror (xor 15) then row_half_mirror (xor 7)
//   s = 16        v_permlane16_swap and a per-lane select
//   s = 31        row_mirror (xor 15) then the xor-16 move
// None of these touch LDS, so a compare-exchange stage costs a few VALU
// cycles instead of an LDS round trip.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tod {

template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xf, 0xf, true);
}

template <int S>
__device__ __forceinline__ uint32_t xor_lane(uint32_t v, int lane) {
  if constexpr (S == 1) {
    return dpp<0xB1>(v);
  } else if constexpr (S == 2) {
    return dpp<0x4E>(v);
  } else if constexpr (S == 4) {
    return dpp<0x1B>(dpp<0x141>(v));
  } else if constexpr (S == 8) {
    return dpp<0x141>(dpp<0x140>(v));
  } else if constexpr (S == 16) {
    const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return (lane & 16) ? p[0] : p[1];
  } else {
    static_assert(S == 31, "unsupported lane distance");
    const uint32_t m = dpp<0x140>(v);
    const auto p = __builtin_amdgcn_permlane16_swap(m, m, false, false);
    return (lane & 16) ? p[0] : p[1];
  }
}

template <int S>
__device__ __forceinline__ uint64_t xor_lane64(uint64_t v, int lane) {
  const uint32_t lo = xor_lane<S>((uint32_t)v, lane);
  const uint32_t hi = xor_lane<S>((uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t xor_lane64_dyn(uint64_t v, int s, int lane) {
  switch (s) {
    case 1: return xor_lane64<1>(v, lane);
    case 2: return xor_lane64<2>(v, lane);
    case 4: return xor_lane64<4>(v, lane);
    case 8: return xor_lane64<8>(v, lane);
    default: return xor_lane64<16>(v, lane);
  }
}

// One compare-exchange stage over 32*R elements per half (element
// e = r*32 + lane%32).  Blocks of `size` are ascending where e & size == 0.
template <int R>
__device__ __forceinline__ void half_stage(uint64_t (&v)[R], int size, int stride, int lane) {
  const int j = lane & 31;
  if (stride >= 32) {
    const int rs = stride >> 5;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      if (r & rs) continue;
      const int e = r * 32 + j;
      const bool asc = (e & size) == 0;
      const uint64_t a = v[r], b = v[r | rs];
      const bool sw = asc ? (b < a) : (a < b);
      v[r] = sw ? b : a;
      v[r | rs] = sw ? a : b;
    }
  } else {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int e = r * 32 + j;
      const bool keep_min = ((e & size) == 0) == ((e & stride) == 0);
      const uint64_t o = xor_lane64_dyn(v[r], stride, lane);
      const bool take = keep_min ? (o < v[r]) : (v[r] < o);
      v[r] = take ? o : v[r];
    }
  }
}

// Sort 32 elements per half ascending (one register).
__device__ __forceinline__ void half_sort32(uint64_t& x, int lane) {
  uint64_t v[1] = {x};
#pragma unroll
  for (int size = 2; size <= 32; size <<= 1)
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) half_stage<1>(v, size, stride, lane);
  x = v[0];
}

// list: 32*R ascending elements per half; q: 32 ascending elements per half.
// Leaves the 32*R smallest of both in `list`, ascending.
template <int R>
__device__ __forceinline__ void half_merge(uint64_t (&list)[R], uint64_t q, int lane) {
  const uint64_t rq = xor_lane64<31>(q, lane);  // q reversed within the half
  list[R - 1] = rq < list[R - 1] ? rq : list[R - 1];
#pragma unroll
  for (int stride = 16 * R; stride > 0; stride >>= 1) half_stage<R>(list, 64 * R, stride, lane);
}

}  // namespace tod
