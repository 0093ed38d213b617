// Wave64 building blocks for the fused top-K' selection (CDNA4, gfx950).
//
// A shortlist entry is one 64-bit word: the high half is the fp32 key mapped
// to an order-preserving unsigned integer, the low half is the reference
// index.  Unsigned comparison of two words is then exactly the paper-level
// order "smaller distance first, lower index on ties" (Section 6.1 keeps the
// k smallest of each row; ties broken by index are this library's rule).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tod {

constexpr uint64_t kEmpty = ~0ull;  // larger than every real entry

__device__ __forceinline__ uint32_t key_bits(float f) {
  uint32_t u = __float_as_uint(f + 0.0f);  // -0 becomes +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_of(uint64_t e) {
  uint32_t u = (uint32_t)(e >> 32);
  u = (u & 0x80000000u) ? (u & 0x7fffffffu) : ~u;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint64_t make_entry(float key, uint32_t idx) {
  return ((uint64_t)key_bits(key) << 32) | idx;
}

__device__ __forceinline__ uint32_t index_of(uint64_t e) { return (uint32_t)e; }

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int mask) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = __shfl_xor(lo, mask, 64);
  hi = __shfl_xor(hi, mask, 64);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = __shfl(lo, src, 64);
  hi = __shfl(hi, src, 64);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }
__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a < b ? b : a; }

// One compare-exchange stage of a bitonic network over 64*E elements held as
// E registers per lane (element e = r*64 + lane).  `size` is the length of
// the blocks being built (ascending where e & size == 0), `stride` the
// partner distance.
template <int E>
__device__ __forceinline__ void bitonic_stage(uint64_t (&v)[E], int size, int stride, int lane) {
  if (stride >= 64) {
    const int rs = stride >> 6;
#pragma unroll
    for (int r = 0; r < E; ++r) {
      if (r & rs) continue;
      const int e = r * 64 + lane;
      const bool asc = (e & size) == 0;
      const uint64_t lo = umin64(v[r], v[r | rs]);
      const uint64_t hi = umax64(v[r], v[r | rs]);
      v[r] = asc ? lo : hi;
      v[r | rs] = asc ? hi : lo;
    }
  } else {
#pragma unroll
    for (int r = 0; r < E; ++r) {
      const int e = r * 64 + lane;
      const bool asc = (e & size) == 0;
      const bool lower = (e & stride) == 0;
      const uint64_t o = shfl_xor64(v[r], stride);
      v[r] = (asc == lower) ? umin64(v[r], o) : umax64(v[r], o);
    }
  }
}

// Sort 64*E elements ascending.
template <int E>
__device__ __forceinline__ void bitonic_sort(uint64_t (&v)[E], int lane) {
#pragma unroll
  for (int size = 2; size <= 64 * E; size <<= 1)
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) bitonic_stage<E>(v, size, stride, lane);
}

// Sort a bitonic sequence of 64*E elements ascending.
template <int E>
__device__ __forceinline__ void bitonic_merge(uint64_t (&v)[E], int lane) {
#pragma unroll
  for (int stride = 32 * E; stride > 0; stride >>= 1) bitonic_stage<E>(v, 128 * E, stride, lane);
}

// list: ascending, 64*E elements.  other: ascending, 64*E elements.
// Leaves in `list` the 64*E smallest of both, ascending.
template <int E>
__device__ __forceinline__ void merge_lists(uint64_t (&list)[E], const uint64_t (&other)[E],
                                            int lane) {
#pragma unroll
  for (int r = 0; r < E; ++r) list[r] = umin64(list[r], shfl_xor64(other[E - 1 - r], 63));
  bitonic_merge<E>(list, lane);
}

// list: ascending, 64*E elements.  q: ascending, 64 elements (one per lane).
// Leaves in `list` the 64*E smallest of both, ascending.
template <int E>
__device__ __forceinline__ void merge_queue(uint64_t (&list)[E], uint64_t q, int lane) {
  list[E - 1] = umin64(list[E - 1], shfl_xor64(q, 63));
  bitonic_merge<E>(list, lane);
}

}  // namespace tod
