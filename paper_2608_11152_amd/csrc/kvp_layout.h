// Element order inside one (page, kv head) block of the pool.  See the pool layout in kvpattn.h.
//
//   K block, token t, dim c:  ((c / 8) * 16 + t) * 8 + c % 8         (chunk-major: 16 tokens x 8 dims)
//   V block, token t, dim c:  (((c / 16) * 2 + s / 8) * 16 + c % 16) * 8 + s % 8,   s = slot_token(t)
//
// slot_token swaps bits 2 and 3 (an involution, so it maps slots to tokens and tokens to slots).  With
// this order a wave's MFMA operands are contiguous 16-byte rows: for the 16x16 score tile a lane that
// holds scores of tokens {0-3, 8-11} (or {4-7, 12-15}) reads exactly V slots 0-7 (or 8-15) of one dim.
#pragma once
#include <hip/hip_runtime.h>

namespace kvp {

__host__ __device__ constexpr inline int slot_token(int s) { return (s & ~12) | ((s & 4) << 1) | ((s & 8) >> 1); }

template <int D>
__host__ __device__ constexpr inline int k_index(int t, int c) {
  return ((c >> 3) * 16 + t) * 8 + (c & 7);
}

template <int D>
__host__ __device__ constexpr inline int v_index(int t, int c) {
  const int s = slot_token(t);
  return (((c >> 4) * 2 + (s >> 3)) * 16 + (c & 15)) * 8 + (s & 7);
}

// FP8 (one byte per element) block positions: one 16-byte piece holds the operands of two matrix-core
// steps.  K piece X = (c/64)*4 + (c%32)/8 of token t carries dims c%8 of step c/32 (even half, then odd).
// V piece (Y = c/32, slot half s/8, dim c%16) carries slots s%8 of d-tiles 2Y and 2Y+1.
template <int D>
__host__ __device__ constexpr inline int k8_index(int t, int c) {
  return ((((c >> 6) << 2) + ((c & 31) >> 3)) * 16 + t) * 16 + ((c >> 5) & 1) * 8 + (c & 7);
}

template <int D>
__host__ __device__ constexpr inline int v8_index(int t, int c) {
  const int s = slot_token(t);
  return (((c >> 5) * 2 + (s >> 3)) * 16 + (c & 15)) * 16 + ((c >> 4) & 1) * 8 + (s & 7);
}

}  // namespace kvp
