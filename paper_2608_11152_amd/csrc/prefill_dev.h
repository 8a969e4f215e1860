// Device helpers of the chunked prefix prefill (one workgroup per (session, KV head, 128 flattened query
// rows, key range) item; the workgroup body is prefill_body.inc).  Included by prefill.hip (the prefill
// kernel) and mixed.hip (the mixed-step launch); everything here is inline.
#pragma once

#include "kvp_kernels.h"
#include "kvp_layout.h"

namespace kvp {
namespace pf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                 c, 0, 0, 0);
}

__device__ __forceinline__ unsigned pack_bf16(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(unsigned, v);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// FP8 pages (FP8 = true): a stage moves half the bytes from the pool and is converted exactly to bf16
// once, on its way into LDS; the matrix-core loop is the bf16 one.  The K scale is folded into the score
// scale and the V scale into the output.
__device__ __forceinline__ unsigned cvt_fp8x2(unsigned w, bool hi) {
  return __builtin_bit_cast(unsigned, hi ? __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true)
                                         : __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false));
}

__device__ __forceinline__ u32x4 cvt8(unsigned w0, unsigned w1) {
  return u32x4{cvt_fp8x2(w0, false), cvt_fp8x2(w0, true), cvt_fp8x2(w1, false), cvt_fp8x2(w1, true)};
}

// LDS of one prefill workgroup: two stages of 4 pages (K and V blocks of one KV head, bf16).  The array is
// a static of this function, so every kernel that calls it holds one copy.
template <int D>
struct PrefillLds {
  static constexpr int bytes = 2 * 4 * 2 * 32 * D;
};

template <int D>
__device__ __forceinline__ unsigned char* prefill_lds() {
  __shared__ __attribute__((aligned(16))) unsigned char lds[PrefillLds<D>::bytes];
  return lds;
}


}  // namespace pf
}  // namespace kvp
