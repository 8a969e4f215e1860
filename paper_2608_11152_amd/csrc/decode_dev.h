// Device code of the paged decode path: the split-KV wave chunks, the LDS-staged shared-prefix
// blocks and the block-level entry points the kernels call (bf16 and FP8 pages).  Included by
// decode.hip (the decode kernels) and mixed.hip (the mixed-step launch); everything here is inline.
#pragma once

#include "kvp_kernels.h"
#include "kvp_layout.h"

namespace kvp {
namespace dec {


typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

// KV pages are read exactly once per call: stream them past the caches (nontemporal loads measure
// ~7.0 TB/s on MI355X against ~6.2 TB/s for ordinary loads in a plain streaming-read test).
__device__ __forceinline__ u32x4 ld16_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
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

// Per-lane online-softmax state for one query column and the 8 token slots this lane holds.
template <int NT>
struct SoftState {
  f32x4 acc[NT];
  float m;  // running max in log2 units (may lag the true max by < 8, see update)
  float l;  // this lane's share of the weight sum (reduced over the 4 lane groups at the end)
};

// One two-page step: scale the 8 raw scores, mask invalid tokens, update the running max, accumulate
// P^T V^T into acc.  `vv` are the lane's V^T operand tiles.  The max is only moved when a score exceeds
// it by more than 2^8, so weights stay <= 256 (exact in bf16 range) and the rescale of acc is usually
// skipped; the final normalisation uses the same max, so the result is unchanged.
template <int NT>
__device__ __forceinline__ void softmax_pv(SoftState<NT>& st, f32x4 sx, f32x4 sy, float scale_log2,
                                           const bool (&ok)[8], bool masked, u32x4 (&vv)[NT]) {
  float t[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    t[i] = sx[i] * scale_log2;
    t[4 + i] = sy[i] * scale_log2;
  }
  if (masked) {
    unsigned vm[4];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (!ok[j]) t[j] = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) vm[w] = (ok[2 * w] ? 0xFFFFu : 0u) | (ok[2 * w + 1] ? 0xFFFF0000u : 0u);
#pragma unroll
    for (int d = 0; d < NT; ++d)
#pragma unroll
      for (int w = 0; w < 4; ++w) vv[d][w] &= vm[w];
  }
  float mx = fmaxf(fmaxf(fmaxf(t[0], t[1]), fmaxf(t[2], t[3])), fmaxf(fmaxf(t[4], t[5]), fmaxf(t[6], t[7])));
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const bool need = mx > st.m + 8.0f;
  if (__any(need)) {
    const float alpha = need ? fast_exp2(st.m - mx) : 1.0f;
    st.m = need ? mx : st.m;
    st.l *= alpha;
#pragma unroll
    for (int d = 0; d < NT; ++d) st.acc[d] *= alpha;
  }
  const float mr = (st.m == -INFINITY) ? 0.0f : st.m;
  float p[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    p[j] = fast_exp2(t[j] - mr);
    st.l += p[j];
  }
  u32x4 pp;
  pp[0] = pack_bf16(p[0], p[1]);
  pp[1] = pack_bf16(p[2], p[3]);
  pp[2] = pack_bf16(p[4], p[5]);
  pp[3] = pack_bf16(p[6], p[7]);
#pragma unroll
  for (int d = 0; d < NT; ++d) st.acc[d] = mfma16(vv[d], pp, st.acc[d]);
}

// Validity of the 8 tokens a lane holds in the step over pages (p, p+1): slots 8*(q4&1)+j of page
// p + (q4>>1), i.e. tokens 4*(q4&1)+j (j<4) and 8+4*(q4&1)+j-4 (j>=4).
__device__ __forceinline__ void lane_token_ok(int p, int q4, bool page_ok, int tok_end, bool (&ok)[8]) {
  const int pos0 = (p + (q4 >> 1)) * 16 + (q4 & 1) * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    ok[i] = page_ok && pos0 + i < tok_end;
    ok[4 + i] = page_ok && pos0 + 8 + i < tok_end;
  }
}

// A group hint (kvp_group_prefix) promises that every member's table names the representative row's pages
// for the shared prefix; the kernels read those pages through the representative row only.  Lanes of the
// other members compare their own table entry for a page of each step with the row's, and a mismatch is
// recorded as KVP_EGROUP in the pool's error word (the loads go out with the step's own page-id loads).
__device__ __forceinline__ void report_group_mismatch(const DecodeArgs& a, bool differs, int lane) {
  if (__any(differs) && lane == 0) atomicCAS(a.err, 0, KVP_EGROUP);
}

// Store one column's state: normalised output (slot < 0) or a partial for the merge kernel.
template <int D, int NT>
__device__ __forceinline__ void write_state(const DecodeArgs& a, const DecodeItem& it, const SoftState<NT>& st,
                                            int seq, int head, int q4) {
  if (it.slot < 0) {
    const float inv = st.l > 0.0f ? a.v_scale / st.l : 0.0f;
    const int64_t o = ((int64_t)seq * a.Hq + head) * D + 4 * q4;
#pragma unroll
    for (int d = 0; d < NT; ++d) {
      const f32x4 v = st.acc[d] * inv;
      if (a.out_f32) {
        *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.out) + o + 16 * d) = v;
      } else {
        uint2 u;
        u.x = pack_bf16(v[0], v[1]);
        u.y = pack_bf16(v[2], v[3]);
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + o + 16 * d) = u;
      }
    }
  } else {
    const int64_t pidx = (int64_t)a.part_base[seq] + it.slot;
    float* pa = a.part_acc + (pidx * a.Hq + head) * D + 4 * q4;
#pragma unroll
    for (int d = 0; d < NT; ++d) *reinterpret_cast<f32x4*>(pa + 16 * d) = st.acc[d] * a.v_scale;
    if (q4 == 0) a.part_ml[pidx * a.Hq + head] = make_float2(st.m, st.l);
  }
}

// ---------------------------------------------------------------------------------------------------
// One wave per (item, KV head): private page ranges, and shared-prefix ranges of groups with <= 16
// query columns.  Operands are loaded straight from HBM; each two-page step issues 2*D/32 K loads and
// D/16 V loads of 16 bytes per lane (16 KB per wave at d = 128).
// ---------------------------------------------------------------------------------------------------
template <int D>
__device__ __forceinline__ void decode_wave_chunk(const DecodeArgs& a, const DecodeItem& it, int kvh, int lane) {
  constexpr int NS = D / 32;
  constexpr int NT = D / 16;
  constexpr int KB = 16 * D;
  const int q4 = lane >> 4, c16 = lane & 15;
  const int ncols = it.n_mem * a.G;
  const bool col_ok = c16 < ncols;
  int seq = 0, head = 0;
  if (col_ok) {
    const int m = c16 / a.G;
    seq = a.members[it.mem_off + m];
    head = kvh * a.G + (c16 - m * a.G);
  }
  u32x4 qt[NS];
  {
    const uint16_t* qr = a.q + ((int64_t)seq * a.Hq + head) * D;
#pragma unroll
    for (int s = 0; s < NS; ++s) qt[s] = col_ok ? ld16(qr + 8 * (4 * s + q4)) : u32x4{0u, 0u, 0u, 0u};
  }
  SoftState<NT> st;
#pragma unroll
  for (int d = 0; d < NT; ++d) st.acc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;

  const int64_t page_stride = (int64_t)a.Hkv * 2 * KB;
  const uint16_t* hbase = a.layer + (int64_t)kvh * 2 * KB;
  const int32_t* btr = a.bt + (int64_t)it.row * a.maxp;
  const int32_t* btm = a.bt + (int64_t)seq * a.maxp;
  const bool chk = it.kind == 1 && col_ok && seq != it.row;  // a member other than the representative
  const int k_off = (c16 & 7) * 8;
  const int v_off = KB + ((q4 & 1) * 16 + c16) * 8;
  bool bad = false, differs = false;
  for (int p = it.page_lo; p < it.page_hi; p += 2) {
    const bool has_b = p + 1 < it.page_hi;
    int ida = btr[p];
    int idb = has_b ? btr[p + 1] : ida;
    if (chk && (!(q4 & 1) || has_b)) differs |= btm[p + (q4 & 1)] != ((q4 & 1) ? idb : ida);
    const bool va = (unsigned)ida < (unsigned)a.num_pages;
    const bool vb = has_b && (unsigned)idb < (unsigned)a.num_pages;
    bad |= !va || (has_b && !vb);
    if (!va) ida = 0;
    if (!vb) idb = ida;
    const uint16_t* pa = hbase + (int64_t)ida * page_stride;
    const uint16_t* pb = hbase + (int64_t)idb * page_stride;
    const uint16_t* kp = (c16 < 8 ? pa : pb) + k_off;
    const uint16_t* vp = (q4 < 2 ? pa : pb) + v_off;
    u32x4 kx[NS], ky[NS], vv[NT];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      kx[s] = ld16_stream(kp + (4 * s + q4) * 128);
      ky[s] = ld16_stream(kp + (4 * s + q4) * 128 + 64);
    }
#pragma unroll
    for (int d = 0; d < NT; ++d) vv[d] = ld16_stream(vp + d * 256);
    f32x4 sx = {0.f, 0.f, 0.f, 0.f}, sy = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      sx = mfma16(kx[s], qt[s], sx);
      sy = mfma16(ky[s], qt[s], sy);
    }
    const bool masked = !has_b || !va || !vb || (p + 2) * 16 > it.tok_end;
    bool ok[8];
    lane_token_ok(p, q4, q4 < 2 ? va : vb, it.tok_end, ok);
    softmax_pv<NT>(st, sx, sy, a.scale_log2, ok, masked, vv);
  }
  if (bad && lane == 0) atomicCAS(a.err, 0, KVP_ERANGE);
  report_group_mismatch(a, differs, lane);
  st.l += __shfl_xor(st.l, 16);
  st.l += __shfl_xor(st.l, 32);
  if (col_ok) write_state<D, NT>(a, it, st, seq, head, q4);
}

// ---------------------------------------------------------------------------------------------------
// One 4-wave workgroup per (shared-prefix item, KV head) for groups with 17..64 query columns (e.g. 8
// samples x 8 heads).  Each two-page step is staged once in LDS by all 256 threads (double-buffered,
// register-staged so the next step's HBM reads overlap this step's math); wave w then computes query
// columns 16w..16w+15 from LDS.  The prefix pages therefore cross HBM once per group.
// ---------------------------------------------------------------------------------------------------
template <int D>
struct GroupLds {
  static constexpr int KB = 16 * D;      // elements per K (or V) block
  static constexpr int PB = 4 * KB;      // bytes per (page, head): K + V blocks
  static constexpr int PAD = 128;        // keeps the two staged pages on different LDS banks
  static constexpr int SB = 2 * PB + PAD;
  static constexpr int bytes = 2 * SB;   // double-buffered two-page stage
};

template <int D>
__device__ __forceinline__ void decode_group_block(const DecodeArgs& a, int block, unsigned char* lds) {
  constexpr int NS = D / 32;
  constexpr int NT = D / 16;
  constexpr int KB = GroupLds<D>::KB;
  constexpr int PB = GroupLds<D>::PB;
  constexpr int PAD = GroupLds<D>::PAD;
  constexpr int SB = GroupLds<D>::SB;
  constexpr int NCH = 2 * PB / (256 * 16);

  const int item = block / a.Hkv;
  const int kvh = block - item * a.Hkv;
  if (item >= a.n_group_items) return;
  const DecodeItem it = a.group_items[item];
  const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, q4 = lane >> 4, c16 = lane & 15;
  const int ncols = it.n_mem * a.G;
  const int col = wv * 16 + c16;
  const bool wave_on = wv * 16 < ncols;
  const bool col_ok = col < ncols;
  int seq = 0, head = 0;
  if (col_ok) {
    const int m = col / a.G;
    seq = a.members[it.mem_off + m];
    head = kvh * a.G + (col - m * a.G);
  }
  u32x4 qt[NS];
  {
    const uint16_t* qr = a.q + ((int64_t)seq * a.Hq + head) * D;
#pragma unroll
    for (int s = 0; s < NS; ++s) qt[s] = col_ok ? ld16(qr + 8 * (4 * s + q4)) : u32x4{0u, 0u, 0u, 0u};
  }
  SoftState<NT> st;
#pragma unroll
  for (int d = 0; d < NT; ++d) st.acc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;

  const int64_t page_stride = (int64_t)a.Hkv * 2 * KB;
  const uint16_t* hbase = a.layer + (int64_t)kvh * 2 * KB;
  const int32_t* btr = a.bt + (int64_t)it.row * a.maxp;
  const int32_t* btm = a.bt + (int64_t)seq * a.maxp;
  const bool chk = col_ok && seq != it.row;  // a member other than the representative
  bool bad = false, differs = false;

  // Stage pages (p, p+1) into registers; pages past the range or with invalid ids become zeros.
  auto fetch = [&](int p, u32x4 (&r)[NCH]) {
    const bool has_b = p + 1 < it.page_hi;
    const int ida = btr[p];
    const int idb = has_b ? btr[p + 1] : 0;
    const bool va = (unsigned)ida < (unsigned)a.num_pages;
    const bool vb = has_b && (unsigned)idb < (unsigned)a.num_pages;
    bad |= !va || (has_b && !vb);
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const int off = (k * 256 + tid) * 16;
      const int pg = off / PB, inb = off - pg * PB;
      const bool ok = pg == 0 ? va : vb;
      const int id = pg == 0 ? ida : idb;
      r[k] = ok ? ld16_stream(reinterpret_cast<const unsigned char*>(hbase + (int64_t)id * page_stride) + inb)
                : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store = [&](int buf, const u32x4 (&r)[NCH]) {
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const int off = (k * 256 + tid) * 16;
      const int pg = off / PB, inb = off - pg * PB;
      *reinterpret_cast<u32x4*>(lds + buf * SB + pg * (PB + PAD) + inb) = r[k];
    }
  };

  u32x4 r[NCH];
  fetch(it.page_lo, r);
  store(0, r);
  __syncthreads();
  int buf = 0;
  for (int p = it.page_lo; p < it.page_hi; p += 2) {
    const bool more = p + 2 < it.page_hi;
    // Group-hint check of this step's pages, loaded before the next step's staging loads so that the
    // comparison below waits only for these two loads, not for the staging ones.
    const int pc = min(p + (q4 & 1), it.page_hi - 1);
    const int mine = btm[pc], theirs = btr[pc];
    __builtin_amdgcn_sched_barrier(0);
    if (more) fetch(p + 2, r);
    if (wave_on) {
      const unsigned char* sb = lds + buf * SB;
      const unsigned char* kp = sb + (c16 < 8 ? 0 : PB + PAD) + (c16 & 7) * 16;
      const unsigned char* vp = sb + (q4 < 2 ? 0 : PB + PAD) + 2 * KB + ((q4 & 1) * 16 + c16) * 16;
      u32x4 kx[NS], ky[NS], vv[NT];
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        kx[s] = ld16(kp + (4 * s + q4) * 256);
        ky[s] = ld16(kp + (4 * s + q4) * 256 + 128);
      }
#pragma unroll
      for (int d = 0; d < NT; ++d) vv[d] = ld16(vp + d * 512);
      f32x4 sx = {0.f, 0.f, 0.f, 0.f}, sy = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        sx = mfma16(kx[s], qt[s], sx);
        sy = mfma16(ky[s], qt[s], sy);
      }
      const bool has_b = p + 1 < it.page_hi;
      const bool va = (unsigned)btr[p] < (unsigned)a.num_pages;
      const bool vb = has_b && (unsigned)btr[p + 1] < (unsigned)a.num_pages;
      const bool masked = !has_b || !va || !vb || (p + 2) * 16 > it.tok_end;
      bool ok[8];
      lane_token_ok(p, q4, q4 < 2 ? va : vb, it.tok_end, ok);
      softmax_pv<NT>(st, sx, sy, a.scale_log2, ok, masked, vv);
    }
    differs |= chk && mine != theirs;
    if (more) store(buf ^ 1, r);
    __syncthreads();
    buf ^= 1;
  }
  if (bad && tid == 0) atomicCAS(a.err, 0, KVP_ERANGE);
  if (!wave_on) return;
  report_group_mismatch(a, differs, lane);
  st.l += __shfl_xor(st.l, 16);
  st.l += __shfl_xor(st.l, 32);
  if (!col_ok) return;
  write_state<D, NT>(a, it, st, seq, head, q4);
}

// ---------------------------------------------------------------------------------------------------
// FP8 (E4M3) pages.  One 16-byte piece of a page block carries the operands of two matrix-core steps
// (kvp_layout.h), converted exactly to bf16 in registers; the K scale is folded into the score scale and
// the V scale into the output.  A step covers four pages (16 KB of K and V per wave, as the bf16 path
// moves per two pages) and computes them as two two-page sub-steps.
// ---------------------------------------------------------------------------------------------------
__device__ __forceinline__ unsigned cvt_fp8x2(unsigned w, bool hi) {
  return __builtin_bit_cast(unsigned, hi ? __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true)
                                         : __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false));
}

// 16 codes -> the bf16 operand of bytes 0-7 (lo) and of bytes 8-15 (hi).
__device__ __forceinline__ void cvt_piece(u32x4 r, u32x4& lo, u32x4& hi) {
  lo = u32x4{cvt_fp8x2(r[0], false), cvt_fp8x2(r[0], true), cvt_fp8x2(r[1], false), cvt_fp8x2(r[1], true)};
  hi = u32x4{cvt_fp8x2(r[2], false), cvt_fp8x2(r[2], true), cvt_fp8x2(r[3], false), cvt_fp8x2(r[3], true)};
}

// Scores and PV of one two-page sub-step from raw K / V pieces (NS/2 K pieces per score tile, NT/2 V
// pieces), for pages whose validity the caller has resolved.
template <int NS, int NT>
__device__ __forceinline__ void fp8_substep(SoftState<NT>& st, const u32x4 (&qt)[NS], const u32x4 (&kxr)[NS / 2],
                                            const u32x4 (&kyr)[NS / 2], const u32x4 (&vr)[NT / 2], float scale_log2,
                                            const bool (&ok)[8], bool masked) {
  f32x4 sx = {0.f, 0.f, 0.f, 0.f}, sy = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int p2 = 0; p2 < NS / 2; ++p2) {
    u32x4 a0, a1, b0, b1;
    cvt_piece(kxr[p2], a0, a1);
    cvt_piece(kyr[p2], b0, b1);
    sx = mfma16(a0, qt[2 * p2], sx);
    sy = mfma16(b0, qt[2 * p2], sy);
    sx = mfma16(a1, qt[2 * p2 + 1], sx);
    sy = mfma16(b1, qt[2 * p2 + 1], sy);
  }
  u32x4 vv[NT];
#pragma unroll
  for (int y = 0; y < NT / 2; ++y) cvt_piece(vr[y], vv[2 * y], vv[2 * y + 1]);
  softmax_pv<NT>(st, sx, sy, scale_log2, ok, masked, vv);
}

template <int D>
__device__ __forceinline__ void decode_wave_chunk_fp8(const DecodeArgs& a, const DecodeItem& it, int kvh, int lane) {
  constexpr int NS = D / 32;
  constexpr int NT = D / 16;
  constexpr int KB = 16 * D;  // bytes per K (or V) block
  const int q4 = lane >> 4, c16 = lane & 15;
  const int ncols = it.n_mem * a.G;
  const bool col_ok = c16 < ncols;
  int seq = 0, head = 0;
  if (col_ok) {
    const int m = c16 / a.G;
    seq = a.members[it.mem_off + m];
    head = kvh * a.G + (c16 - m * a.G);
  }
  u32x4 qt[NS];
  {
    const uint16_t* qr = a.q + ((int64_t)seq * a.Hq + head) * D;
#pragma unroll
    for (int s = 0; s < NS; ++s) qt[s] = col_ok ? ld16(qr + 8 * (4 * s + q4)) : u32x4{0u, 0u, 0u, 0u};
  }
  SoftState<NT> st;
#pragma unroll
  for (int d = 0; d < NT; ++d) st.acc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;

  const int64_t page_stride = (int64_t)a.Hkv * 2 * KB;
  const unsigned char* hbase = reinterpret_cast<const unsigned char*>(a.layer) + (int64_t)kvh * 2 * KB;
  const int32_t* btr = a.bt + (int64_t)it.row * a.maxp;
  const int32_t* btm = a.bt + (int64_t)seq * a.maxp;
  const bool chk = it.kind == 1 && col_ok && seq != it.row;  // a member other than the representative
  const int k_off = ((q4)*16 + (c16 & 7)) * 16;                       // + p2 * 1024 (4 chunks of 256 B)
  const int v_off = KB + (((q4 & 1)) * 16 + c16) * 16;                // + y * 512
  bool bad = false, differs = false;
  for (int p = it.page_lo; p < it.page_hi; p += 4) {
    int id[4];
    bool val[4], has[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      has[j] = p + j < it.page_hi;
      id[j] = has[j] ? btr[p + j] : 0;
    }
    // group-hint check: the member's entry for page p + q4 is loaded with the step's page ids
    const bool ck = chk && p + q4 < it.page_hi;
    const int mine = ck ? btm[p + q4] : 0;
    differs |= ck && mine != (q4 == 0 ? id[0] : q4 == 1 ? id[1] : q4 == 2 ? id[2] : id[3]);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      val[j] = has[j] && (unsigned)id[j] < (unsigned)a.num_pages;
      bad |= has[j] && !val[j];
      if (!val[j]) id[j] = 0;
    }
    const bool two = has[2];
    u32x4 kxr[2][NS / 2], kyr[2][NS / 2], vr[2][NT / 2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (u == 1 && !two) break;
      const unsigned char* px = hbase + (int64_t)id[2 * u] * page_stride;
      const unsigned char* py = hbase + (int64_t)(has[2 * u + 1] ? id[2 * u + 1] : id[2 * u]) * page_stride;
      const unsigned char* kp = (c16 < 8 ? px : py) + k_off;
      const unsigned char* vp = (q4 < 2 ? px : py) + v_off;
#pragma unroll
      for (int p2 = 0; p2 < NS / 2; ++p2) {
        kxr[u][p2] = ld16_stream(kp + p2 * 1024);
        kyr[u][p2] = ld16_stream(kp + p2 * 1024 + 128);
      }
#pragma unroll
      for (int y = 0; y < NT / 2; ++y) vr[u][y] = ld16_stream(vp + y * 512);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (u == 1 && !two) break;
      const int x = p + 2 * u;
      const bool hb = has[2 * u + 1];
      const bool va = val[2 * u], vb = hb && val[2 * u + 1];
      const bool masked = !hb || !va || !vb || (x + 2) * 16 > it.tok_end;
      bool ok[8];
      lane_token_ok(x, q4, q4 < 2 ? va : vb, it.tok_end, ok);
      fp8_substep<NS, NT>(st, qt, kxr[u], kyr[u], vr[u], a.scale_log2, ok, masked);
    }
  }
  if (bad && lane == 0) atomicCAS(a.err, 0, KVP_ERANGE);
  report_group_mismatch(a, differs, lane);
  st.l += __shfl_xor(st.l, 16);
  st.l += __shfl_xor(st.l, 32);
  if (col_ok) write_state<D, NT>(a, it, st, seq, head, q4);
}

template <int D>
struct GroupLds8 {
  static constexpr int KB = 16 * D;      // bytes per K (or V) block
  static constexpr int PB = 2 * KB;      // bytes per (page, head): K + V blocks
  static constexpr int PAD = 128;        // keeps consecutive staged pages on different LDS banks
  static constexpr int SB = 4 * (PB + PAD);
  static constexpr int bytes = 2 * SB;   // double-buffered four-page stage
};

template <int D>
__device__ __forceinline__ void decode_group_block_fp8(const DecodeArgs& a, int block, unsigned char* lds) {
  constexpr int NS = D / 32;
  constexpr int NT = D / 16;
  constexpr int KB = GroupLds8<D>::KB;
  constexpr int PB = GroupLds8<D>::PB;
  constexpr int PAD = GroupLds8<D>::PAD;
  constexpr int SB = GroupLds8<D>::SB;
  constexpr int NCH = 4 * PB / (256 * 16);

  const int item = block / a.Hkv;
  const int kvh = block - item * a.Hkv;
  if (item >= a.n_group_items) return;
  const DecodeItem it = a.group_items[item];
  const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, q4 = lane >> 4, c16 = lane & 15;
  const int ncols = it.n_mem * a.G;
  const int col = wv * 16 + c16;
  const bool wave_on = wv * 16 < ncols;
  const bool col_ok = col < ncols;
  int seq = 0, head = 0;
  if (col_ok) {
    const int m = col / a.G;
    seq = a.members[it.mem_off + m];
    head = kvh * a.G + (col - m * a.G);
  }
  u32x4 qt[NS];
  {
    const uint16_t* qr = a.q + ((int64_t)seq * a.Hq + head) * D;
#pragma unroll
    for (int s = 0; s < NS; ++s) qt[s] = col_ok ? ld16(qr + 8 * (4 * s + q4)) : u32x4{0u, 0u, 0u, 0u};
  }
  SoftState<NT> st;
#pragma unroll
  for (int d = 0; d < NT; ++d) st.acc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;

  const int64_t page_stride = (int64_t)a.Hkv * 2 * KB;
  const unsigned char* hbase = reinterpret_cast<const unsigned char*>(a.layer) + (int64_t)kvh * 2 * KB;
  const int32_t* btr = a.bt + (int64_t)it.row * a.maxp;
  const int32_t* btm = a.bt + (int64_t)seq * a.maxp;
  const bool chk = col_ok && seq != it.row;  // a member other than the representative
  bool bad = false, differs = false;

  // Stage pages p..p+3 into registers; pages past the range or with invalid ids become zeros.
  auto fetch = [&](int p, u32x4 (&r)[NCH]) {
    int id[4];
    bool okp[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool has = p + j < it.page_hi;
      id[j] = has ? btr[p + j] : 0;
      okp[j] = has && (unsigned)id[j] < (unsigned)a.num_pages;
      bad |= has && !okp[j];
    }
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const int off = (k * 256 + tid) * 16;
      const int pg = off / PB, inb = off - pg * PB;
      r[k] = okp[pg] ? ld16_stream(hbase + (int64_t)id[pg] * page_stride + inb) : u32x4{0u, 0u, 0u, 0u};
    }
  };
  auto store = [&](int buf, const u32x4 (&r)[NCH]) {
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const int off = (k * 256 + tid) * 16;
      const int pg = off / PB, inb = off - pg * PB;
      *reinterpret_cast<u32x4*>(lds + buf * SB + pg * (PB + PAD) + inb) = r[k];
    }
  };

  u32x4 r[NCH];
  fetch(it.page_lo, r);
  store(0, r);
  __syncthreads();
  int buf = 0;
  for (int p = it.page_lo; p < it.page_hi; p += 4) {
    const bool more = p + 4 < it.page_hi;
    // Group-hint check of this step's pages, loaded before the next step's staging loads (see the bf16
    // block).
    const int pc = min(p + q4, it.page_hi - 1);
    const int mine = btm[pc], theirs = btr[pc];
    __builtin_amdgcn_sched_barrier(0);
    if (more) fetch(p + 4, r);
    if (wave_on) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int x = p + 2 * u;
        if (x >= it.page_hi) break;
        const unsigned char* sx0 = lds + buf * SB + (2 * u) * (PB + PAD);
        const unsigned char* sy0 = sx0 + (PB + PAD);
        const unsigned char* kp = (c16 < 8 ? sx0 : sy0) + (q4 * 16 + (c16 & 7)) * 16;
        const unsigned char* vp = (q4 < 2 ? sx0 : sy0) + KB + ((q4 & 1) * 16 + c16) * 16;
        u32x4 kxr[NS / 2], kyr[NS / 2], vr[NT / 2];
#pragma unroll
        for (int p2 = 0; p2 < NS / 2; ++p2) {
          kxr[p2] = ld16(kp + p2 * 1024);
          kyr[p2] = ld16(kp + p2 * 1024 + 128);
        }
#pragma unroll
        for (int y = 0; y < NT / 2; ++y) vr[y] = ld16(vp + y * 512);
        const bool hb = x + 1 < it.page_hi;
        const bool va = (unsigned)btr[x] < (unsigned)a.num_pages;
        const bool vb = hb && (unsigned)btr[x + 1] < (unsigned)a.num_pages;
        const bool masked = !hb || !va || !vb || (x + 2) * 16 > it.tok_end;
        bool ok[8];
        lane_token_ok(x, q4, q4 < 2 ? va : vb, it.tok_end, ok);
        fp8_substep<NS, NT>(st, qt, kxr, kyr, vr, a.scale_log2, ok, masked);
      }
    }
    differs |= chk && mine != theirs;
    if (more) store(buf ^ 1, r);
    __syncthreads();
    buf ^= 1;
  }
  if (bad && tid == 0) atomicCAS(a.err, 0, KVP_ERANGE);
  if (!wave_on) return;
  report_group_mismatch(a, differs, lane);
  st.l += __shfl_xor(st.l, 16);
  st.l += __shfl_xor(st.l, 32);
  if (!col_ok) return;
  write_state<D, NT>(a, it, st, seq, head, q4);
}

// ---------------------------------------------------------------------------------------------------
// Wave path: private page ranges, and shared-prefix ranges of groups with <= 16 query columns.  The
// planner cuts the concatenated page ranges into equal segments; waves s*Hkv .. s*Hkv+Hkv-1 process
// segment s, one KV head each, chunk after chunk.  Operands are loaded straight from HBM; each
// two-page step issues 2*D/32 K loads and D/16 V loads of 16 bytes per lane (16 KB per wave, d = 128).
// ---------------------------------------------------------------------------------------------------
template <int D, bool FP8>
__device__ __forceinline__ void decode_wave_block(const DecodeArgs& a, int block) {
  const int lane = threadIdx.x & 63;
  const int wid = block * (int)(blockDim.x >> 6) + (threadIdx.x >> 6);
  const int seg = wid / a.Hkv;
  const int kvh = wid - seg * a.Hkv;
  if (seg >= a.n_items) return;
  const int c1 = a.seg_off[seg + 1];
  for (int c = a.seg_off[seg]; c < c1; ++c) {
    if constexpr (FP8) decode_wave_chunk_fp8<D>(a, a.items[c], kvh, lane);
    else decode_wave_chunk<D>(a, a.items[c], kvh, lane);
  }
}

}  // namespace dec
}  // namespace kvp
