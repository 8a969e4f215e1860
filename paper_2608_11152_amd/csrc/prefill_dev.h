// Device code of the chunked prefix prefill: one workgroup processes one (session, KV head, 128
// flattened query rows, key range) item.  Included by prefill.hip (the prefill kernel) and mixed.hip
// (the mixed-step launch); everything here is inline.
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
// a static of this function, so every kernel that calls it holds one copy, and a kernel that also runs
// other block types can lend the same bytes to them.
template <int D>
struct PrefillLds {
  static constexpr int bytes = 2 * 4 * 2 * 32 * D;
};

template <int D>
__device__ __forceinline__ unsigned char* prefill_lds() {
  __shared__ __attribute__((aligned(16))) unsigned char lds[PrefillLds<D>::bytes];
  return lds;
}

// One workgroup's work: item `item` of the list.
template <int D, bool FP8>
__device__ __forceinline__ void prefill_block(const PrefillArgs& a, unsigned item) {
  constexpr int NS = D / 16;           // k-steps of the score product
  constexpr int NDT = D / 32;          // 32-row d tiles of the output
  constexpr int KB = 16 * D;           // elements per K (or V) block
  constexpr int KBB = 2 * KB;          // bytes per bf16 K (or V) block: the LDS stages are always bf16
  constexpr int PB = 2 * KBB;          // bytes per (page, head) block in LDS
  constexpr int PBG = FP8 ? 2 * KB : PB;  // bytes per (page, head) block in the pool
  constexpr int NPG = 4;               // pages per stage
  constexpr int SB = NPG * PB;         // bytes per LDS stage
  constexpr int NCH = NPG * PBG / (256 * 16);  // 16-byte pool pieces per thread per stage
  static_assert(2 * SB == PrefillLds<D>::bytes, "LDS size");
  unsigned char* lds = prefill_lds<D>();

  const PrefillItem it = a.items[item];
  if (it.seq < 0) return;
  const int tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, l32 = lane & 31, g = lane >> 5;
  const int wvu = __builtin_amdgcn_readfirstlane(wv);  // the same value, known to be wave-uniform
  const int G = a.G;
  const int ctx = a.ctx_lens[it.seq];
  const int q0 = a.cu_q[it.seq];
  const int C = a.cu_q[it.seq + 1] - q0;
  const int nrows = C * G;
  const int f = it.row0 + wv * 32 + l32;  // this lane's query column (flattened row)
  const bool row_ok = f < nrows;
  const int fpos = (row_ok ? f : nrows - 1) / G;
  const int hl = (row_ok ? f : nrows - 1) - fpos * G;
  const int qpos = ctx + fpos;
  const int n_keys = ctx + (min(nrows - 1, it.row0 + 127) / G) + 1;  // keys any row of the tile sees
  const int wave_min_pos = ctx + min(it.row0 + wv * 32, nrows - 1) / G;
  const int n_pages = (n_keys + 15) / 16;
  const int st_end = min(it.st_hi, (n_keys + 63) / 64);  // this workgroup's key range: stages [st_lo, st_end)

  u32x4 qt[NS];
  {
    const uint16_t* qr = a.q + ((int64_t)(q0 + fpos) * a.Hq + it.kvh * G + hl) * D + 8 * g;
#pragma unroll
    for (int s = 0; s < NS; ++s) qt[s] = ld16(qr + 16 * s);
  }
  f32x16 acc[NDT];
#pragma unroll
  for (int d = 0; d < NDT; ++d) acc[d] = f32x16{};
  float m_run = -INFINITY, l_run = 0.0f;
  const float cs = a.scale_log2;

  const int64_t page_stride = (int64_t)a.Hkv * PBG;  // bytes
  const unsigned char* hbase = reinterpret_cast<const unsigned char*>(a.layer) + (int64_t)it.kvh * PBG;
  // The block table is read-only for the kernel's lifetime: read it through the constant address space
  // so page ids are scalar loads.
  typedef const __attribute__((address_space(4))) int32_t* const_i32p;
  const_i32p btr = (const_i32p)(a.bt + (int64_t)it.seq * a.maxp);
  bool bad = false;

  const int seq_tokens = ctx + C;
  constexpr int CPP = NCH / NPG;  // 16-byte pool pieces per page per thread
  // Stage `st` = logical pages 4*st .. 4*st+3.  Piece k of a stage is its bytes [4096k + 1024w, +1024)
  // for wave w (one page's contiguous kilobyte, 16 bytes per lane).  The next stage's pieces are loaded
  // into registers at the top of a step and stored to the other LDS buffer at its end, so their
  // latency hides behind the step's MFMA work; staging through registers measured faster than direct
  // global->LDS copies.  Page ids: four scalar loads, index clamped into the tile's page range so each
  // is in bounds.  A missing or invalid page is read from page 0 and `patch` zeroes it once stored,
  // together with the slots past the end of the sequence in its last page (stale pool contents).
  u32x4 stg[NCH];
  auto fetch = [&](int st, unsigned& okm) {
    okm = 0u;
    int ids[NPG];
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) ids[pg] = btr[min(st * NPG + pg, n_pages - 1)];
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) {
      const bool inr = st * NPG + pg < n_pages;
      const bool ok = inr && (unsigned)ids[pg] < (unsigned)a.num_pages;
      okm |= ok ? 1u << pg : 0u;
      bad |= inr && !ok;
      ids[pg] = ok ? ids[pg] : 0;
      if constexpr (CPP >= 1) {
        // wave-uniform page base + a 32-bit lane offset
        const unsigned char* pbase = hbase + (int64_t)ids[pg] * page_stride;
#pragma unroll
        for (int c = 0; c < CPP; ++c) stg[pg * CPP + c] = ld16(pbase + (uint32_t)(c * 4096 + tid * 16));
      }
    }
    if constexpr (CPP == 0) {
      // A page block is smaller than one 4 KB round: round k's wave pieces span 4096 / PBG pages.
#pragma unroll
      for (int k = 0; k < NCH; ++k) {
        const int o = k * 4096 + wvu * 1024;
        stg[k] = ld16(hbase + (int64_t)ids[o / PBG] * page_stride + (uint32_t)((o % PBG) + lane * 16));
      }
    }
  };
  // bf16 pools: the pieces go to LDS as they are.  FP8 pools: each 16-byte piece is converted (exactly)
  // into the two 16-byte bf16 rows it holds (a K piece: two 8-dim chunks of one token; a V piece: 8
  // slots of two dims), so the LDS stage has the bf16 layout and the MFMA loop is shared.  Tokens past
  // the sequence end and pages that are missing or invalid are zeroed here, in registers.
  auto store_stage = [&](int st, int buf, unsigned okm) {
    if constexpr (!FP8) {
#pragma unroll
      for (int k = 0; k < NCH; ++k) *reinterpret_cast<u32x4*>(lds + buf * SB + k * 4096 + tid * 16) = stg[k];
    } else {
      const bool whole = (st + 1) * NPG * 16 <= seq_tokens && okm == (1u << NPG) - 1u;
#pragma unroll
      for (int k = 0; k < NCH; ++k) {
        const int o = k * 4096 + wvu * 1024;
        const int pg = o / PBG;
        const int ob = (o % PBG) + lane * 16;  // byte of the piece in its (page, head) block
        u32x4 lo = cvt8(stg[k][0], stg[k][1]), hi = cvt8(stg[k][2], stg[k][3]);
        int dlo, dhi;
        if (ob < KB) {
          const int X = ob >> 8, t = (ob >> 4) & 15;  // piece X of token t
          const int ca = 8 * (X >> 2) + (X & 3);     // its 8-dim chunks ca and ca + 4
          dlo = (ca * 16 + t) * 16;
          dhi = ((ca + 4) * 16 + t) * 16;
          if (!whole) {
            const int valid = (okm >> pg) & 1u ? seq_tokens - (st * NPG + pg) * 16 : 0;
            if (t >= valid) lo = hi = u32x4{0u, 0u, 0u, 0u};
          }
        } else {
          const int vp = (ob - KB) >> 4;
          const int Y = vp >> 5, sh = (vp >> 4) & 1, c16 = vp & 15;  // slots 8sh.. of dims 32Y+c16, +16
          dlo = KBB + ((4 * Y + sh) * 16 + c16) * 16;
          dhi = KBB + ((4 * Y + 2 + sh) * 16 + c16) * 16;
          if (!whole) {
            const int valid = (okm >> pg) & 1u ? seq_tokens - (st * NPG + pg) * 16 : 0;
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              const unsigned m = (slot_token(8 * sh + 2 * w) < valid ? 0xFFFFu : 0u) |
                                 (slot_token(8 * sh + 2 * w + 1) < valid ? 0xFFFF0000u : 0u);
              lo[w] &= m;
              hi[w] &= m;
            }
          }
        }
        unsigned char* dst = lds + buf * SB + pg * PB;
        *reinterpret_cast<u32x4*>(dst + dlo) = lo;
        *reinterpret_cast<u32x4*>(dst + dhi) = hi;
      }
    }
  };
  // bf16 pools: zero, in this thread's own pieces of stage st, the pages that are missing or invalid and
  // the slots past the end of the sequence (stale pool contents), after they are stored.
  auto patch = [&](int st, int buf, unsigned okm) {
    if constexpr (FP8) return;  // masked on the way to LDS
    if ((st + 1) * NPG * 16 <= seq_tokens && okm == (1u << NPG) - 1u) return;
    // Piece k of this thread: stage bytes [4096k + 16 tid, +16), in page (4096k + 1024 wv) / PB.
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const int o = k * 4096 + wvu * 1024;
      const int pg = o / PB;
      const int valid = (okm >> pg) & 1u ? seq_tokens - (st * NPG + pg) * 16 : 0;  // usable tokens of this page
      if (valid >= 16) continue;
      const int inb = (o % PB) + lane * 16;
      u32x4* lp = reinterpret_cast<u32x4*>(lds + buf * SB + o + lane * 16);
      u32x4 v = *lp;
      if (inb < KBB) {
        if (((inb >> 4) & 15) >= valid) v = u32x4{0u, 0u, 0u, 0u};
      } else {
        const int h = ((inb - KBB) >> 8) & 1;  // V chunk holds slots 8h..8h+7
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const unsigned lo = slot_token(8 * h + 2 * w) < valid ? 0xFFFFu : 0u;
          const unsigned hi = slot_token(8 * h + 2 * w + 1) < valid ? 0xFFFF0000u : 0u;
          v[w] &= lo | hi;
        }
      }
      *lp = v;
    }
  };
  unsigned okm;  // bit pg: page pg of the stage in flight is valid
  fetch(it.st_lo, okm);
  store_stage(it.st_lo, 0, okm);
  // All earlier global loads (the query fragments) have landed: without this, the compiler's waits
  // for them inside the loop would also wait for each step's staging loads.
  __builtin_amdgcn_s_waitcnt(0x0F70);
  patch(it.st_lo, 0, okm);
  __syncthreads();
  int buf = 0;
  for (int st = it.st_lo; st < st_end; ++st) {
    const bool more = st + 1 < st_end;
    if (more) fetch(st + 1, okm);
    const unsigned char* sb = lds + buf * SB;
    // The two 32-key tiles' MFMA chains are interleaved.  K operands are read from LDS KD k-steps ahead
    // of their MFMAs, V operands one page ahead (page 0's before the softmax), which leaves registers for
    // the staged next stage.  Scheduling barriers keep this order.
    f32x16 S[2] = {f32x16{}, f32x16{}};
    {
      constexpr int KD = 4;
      const unsigned char* kp0 = sb + (l32 >> 4) * PB + (g * 16 + (l32 & 15)) * 16;
      const unsigned char* kp1 = kp0 + 2 * PB;
      u32x4 k0[NS], k1[NS];
#pragma unroll
      for (int s = 0; s < KD; ++s) {
        k0[s] = ld16(kp0 + s * 512);
        k1[s] = ld16(kp1 + s * 512);
      }
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        if (s + KD < NS) {
          k0[s + KD] = ld16(kp0 + (s + KD) * 512);
          k1[s + KD] = ld16(kp1 + (s + KD) * 512);
        }
        S[0] = mfma32(k0[s], qt[s], S[0]);
        S[1] = mfma32(k1[s], qt[s], S[1]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    u32x4 vf[NPG][NDT];
    auto load_v = [&](int pg) {
      const unsigned char* vp = sb + pg * PB + KBB + (g * 16 + (l32 & 15)) * 16 + (l32 >> 4) * 512;
#pragma unroll
      for (int d = 0; d < NDT; ++d) vf[pg][d] = ld16(vp + d * 1024);
    };
    load_v(0);
    __builtin_amdgcn_sched_barrier(0);
    // Softmax against a reference max.  With c = scale * log2(e) > 0 (the host rejects other scales),
    // the weights are exp2(c*s - m_run), m_run being the running row max of the earlier stages (exact
    // from the range's first stage on: every row sees that stage's first key, which the planner
    // guarantees).  The stage's own max is taken only at that first stage
    // or when a lane's weight sum passes 256 (some score rose above m_run): otherwise every weight is at
    // most 256 and, numerator and denominator sharing the reference, the result is unchanged.  So the
    // common path has no max reduction: one FMA and one exponential per score.
    float t[32];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int i = 0; i < 16; ++i) t[kk * 16 + i] = S[kk][i];
    const int kbase = st * 64;
    if (kbase + 63 > wave_min_pos) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = kbase + kk * 32 + 8 * (i >> 2) + 4 * g + (i & 3);
          if (key > qpos) t[kk * 16 + i] = -INFINITY;
        }
    }
    u32x4 pb[NPG];
    float ssum = 0.0f;
    auto weights = [&](float mr) {
      ssum = 0.0f;
#pragma unroll
      for (int pg = 0; pg < NPG; ++pg) {
        float p[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          p[j] = fast_exp2(__builtin_fmaf(t[(pg >> 1) * 16 + (pg & 1) * 8 + j], cs, -mr));
          ssum += p[j];
        }
#pragma unroll
        for (int w = 0; w < 4; ++w) pb[pg][w] = pack_bf16(p[2 * w], p[2 * w + 1]);
      }
    };
    bool slow = st == it.st_lo;
    if (!slow) {
      weights(m_run);
      slow = __any(!(ssum <= 256.0f));
    }
    if (slow) {
      float mx = fmaxf(fmaxf(t[0], t[1]), t[2]);
#pragma unroll
      for (int i = 3; i < 31; i += 2) mx = fmaxf(fmaxf(mx, t[i]), t[i + 1]);
      mx = fmaxf(mx, t[31]);
      mx = fmaxf(mx, __shfl_xor(mx, 32)) * cs;
      const float mnew = fmaxf(m_run, mx);
      const float alpha = fast_exp2(m_run - mnew);  // 0 at the first stage (m_run = -inf), acc and l are 0
      m_run = mnew;
      l_run *= alpha;
#pragma unroll
      for (int d = 0; d < NDT; ++d) acc[d] *= alpha;
      weights(m_run);
    }
    l_run += ssum;
#pragma unroll
    for (int pg = 0; pg < NPG; ++pg) {
      if (pg + 1 < NPG) load_v(pg + 1);
#pragma unroll
      for (int d = 0; d < NDT; ++d) acc[d] = mfma32(vf[pg][d], pb[pg], acc[d]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (more) {
      store_stage(st + 1, buf ^ 1, okm);
      // vmcnt(0): every staging load has been consumed; stating it lets the compiler drop later waits
      __builtin_amdgcn_s_waitcnt(0x0F70);
      patch(st + 1, buf ^ 1, okm);
    }
    __syncthreads();
    buf ^= 1;
  }
  if (bad) atomicCAS(a.err, 0, KVP_ERANGE);
  l_run += __shfl_xor(l_run, 32);
  if (!row_ok) return;
  if (it.slot >= 0) {
    // One key range of a split tile: the partial state of this query row, for the merge.
    const int64_t pidx = (int64_t)a.part_base[it.seq] + (int64_t)fpos * a.nsplit[it.seq] + it.slot;
    const int head = it.kvh * G + hl;
    float* pa = a.part_acc + (pidx * a.Hq + head) * D + 4 * g;
#pragma unroll
    for (int d = 0; d < NDT; ++d)
#pragma unroll
      for (int t4 = 0; t4 < 4; ++t4)
        *reinterpret_cast<float4*>(pa + 32 * d + 8 * t4) =
            make_float4(acc[d][4 * t4] * a.v_scale, acc[d][4 * t4 + 1] * a.v_scale, acc[d][4 * t4 + 2] * a.v_scale,
                        acc[d][4 * t4 + 3] * a.v_scale);
    if (g == 0) a.part_ml[pidx * a.Hq + head] = make_float2(m_run, l_run);
    return;
  }
  const float inv = l_run > 0.0f ? a.v_scale / l_run : 0.0f;
  const int64_t o = ((int64_t)(q0 + fpos) * a.Hq + it.kvh * G + hl) * D + 4 * g;
#pragma unroll
  for (int d = 0; d < NDT; ++d)
#pragma unroll
    for (int t4 = 0; t4 < 4; ++t4) {
      const int64_t oi = o + 32 * d + 8 * t4;
      const float v0 = acc[d][4 * t4] * inv, v1 = acc[d][4 * t4 + 1] * inv;
      const float v2 = acc[d][4 * t4 + 2] * inv, v3 = acc[d][4 * t4 + 3] * inv;
      if (a.out_f32) {
        *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.out) + oi) = make_float4(v0, v1, v2, v3);
      } else {
        uint2 u;
        u.x = pack_bf16(v0, v1);
        u.y = pack_bf16(v2, v3);
        *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.out) + oi) = u;
      }
    }
}

}  // namespace pf
}  // namespace kvp
