// One launch for a mixed serving step: the decode work of the step's decoding sequences (one query token
// each, Sec. 3.1 groups) and the chunked prefill of its prefilling sessions (Eq. 1) share the CUs, as
// the rollout classes of Table 1 share one inference instance (Sec. 2.4).
//
// Grid: the decode's wave-path blocks first (the prefill's kPrefillWaves waves each, padded with empty
// blocks to a multiple of 8), then one block per prefill item.  Blocks are dispatched in index order,
// round-robin over the 8 XCDs, so the decode work takes the CUs first and prefill workgroups fill every
// slot a decode workgroup leaves: the decode's tail and the launch boundary between the two no longer
// idle the chip.  The padding keeps each prefill item on the XCD the planner placed it on (workgroup b
// on XCD b mod 8).  No block waits for another; split-KV partials of both parts are merged by the
// log-sum-exp merge kernel after this launch.
//
// The block bodies are the decode and prefill kernels' own (decode_dev.h, prefill_body.inc), so every
// output is bitwise identical to the two separate calls with the same plans.  The kernel carries the
// prefill's register and LDS budget (one 8-wave workgroup per CU), which is also the wave path's
// occupancy in its own launch (8 waves per CU).  The LDS-staged shared-prefix blocks are not compiled
// into this kernel: with their code beside the other two the compiler schedules the prefill's stage
// loop differently and the prefill part ran 2.5% slower (with only the wave path beside it, the stage
// loop is instruction for instruction the prefill kernel's and runs as fast); the caller launches them
// separately.
#include "decode_dev.h"
#include "prefill_dev.h"

namespace kvp {
namespace {

template <int D, bool FP8>
__global__ __launch_bounds__(64 * kPrefillWaves, 8 / kPrefillWaves) void mixed_step_kernel(DecodeArgs d, PrefillArgs p,
                                                                                          int n_dec_blocks) {
  const int b = blockIdx.x;
  if (b >= n_dec_blocks) {
    using namespace pf;
    const PrefillArgs& a = p;
    const unsigned item = (unsigned)(b - n_dec_blocks);
    unsigned char* lds = prefill_lds<D>();
#include "prefill_body.inc"
    return;
  }
  if (b < d.n_wave_blocks) dec::decode_wave_block<D, FP8>(d, b);  // the rest is padding
}

}  // namespace

int mixed_step_decode_blocks(const DecodeArgs& d) {
  const int64_t waves = (int64_t)d.n_items * d.Hkv;  // one per (segment, KV head)
  const int blocks = (int)((waves + kPrefillWaves - 1) / kPrefillWaves);
  return (blocks + 7) / 8 * 8;
}

hipError_t launch_mixed_step(const DecodeArgs& d, const PrefillArgs& p, int D, bool fp8, hipStream_t s) {
  // The fused kernel's workgroups are the prefill's (kPrefillWaves waves): the wave path's block count
  // follows from that.
  DecodeArgs w = d;
  w.n_wave_blocks = (int)(((int64_t)d.n_items * d.Hkv + kPrefillWaves - 1) / kPrefillWaves);
  const int n_dec = w.n_wave_blocks > 0 ? mixed_step_decode_blocks(d) : 0;
  const int64_t blocks = (int64_t)n_dec + p.n_items;
  if (blocks == 0) return hipSuccess;
  const dim3 grid((unsigned)blocks), block(64 * kPrefillWaves);
  if (fp8) {
    if (D == 128) hipLaunchKernelGGL((mixed_step_kernel<128, true>), grid, block, 0, s, w, p, n_dec);
    else hipLaunchKernelGGL((mixed_step_kernel<64, true>), grid, block, 0, s, w, p, n_dec);
  } else if (D == 128) {
    hipLaunchKernelGGL((mixed_step_kernel<128, false>), grid, block, 0, s, w, p, n_dec);
  } else {
    hipLaunchKernelGGL((mixed_step_kernel<64, false>), grid, block, 0, s, w, p, n_dec);
  }
  return hipGetLastError();
}

}  // namespace kvp
