"""mixed_step_attn: the decode and chunk-prefill work of one step in one launch.  Its outputs must equal,
bit for bit, paged_decode_attn followed by prefix_chunk_prefill_attn with the same arguments (the same
plans and the same block bodies), and stay within tolerance of the oracle; either part may be empty, and
a host-detected error leaves the outputs untouched."""
import numpy as np
import pytest

from gpu_helpers import GpuCase, assert_close, note, to_dev_bits
from oracle import fp8 as F
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W
from test_gpu_fp8 import Fp8Case

pytestmark = pytest.mark.gpu


def _prefill_rows(w, bt):
    s0, s1 = int(w.prefill_seqs[0]), int(w.prefill_seqs[-1]) + 1
    return bt[s0:s1], s0, s1


def _run_both_ways(pool, w, q, qp, bt, gp):
    """mixed_step_attn, then the two separate calls, on the same pool; f32 outputs."""
    import torch
    btp, _, _ = _prefill_rows(w, bt)
    od, op = kp.mixed_step_attn(pool, 0, q, bt, w.decode_len, qp, btp, w.prefill_ctx, w.cu_q(), group_prefix=gp,
                                scale=w.scale, out_dtype=torch.float32)
    rd = kp.paged_decode_attn(q, pool, 0, bt, w.decode_len, group_prefix=gp, scale=w.scale, out_dtype=torch.float32)
    rp = kp.prefix_chunk_prefill_attn(qp, pool, 0, btp, w.prefill_ctx, w.cu_q(), scale=w.scale,
                                      out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    return od, op, rd, rp


@pytest.mark.parametrize("name,over", [("mixed_s", {}), ("agentic_s", {}), ("mixed_s", dict(Hq=8, Hkv=2, d=64))])
def test_mixed_step_equals_the_two_calls(name, over):
    """mixed_s: split-KV decode partials and prefill history splits (fewer than 512 tiles) in the fused
    launch, wide groups on the LDS-staged prefix blocks in their own launch ahead of it; agentic_s: no
    groups; d = 64 with GQA 8/2."""
    import torch
    note(f"mixed_step {name} {over}")
    w = W.make_workload(name, **over)
    c = GpuCase(w)
    items, _, _ = kp.kvp_plan_decode(w.decode_len, w.Hq, w.Hkv, c.gp)
    note(f"mixed_step {name}: {len(items)} decode items ({int((items[:, 0] == 1).sum())} prefix), "
         f"{int(w.cu_q()[-1])} prefill rows")
    q, qp = to_dev_bits(c.vals.q), to_dev_bits(c.vals.qp)
    od, op, rd, rp = _run_both_ways(c.pool, w, q, qp, c.bt, c.gp)
    assert torch.equal(od, rd), "decode part differs from paged_decode_attn"
    assert torch.equal(op, rp), "prefill part differs from prefix_chunk_prefill_attn"
    assert_close(od, c.oracle_decode(), f"mixed_step decode {name} {over}")
    assert_close(op, c.oracle_prefill(), f"mixed_step prefill {name} {over}")


def test_mixed_step_fp8_pages():
    import torch
    note("mixed_step fp8 mixed_s scales 0.37 1.9")
    c = Fp8Case("mixed_s", 0.37, 1.9)
    w = c.w
    q, qp = to_dev_bits(c.vals.q), to_dev_bits(c.vals.qp)
    od, op, rd, rp = _run_both_ways(c.pool, w, q, qp, c.bt, c.gp)
    assert torch.equal(od, rd) and torch.equal(op, rp)
    _, s0, s1 = _prefill_rows(w, c.bt)
    ref_d = F.decode(c.vals.q, c.ck, c.cv, w.block_tables, w.decode_len, w.scale, c.ks, c.vs)
    ref_p = F.prefill(c.vals.qp, c.ck, c.cv, w.block_tables[s0:s1], w.prefill_ctx, w.cu_q(), w.scale, c.ks, c.vs)
    assert_close(od, ref_d, "mixed_step fp8 decode")
    assert_close(op, ref_p, "mixed_step fp8 prefill")


def test_mixed_step_with_one_part_empty():
    """Decode only (rlvr_s: 14 LDS-staged prefix items) and prefill only (agentic_s), each bitwise equal
    to its own call; both parts empty enqueues nothing."""
    import torch
    note("mixed_step decode only rlvr_s")
    c = GpuCase(W.make_workload("rlvr_s"))
    w = c.w
    q = to_dev_bits(c.vals.q)
    q0 = torch.empty((0, w.Hq, w.d), dtype=torch.bfloat16, device="cuda")
    bt0 = torch.empty((0, c.bt.shape[1]), dtype=torch.int32, device="cuda")
    od, op = kp.mixed_step_attn(c.pool, 0, q, c.bt, w.decode_len, q0, bt0, [], [0], group_prefix=c.gp,
                                scale=w.scale, out_dtype=torch.float32)
    rd = kp.paged_decode_attn(q, c.pool, 0, c.bt, w.decode_len, group_prefix=c.gp, scale=w.scale,
                              out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert op.shape[0] == 0 and torch.equal(od, rd)
    assert_close(od, c.oracle_decode(), "mixed_step decode only rlvr_s")

    note("mixed_step prefill only agentic_s")
    c = GpuCase(W.make_workload("agentic_s"))
    w = c.w
    qp = to_dev_bits(c.vals.qp)
    btp, _, _ = _prefill_rows(w, c.bt)
    q0 = torch.empty((0, w.Hq, w.d), dtype=torch.bfloat16, device="cuda")
    bt0 = torch.empty((0, c.bt.shape[1]), dtype=torch.int32, device="cuda")
    od, op = kp.mixed_step_attn(c.pool, 0, q0, bt0, [], qp, btp, w.prefill_ctx, w.cu_q(), scale=w.scale,
                                out_dtype=torch.float32)
    rp = kp.prefix_chunk_prefill_attn(qp, c.pool, 0, btp, w.prefill_ctx, w.cu_q(), scale=w.scale,
                                      out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert od.shape[0] == 0 and torch.equal(op, rp)

    note("mixed_step both parts empty")
    od, op = kp.mixed_step_attn(c.pool, 0, q0, bt0, [], q0, bt0, [], [0], out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert od.shape[0] == 0 and op.shape[0] == 0 and c.pool.device_error() == kp.KVP_OK


def test_mixed_step_rejects_before_launch():
    """A short workspace or a chunk past the table is refused on the host: nothing is enqueued and the
    outputs keep their contents."""
    import torch
    note("mixed_step host errors mixed_s")
    c = GpuCase(W.make_workload("mixed_s"))
    w = c.w
    q, qp = to_dev_bits(c.vals.q), to_dev_bits(c.vals.qp)
    btp, _, _ = _prefill_rows(w, c.bt)
    od = torch.full((w.B, w.Hq, w.d), 7.0, dtype=torch.float32, device="cuda")
    op = torch.full((int(w.cu_q()[-1]), w.Hq, w.d), 7.0, dtype=torch.float32, device="cuda")
    need = kp.mixed_step_workspace_size(c.pool, w.decode_len, w.prefill_ctx, w.cu_q(), w.Hq, c.gp)
    small = torch.empty(need - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(kp.KvpError) as e:
        kp.mixed_step_attn(c.pool, 0, q, c.bt, w.decode_len, qp, btp, w.prefill_ctx, w.cu_q(), group_prefix=c.gp,
                           scale=w.scale, out_dec=od, out_pf=op, ws=small)
    assert e.value.code == kp.KVP_EWORKSPACE
    too_long = np.asarray(w.prefill_ctx, np.int32).copy()
    too_long[0] = c.bt.shape[1] * 16
    with pytest.raises(kp.KvpError) as e:
        kp.mixed_step_attn(c.pool, 0, q, c.bt, w.decode_len, qp, btp, too_long, w.cu_q(), group_prefix=c.gp,
                           scale=w.scale, out_dec=od, out_pf=op)
    assert e.value.code == kp.KVP_ERANGE
    torch.cuda.synchronize()
    assert bool((od == 7.0).all()) and bool((op == 7.0).all())
