"""The allocation-free decode entry point (paged_decode_attn_noalloc) against paged_decode_attn: the same
plan and kernels with the work list and partials in the library's per-GPU scratch, so outputs must be
bitwise equal, call after call, as inputs shrink or grow; an input beyond the scratch is refused before
anything is enqueued."""
import numpy as np
import pytest

from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

from gpu_helpers import GpuCase, assert_close, note, to_dev_bits

pytestmark = pytest.mark.gpu


def _pair(c, lens, gp, out_dtype):
    import torch
    w = c.w
    q = to_dev_bits(c.vals.q)
    ref = kp.paged_decode_attn(q, c.pool, 0, c.bt, lens, group_prefix=gp, scale=w.scale, out_dtype=out_dtype)
    out = torch.full_like(ref, 3.0)
    kp.paged_decode_attn_noalloc(q, c.pool, 0, c.bt, lens, out, group_prefix=gp, scale=w.scale)
    torch.cuda.synchronize()
    assert c.pool.device_error() == kp.KVP_OK
    return out, ref


@pytest.mark.parametrize("name", ["rlvr_s", "mixed_s"])
def test_noalloc_equals_decode_on_two_calls_in_a_row(name):
    import torch
    c = GpuCase(W.make_workload(name))
    w = c.w
    note(f"noalloc {name}: full batch")
    out1, ref1 = _pair(c, w.decode_len, c.gp, torch.float32)
    assert torch.equal(out1, ref1)
    assert_close(out1, c.oracle_decode(), f"noalloc {name} vs oracle")
    # a smaller second call: every sequence shorter (down to its shared prefix + 1), some emptied
    floor = np.zeros(w.B, np.int64)
    if w.num_groups:
        grouped = w.group_id >= 0
        floor[grouped] = w.shared_pages[w.group_id[grouped]] * 16
    lens2 = np.maximum(w.decode_len // 3, np.minimum(w.decode_len, floor + 1)).astype(np.int32)
    lens2[-1] = 0 if floor[-1] == 0 else lens2[-1]
    note(f"noalloc {name}: smaller second call")
    out2, ref2 = _pair(c, lens2, c.gp, torch.bfloat16)
    assert torch.equal(out2, ref2)
    # and back to the larger call, ungrouped
    note(f"noalloc {name}: third call, ungrouped")
    out3, ref3 = _pair(c, w.decode_len, None, torch.float32)
    assert torch.equal(out3, ref3)
    c.pool.close()


def test_noalloc_fp8_pool_and_other_head_dim():
    import torch
    from oracle import fp8 as F
    w = W.make_workload("tiny")  # d = 64, 2 KV heads
    vals = W.make_values(w)
    pool = kp.Pool(1, w.num_pages, w.Hkv, w.d, dtype=kp.KVP_FP8_E4M3)
    pool.set_scales(0, 0.37, 1.9)
    bt = torch.from_numpy(w.block_tables).cuda()
    ck, cv = F.new_pool(w.num_pages, w.Hkv, w.d)
    for ab in w.setup_appends + w.step_appends:
        kv = to_dev_bits(vals.kv[ab.src_rows])
        kp.kv_append(pool, 0, kv[:, 0].contiguous(), kv[:, 1].contiguous(), bt, ab.start_pos, ab.cu_new)
        F.append(ck, cv, vals.kv[ab.src_rows, 0], vals.kv[ab.src_rows, 1], w.block_tables, ab.start_pos, ab.cu_new,
                 0.37, 1.9)
    q = to_dev_bits(vals.q)
    note("noalloc fp8 tiny")
    ref = kp.paged_decode_attn(q, pool, 0, bt, w.decode_len, scale=w.scale)
    out = torch.zeros_like(ref)
    kp.paged_decode_attn_noalloc(q, pool, 0, bt, w.decode_len, out, scale=w.scale)
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    assert torch.equal(out, ref)
    assert_close(out, F.decode(vals.q, ck, cv, w.block_tables, w.decode_len, w.scale, 0.37, 1.9), "noalloc fp8")
    pool.close()


def test_noalloc_refuses_a_call_beyond_its_scratch():
    """2100 two-member groups, each member with a shared page and a private page: 4200 partials of
    Hq x d fp32 need more than the 64 MiB scratch, so the call fails before launching anything."""
    import torch
    groups, Hq, Hkv, d = 2100, 32, 4, 128
    B = 2 * groups
    lens = np.full(B, 20, np.int32)
    gid = np.repeat(np.arange(groups, dtype=np.int32), 2)
    bt = np.zeros((B, 2), np.int32)
    bt[:, 0] = gid
    bt[:, 1] = groups + np.arange(B, dtype=np.int32)
    pool = kp.Pool(1, groups + B, Hkv, d)
    q = torch.zeros((B, Hq, d), dtype=torch.bfloat16, device="cuda")
    out = torch.full((B, Hq, d), 5.0, device="cuda")
    gp = kp.group_prefix(gid, np.ones(groups, np.int32))
    note("noalloc: a call beyond the scratch")
    with pytest.raises(kp.KvpError) as e:
        kp.paged_decode_attn_noalloc(q, pool, 0, torch.from_numpy(bt).cuda(), lens, out, group_prefix=gp)
    assert e.value.code == kp.KVP_EWORKSPACE
    torch.cuda.synchronize()
    assert bool(torch.all(out == 5.0))
    pool.close()
