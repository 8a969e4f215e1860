"""Chunked prefill whose tiles are too few to fill the GPU (a short uncached suffix over a long cached
history, Eq. 1): the planner splits each tile's history into key ranges, every range writes a partial
softmax state and the log-sum-exp merge combines them per query row.  Compared with the CPU fp64 oracle on
one session with 32k and 128k cached tokens and chunks of 1 to 256 rows, at other GQA ratios and head
dims, on a batch mixing split and unsplit sessions, on an FP8 pool, with bf16 output, and for run-to-run
determinism."""
import numpy as np
import pytest

import oracle
from oracle import fp8 as F
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

from gpu_helpers import assert_close, note, to_dev_bits

pytestmark = pytest.mark.gpu

HQ, HKV, D = 32, 4, 128
LONG = 131072 + 256  # one sequence long enough for every (ctx, C) case below


@pytest.fixture(scope="module")
def long_seq():
    import torch
    rng = np.random.default_rng(4242)
    npg = (LONG + 15) // 16
    num_pages = npg + 11
    bt = rng.permutation(num_pages)[:npg].astype(np.int32)[None, :]
    kvb = W.f32_to_bf16_bits(rng.standard_normal((LONG, 2, HKV, D), dtype=np.float32))
    note(f"prefill split: append {LONG} tokens")
    pool = kp.Pool(1, num_pages, HKV, D)
    btd = torch.from_numpy(bt).cuda()
    kvd = to_dev_bits(kvb)
    kp.kv_append(pool, 0, kvd[:, 0].contiguous(), kvd[:, 1].contiguous(), btd, [0], [0, LONG])
    torch.cuda.synchronize()
    del kvd
    k64, v64 = oracle.widen_bf16(kvb[:, 0]), oracle.widen_bf16(kvb[:, 1])
    yield pool, btd, k64, v64
    pool.close()


def _rows(C, rng):
    """Rows the oracle checks: all of them up to 128, else the first 32, the last 32 and 32 in between."""
    if C <= 128:
        return [np.arange(C)]
    mid = int(rng.integers(32, C - 64))
    return [np.arange(32), np.arange(mid, mid + 32), np.arange(C - 32, C)]


def _check_single_session(long_seq, ctx, C):
    import torch
    pool, btd, k64, v64 = long_seq
    rng = np.random.default_rng(ctx + C)
    qb = W.f32_to_bf16_bits(rng.standard_normal((C, HQ, D), dtype=np.float32))
    ws_bytes = kp.prefix_chunk_prefill_workspace_size(pool, [ctx], [0, C], HQ)
    assert ws_bytes >= 2 * C * HQ * D * 4, "expected a split history (partials in the workspace)"
    note(f"prefill split ctx={ctx} C={C}")
    out = kp.prefix_chunk_prefill_attn(to_dev_bits(qb), pool, 0, btd, [ctx], [0, C], scale=0.088)
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    o = out.cpu().numpy().astype(np.float64)
    for rows in _rows(C, rng):
        j0 = int(rows[0])
        ref = oracle.prefill_seq(qb[j0:j0 + len(rows)], k64, v64, 0.088, ctx + j0)
        assert_close(o[rows], ref, f"split prefill ctx={ctx} C={C} rows {j0}..{j0 + len(rows) - 1}")


@pytest.mark.parametrize("ctx", [32768, 131072])
@pytest.mark.parametrize("C", [1, 16, 64, 256])
def test_split_history_single_session(long_seq, ctx, C):
    _check_single_session(long_seq, ctx, C)


@pytest.mark.parametrize("ctx,C", [(32768, 96), (32768, 192)])
def test_split_history_one_round(long_seq, ctx, C):
    """Chunks of 3 and of 6 tiles per KV head over 32k cached keys.  Shares by work alone gave one XCD 33
    of 252 workgroups (C = 96), and the first range length 264 workgroups (C = 192): a second round for a
    few of them.  The planner now deals workgroups out within each XCD's 32 CUs and lengthens the ranges
    until the call fits one round."""
    _check_single_session(long_seq, ctx, C)


@pytest.mark.parametrize("G,Hkv,d,ctx,C", [(1, 4, 64, 20000, 40), (4, 2, 64, 30000, 7), (16, 2, 128, 25000, 17),
                                             (2, 8, 128, 9000, 100)])
def test_split_history_other_gqa_ratios(G, Hkv, d, ctx, C):
    """Split histories where C x G rows fill a 256-row tile only partly (G = 1, 4) or several times
    over (G = 16), at both head dims, with ragged chunk and history lengths."""
    import torch
    Hq = G * Hkv
    rng = np.random.default_rng(G * 1000 + C)
    n = ctx + C
    npg = (n + 15) // 16
    num_pages = npg + 5
    bt = rng.permutation(num_pages)[:npg].astype(np.int32)[None, :]
    kvb = W.f32_to_bf16_bits(rng.standard_normal((n, 2, Hkv, d), dtype=np.float32))
    qb = W.f32_to_bf16_bits(rng.standard_normal((C, Hq, d), dtype=np.float32))
    pool = kp.Pool(1, num_pages, Hkv, d)
    assert kp.prefix_chunk_prefill_workspace_size(pool, [ctx], [0, C], Hq) > 0, "expected a split history"
    btd = torch.from_numpy(bt).cuda()
    kvd = to_dev_bits(kvb)
    note(f"prefill split G={G} Hkv={Hkv} d={d} ctx={ctx} C={C}")
    kp.kv_append(pool, 0, kvd[:, 0].contiguous(), kvd[:, 1].contiguous(), btd, [0], [0, n])
    out = kp.prefix_chunk_prefill_attn(to_dev_bits(qb), pool, 0, btd, [ctx], [0, C], scale=1.0 / np.sqrt(d))
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    ref = oracle.prefill_seq(qb, oracle.widen_bf16(kvb[:, 0]), oracle.widen_bf16(kvb[:, 1]), 1.0 / np.sqrt(d), ctx)
    assert_close(out, ref, f"split prefill G={G} d={d} ctx={ctx} C={C}")
    pool.close()


def test_split_and_unsplit_sessions_in_one_call():
    """Three sessions: a long history (split), a short one (split into fewer ranges) and one whose
    history is under one 64-key stage (never split), with chunks of 64, 16 and 1 rows."""
    import torch
    rng = np.random.default_rng(77)
    ctx = np.array([100000, 5000, 40], np.int32)
    C = np.array([64, 16, 1], np.int32)
    n = ctx + C
    npg = (n + 15) // 16
    num_pages = int(npg.sum()) + 9
    perm = rng.permutation(num_pages).astype(np.int32)
    bt = np.full((3, int(npg.max())), -1, np.int32)
    off = 0
    for i in range(3):
        bt[i, :npg[i]] = perm[off:off + npg[i]]
        off += npg[i]
    kvb = W.f32_to_bf16_bits(rng.standard_normal((int(n.sum()), 2, HKV, D), dtype=np.float32))
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    pool = kp.Pool(1, num_pages, HKV, D)
    btd = torch.from_numpy(bt).cuda()
    kvd = to_dev_bits(kvb)
    note("prefill split: mixed batch")
    kp.kv_append(pool, 0, kvd[:, 0].contiguous(), kvd[:, 1].contiguous(), btd, np.zeros(3, np.int32), cu)
    cq = np.concatenate([[0], np.cumsum(C)]).astype(np.int32)
    qb = W.f32_to_bf16_bits(rng.standard_normal((int(C.sum()), HQ, D), dtype=np.float32))
    q = to_dev_bits(qb)
    out = kp.prefix_chunk_prefill_attn(q, pool, 0, btd, ctx, cq, scale=0.09)
    out_bf = kp.prefix_chunk_prefill_attn(q, pool, 0, btd, ctx, cq, scale=0.09, out_dtype=torch.bfloat16)
    again = kp.prefix_chunk_prefill_attn(q, pool, 0, btd, ctx, cq, scale=0.09)
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    assert torch.equal(out, again), "split prefill is not deterministic"
    ref = np.concatenate([oracle.prefill_seq(qb[cq[i]:cq[i + 1]], oracle.widen_bf16(kvb[cu[i]:cu[i + 1], 0]),
                                             oracle.widen_bf16(kvb[cu[i]:cu[i + 1], 1]), 0.09, int(ctx[i]))
                          for i in range(3)])
    assert_close(out, ref, "mixed split batch")
    assert_close(out_bf, ref, "mixed split batch, bf16 out")
    pool.close()


@pytest.mark.parametrize("ks,vs", [(1.0, 1.0), (0.37, 1.9)])
def test_split_history_fp8_pool(ks, vs):
    import torch
    rng = np.random.default_rng(91)
    ctx, C = 40000, 32
    n = ctx + C
    npg = (n + 15) // 16
    num_pages = npg + 3
    bt = rng.permutation(num_pages)[:npg].astype(np.int32)[None, :]
    kvb = W.f32_to_bf16_bits(rng.standard_normal((n, 2, HKV, D), dtype=np.float32))
    qb = W.f32_to_bf16_bits(rng.standard_normal((C, HQ, D), dtype=np.float32))
    pool = kp.Pool(1, num_pages, HKV, D, dtype=kp.KVP_FP8_E4M3)
    pool.set_scales(0, ks, vs)
    btd = torch.from_numpy(bt).cuda()
    kvd = to_dev_bits(kvb)
    note(f"prefill split: fp8 pool scales {ks} {vs}")
    kp.kv_append(pool, 0, kvd[:, 0].contiguous(), kvd[:, 1].contiguous(), btd, [0], [0, n])
    out = kp.prefix_chunk_prefill_attn(to_dev_bits(qb), pool, 0, btd, [ctx], [0, C], scale=0.088)
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    k = F.dequantize(F.quantize_bf16(kvb[:, 0], ks), ks)
    v = F.dequantize(F.quantize_bf16(kvb[:, 1], vs), vs)
    ref = oracle.prefill_seq(qb, k, v, 0.088, ctx)
    assert_close(out, ref, f"fp8 split prefill scales {ks} {vs}")
    pool.close()
