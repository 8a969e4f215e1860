"""Parity at the full workload sizes (RLVR 64x8, RLHF 128x2, agentic 32 x 32k-128k, mixed 40 sessions in a
1.5M-token pool), in the launch configuration the benchmark times (same plan, bf16 output).  The oracle
computes sampled outputs one sequence / one set of query rows at a time from the generator's values."""
import numpy as np
import pytest

import oracle
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

from gpu_helpers import GpuCase, assert_close, note

pytestmark = pytest.mark.gpu


def sample_seqs(w, k=10, seed=0):
    dec = np.flatnonzero(w.decode_len > 0)
    lens = w.decode_len[dec]
    pick = {int(dec[np.argmin(lens)]), int(dec[np.argmax(lens)])}
    if w.num_groups:  # every member of one group, so a shared prefix is checked for all its samples
        pick |= set(np.flatnonzero(w.group_id == 0).tolist())
    rng = np.random.default_rng(seed)
    pick |= set(rng.choice(dec, size=min(k, len(dec)), replace=False).tolist())
    return sorted(pick)


@pytest.fixture(scope="module", params=["rlvr", "rlhf", "agentic", "mixed"])
def full(request):
    import torch
    name = request.param
    note(f"setup full {name}")
    w = W.make_workload(name)
    vals = W.make_values(w, values="torch", device=torch.device("cuda:0"))
    c = GpuCase(w, vals)
    yield c
    c.pool.close()
    del c
    torch.cuda.empty_cache()


def test_full_decode_sampled(full):
    import torch
    c, w = full, full.w
    note(f"full decode {w.name}")
    out = c.decode(out_dtype=torch.bfloat16).float().cpu().numpy().astype(np.float64)
    assert c.pool.device_error() == kp.KVP_OK
    q = W.to_numpy_bits(c.vals.q)
    seqs = sample_seqs(w)
    ref = np.stack([oracle.decode_seq(q[i], *map(oracle.widen_bf16, W.seq_kv_bits(w, c.vals, i, int(w.decode_len[i]))),
                                      w.scale) for i in seqs])
    assert_close(out[seqs], ref, f"full decode {w.name} ({len(seqs)} sampled sequences)")
    assert np.all(np.isfinite(out))


def test_full_append_sampled_bitwise(full):
    import torch
    c, w = full, full.w
    seqs = sample_seqs(w, k=4, seed=1)
    note(f"full kv_gather {w.name}")
    bt = c.bt[torch.as_tensor(seqs, device="cuda")].contiguous()
    k, v = kp.kv_gather(c.pool, 0, bt, w.final_len[seqs])
    kb, vb = W.to_numpy_bits(k), W.to_numpy_bits(v)
    off = 0
    for i in seqs:
        n = int(w.final_len[i])
        ek, ev = W.seq_kv_bits(w, c.vals, i)
        assert np.array_equal(kb[off:off + n], ek) and np.array_equal(vb[off:off + n], ev), i
        off += n


def test_full_prefill_sampled_rows(full):
    c, w = full, full.w
    if not len(w.prefill_seqs):
        pytest.skip("workload has no prefill chunk")
    note(f"full prefill {w.name}")
    out = c.prefill().cpu().numpy().astype(np.float64)
    assert c.pool.device_error() == kp.KVP_OK
    qp = W.to_numpy_bits(c.vals.qp)
    cu = w.cu_q()
    rng = np.random.default_rng(5)
    for j in sorted({0, len(w.prefill_seqs) - 1, int(rng.integers(len(w.prefill_seqs)))}):
        C, ctx, seq = int(w.prefill_chunk[j]), int(w.prefill_ctx[j]), int(w.prefill_seqs[j])
        rows = np.unique(np.r_[0:64, C - 64:C, rng.integers(0, C, 64)])
        k, v = W.seq_kv_bits(w, c.vals, seq, ctx + C)
        ref = oracle.prefill_seq(qp[cu[j]:cu[j + 1]], oracle.widen_bf16(k), oracle.widen_bf16(v), w.scale, ctx,
                                 rows=rows)
        assert_close(out[cu[j] + rows], ref, f"full prefill {w.name} session {j} ({len(rows)} rows)")


def test_full_mixed_fp8_decode_sampled():
    """The mixed step over an FP8 pool at full size (the benchmark's FP8 leg): sampled sequences against
    the oracle's attention over the dequantised values (quantised by the oracle from the same bf16)."""
    import torch
    from oracle import fp8 as F
    w = W.make_workload("mixed")
    vals = W.make_values(w, values="torch", device=torch.device("cuda:0"))
    note("full mixed fp8 decode")
    pool = kp.Pool(1, w.num_pages, w.Hkv, w.d, dtype=kp.KVP_FP8_E4M3)
    bt = torch.from_numpy(w.block_tables).cuda()
    gp = kp.group_prefix(w.group_id, w.shared_pages)
    for ab in w.setup_appends + w.step_appends:
        rows = torch.from_numpy(ab.src_rows).cuda()
        kp.kv_append(pool, 0, vals.kv[rows, 0].contiguous(), vals.kv[rows, 1].contiguous(), bt, ab.start_pos,
                     ab.cu_new, group_prefix=gp if ab.use_group_prefix else None)
    out = kp.paged_decode_attn(vals.q, pool, 0, bt, w.decode_len, group_prefix=gp, scale=w.scale,
                               out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    out = out.float().cpu().numpy().astype(np.float64)
    q = W.to_numpy_bits(vals.q)
    seqs = sample_seqs(w)
    ref = []
    for i in seqs:
        kb, vb = W.seq_kv_bits(w, vals, i, int(w.decode_len[i]))
        k = F.dequantize(F.quantize_bf16(kb, 1.0), 1.0)
        v = F.dequantize(F.quantize_bf16(vb, 1.0), 1.0)
        ref.append(oracle.decode_seq(q[i], k, v, w.scale))
    assert_close(out[seqs], np.stack(ref), f"full mixed fp8 decode ({len(seqs)} sampled sequences)")
    pool.close()
