"""Parity at the full workload sizes (RLVR 64x8, RLHF 128x2, agentic 32 x 32k-128k, mixed 40 sessions in a
1.5M-token pool), in the launch configuration the benchmark times (same plan, bf16 output).  The oracle
computes every decoding sequence, and the prefill rows named in each test, one sequence at a time from the
generator's values."""
import numpy as np
import pytest

import oracle
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

from gpu_helpers import GpuCase, assert_close, note, oracle_by_kv_head

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


def test_full_decode_every_sequence(full):
    """Every decoding sequence of the workload against the oracle (run per KV head on contiguous copies;
    the first sequence also through the oracle's own all-head call, which must agree bitwise)."""
    import time
    import torch
    c, w = full, full.w
    note(f"full decode {w.name}: every sequence")
    out = c.decode(out_dtype=torch.bfloat16).float().cpu().numpy().astype(np.float64)
    assert c.pool.device_error() == kp.KVP_OK
    q = W.to_numpy_bits(c.vals.q)
    dec = np.flatnonzero(w.decode_len > 0)
    t0 = time.time()
    ref = np.zeros((len(dec), w.Hq, w.d))
    for j, i in enumerate(dec):
        kb, vb = W.seq_kv_bits(w, c.vals, int(i), int(w.decode_len[i]))
        ref[j] = oracle_by_kv_head(oracle.decode_seq, q[i], kb, vb, w.scale)
        if j == 0:
            own = oracle.decode_seq(q[i], oracle.widen_bf16(kb), oracle.widen_bf16(vb), w.scale)
            assert np.max(np.abs(ref[j] - own)) <= 1e-12
    note(f"full decode {w.name}: oracle over {len(dec)} sequences took {time.time() - t0:.1f} s")
    assert_close(out[dec], ref, f"full decode {w.name} (all {len(dec)} decoding sequences)")


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


def test_full_prefill_rows(full):
    """Every row of the session with the longest history; in every other session the first 32, the last
    32 and a seeded block of 32 rows (rows are independent, so each is checked exactly as in the full
    result).  One session's rows also go through the oracle's own all-head call."""
    import time
    c, w = full, full.w
    if not len(w.prefill_seqs):
        pytest.skip("workload has no prefill chunk")
    note(f"full prefill {w.name}")
    out = c.prefill().cpu().numpy().astype(np.float64)
    assert c.pool.device_error() == kp.KVP_OK
    qp = W.to_numpy_bits(c.vals.qp)
    cu = w.cu_q()
    rng = np.random.default_rng(5)
    longest = int(np.argmax(w.prefill_ctx))
    t0 = time.time()
    for j in range(len(w.prefill_seqs)):
        C, ctx, seq = int(w.prefill_chunk[j]), int(w.prefill_ctx[j]), int(w.prefill_seqs[j])
        k, v = W.seq_kv_bits(w, c.vals, seq, ctx + C)
        if j == longest:
            blocks = [(0, C)]
        else:
            mid = int(rng.integers(32, max(33, C - 64)))
            blocks = [(0, min(32, C)), (mid, min(mid + 32, C)), (max(0, C - 32), C)]
        for r0, r1 in blocks:
            ref = oracle_by_kv_head(oracle.prefill_seq, qp[cu[j] + r0:cu[j] + r1], k, v, w.scale, ctx + r0)
            if j == 0 and r0 == 0:
                n_own = min(32, r1)
                own = oracle.prefill_seq(qp[cu[j]:cu[j] + n_own], oracle.widen_bf16(k), oracle.widen_bf16(v), w.scale,
                                         ctx)
                assert np.max(np.abs(ref[:n_own] - own)) <= 1e-12
            assert_close(out[cu[j] + r0:cu[j] + r1], ref,
                         f"full prefill {w.name} session {j} rows {r0}..{r1 - 1} (ctx {ctx})")
    note(f"full prefill {w.name}: oracle took {time.time() - t0:.1f} s")


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
