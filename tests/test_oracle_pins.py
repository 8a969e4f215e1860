"""Pins of the CPU fp64 oracle against things other than itself (CPU only).

* brute force in pure Python (no numpy) on tiny inputs;
* torch float64 scaled_dot_product_attention on the contiguous gather (library special case);
* closed forms (equal values, equal keys, zero query, one key, hand-derived examples);
* invariances the method fixes: physical page permutation, shared vs duplicated prefix pages,
  split-at-any-page-boundary + log-sum-exp merge, prefill chunking and ctx = 0;
* planted mistakes: plausible bugs put into a copy of the oracle must make a pin fail.
"""
import math
import os
import struct

import numpy as np
import pytest
import torch

import oracle
from oracle import paged_attention as OP
from paper_2608_11152_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------------------------------------
# helpers (pure Python where it matters)
# ------------------------------------------------------------------------------------------------

def py_bf16(bits: int) -> float:
    return struct.unpack(">f", struct.pack(">I", (int(bits) & 0xFFFF) << 16))[0]


def py_attend(q, ks, vs, scale):
    """Pure-Python softmax attention for one head (lists of floats)."""
    if not ks:
        return [0.0] * len(vs[0]) if vs else [0.0] * len(q)
    s = [scale * sum(a * b for a, b in zip(q, k)) for k in ks]
    m = max(s)
    w = [math.exp(x - m) for x in s]
    tot = sum(w)
    d = len(vs[0])
    return [sum(w[t] * vs[t][c] for t in range(len(ks))) / tot for c in range(d)]


def py_decode(q_bits, pool_k, pool_v, bt, seq_lens, scale):
    """Brute-force paged decode: nested Python loops over sequences, heads, tokens."""
    B, Hq, d = q_bits.shape
    Hkv = pool_k.shape[1]
    out = []
    for i in range(B):
        row = []
        for h in range(Hq):
            g = h // (Hq // Hkv)
            ks, vs = [], []
            for t in range(int(seq_lens[i])):
                page, slot = int(bt[i][t // 16]), t % 16
                ks.append([py_bf16(x) for x in pool_k[page, g, slot].tolist()])
                vs.append([py_bf16(x) for x in pool_v[page, g, slot].tolist()])
            q = [py_bf16(x) for x in q_bits[i, h].tolist()]
            row.append(py_attend(q, ks, vs, scale) if ks else [0.0] * d)
        out.append(row)
    return np.array(out)


def build_pool(w, vals):
    """Run every append of the workload through the oracle's own append (setup, then step)."""
    pk, pv = oracle.new_pool(w.num_pages, w.Hkv, w.d)
    for ab in w.setup_appends + w.step_appends:
        kv = vals.kv[ab.src_rows]
        oracle.append(pk, pv, kv[:, 0], kv[:, 1], w.block_tables, ab.start_pos, ab.cu_new)
    return pk, pv


def rand_bits(rng, shape):
    return W.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def small_case(rng, B=3, Hq=4, Hkv=2, d=8, lens=(5, 17, 33), num_pages=16):
    perm = rng.permutation(num_pages)
    maxp = max((n + 15) // 16 for n in lens)
    bt = np.full((B, maxp), -1, np.int32)
    nxt = 0
    for i, n in enumerate(lens):
        k = (n + 15) // 16
        bt[i, :k] = perm[nxt:nxt + k]
        nxt += k
    pk, pv = oracle.new_pool(num_pages, Hkv, d)
    T = sum(lens)
    k = rand_bits(rng, (T, Hkv, d))
    v = rand_bits(rng, (T, Hkv, d))
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    oracle.append(pk, pv, k, v, bt, np.zeros(B, np.int32), cu)
    q = rand_bits(rng, (B, Hq, d))
    return q, pk, pv, bt, np.asarray(lens, np.int32), k, v, cu


# ------------------------------------------------------------------------------------------------
# p-1 brute force
# ------------------------------------------------------------------------------------------------

def test_brute_force_tiny_config():
    w = W.make_workload("tiny")
    vals = W.make_values(w)
    pk, pv = build_pool(w, vals)
    ref = oracle.decode(vals.q, pk, pv, w.block_tables, w.decode_len, w.scale)
    bf = py_decode(vals.q, pk, pv, w.block_tables, w.decode_len, w.scale)
    assert np.max(np.abs(ref - bf)) <= 1e-12


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_brute_force_random_small(seed):
    rng = np.random.default_rng(seed)
    lens = tuple(int(x) for x in rng.integers(1, 40, size=4))
    q, pk, pv, bt, sl, *_ = small_case(rng, B=4, Hq=6, Hkv=3, d=5, lens=lens, num_pages=20)
    ref = oracle.decode(q, pk, pv, bt, sl, 0.37)
    bf = py_decode(q, pk, pv, bt, sl, 0.37)
    assert np.max(np.abs(ref - bf)) <= 1e-12


def test_brute_force_prefill():
    rng = np.random.default_rng(11)
    Hq, Hkv, d, ctx, C = 4, 2, 8, 21, 6
    n = ctx + C
    q, pk, pv, bt, sl, k, v, cu = small_case(rng, B=1, Hq=Hq, Hkv=Hkv, d=d, lens=(n,), num_pages=4)
    qp = rand_bits(rng, (C, Hq, d))
    ref = oracle.prefill(qp, pk, pv, bt, np.array([ctx], np.int32), np.array([0, C], np.int32), 0.25)
    for j in range(C):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            ks = [[py_bf16(x) for x in k[t, g].tolist()] for t in range(ctx + j + 1)]
            vs = [[py_bf16(x) for x in v[t, g].tolist()] for t in range(ctx + j + 1)]
            qq = [py_bf16(x) for x in qp[j, h].tolist()]
            assert np.max(np.abs(np.array(py_attend(qq, ks, vs, 0.25)) - ref[j, h])) <= 1e-12


# ------------------------------------------------------------------------------------------------
# p-2 library special case: torch float64 SDPA with GQA-expanded K/V
# ------------------------------------------------------------------------------------------------

def _sdpa(q, k, v, scale, mask=None):
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), attn_mask=mask, scale=scale).numpy()


def test_torch_sdpa_decode():
    w = W.make_workload("tiny")
    vals = W.make_values(w)
    pk, pv = build_pool(w, vals)
    ref = oracle.decode(vals.q, pk, pv, w.block_tables, w.decode_len, w.scale)
    for i in range(w.B):
        k, v = W.seq_kv_bits(w, vals, i, int(w.decode_len[i]))
        kk = np.repeat(OP.widen_bf16(k).transpose(1, 0, 2), w.G, axis=0)  # [Hq, n, d]
        vv = np.repeat(OP.widen_bf16(v).transpose(1, 0, 2), w.G, axis=0)
        qq = OP.widen_bf16(vals.q[i])[:, None, :]
        got = _sdpa(qq, kk, vv, w.scale)[:, 0]
        assert np.max(np.abs(got - ref[i])) <= 1e-12


def test_torch_sdpa_prefill_with_context():
    w = W.make_workload("agentic_s")
    vals = W.make_values(w)
    pk, pv = build_pool(w, vals)
    i = 0
    ctx, C = int(w.prefill_ctx[i]), int(w.prefill_chunk[i])
    rows = np.r_[0:40, C - 40:C]
    k, v = W.seq_kv_bits(w, vals, int(w.prefill_seqs[i]), ctx + C)
    ref = oracle.prefill_seq(vals.qp[:C], OP.widen_bf16(k), OP.widen_bf16(v), w.scale, ctx, rows=rows)
    kk = np.repeat(OP.widen_bf16(k).transpose(1, 0, 2), w.G, axis=0)
    vv = np.repeat(OP.widen_bf16(v).transpose(1, 0, 2), w.G, axis=0)
    qq = OP.widen_bf16(vals.qp[rows]).transpose(1, 0, 2)  # [Hq, R, d]
    allowed = np.arange(ctx + C)[None, :] <= (ctx + rows)[:, None]
    got = _sdpa(qq, kk, vv, w.scale, mask=torch.from_numpy(allowed)).transpose(1, 0, 2)
    assert np.max(np.abs(got - ref)) <= 1e-12


# ------------------------------------------------------------------------------------------------
# p-3 closed forms
# ------------------------------------------------------------------------------------------------

def _one_seq_pool(k, v):
    """Pool with one sequence holding k, v ([n, Hkv, d] float values exactly representable)."""
    n, Hkv, d = k.shape
    npg = (n + 15) // 16 + 2
    pk, pv = oracle.new_pool(npg, Hkv, d)
    bt = np.arange(npg - 1, -1, -1, dtype=np.int32)[None, : (n + 15) // 16]
    kb = W.f32_to_bf16_bits(k.astype(np.float32))
    vb = W.f32_to_bf16_bits(v.astype(np.float32))
    oracle.append(pk, pv, kb, vb, bt, np.zeros(1, np.int32), np.array([0, n], np.int32))
    return pk, pv, bt


def test_closed_form_equal_values():
    rng = np.random.default_rng(5)
    n, Hkv, d, Hq = 70, 2, 16, 4
    c = W.bf16_bits_to_f32(rand_bits(rng, (Hkv, d))).astype(np.float64)
    pk, pv, bt = _one_seq_pool(rng.standard_normal((n, Hkv, d)), np.broadcast_to(c, (n, Hkv, d)).copy())
    q = rand_bits(rng, (1, Hq, d))
    out = oracle.decode(q, pk, pv, bt, [n], 1 / 4)
    for h in range(Hq):
        assert np.max(np.abs(out[0, h] - c[h // 2])) <= 1e-14


def test_closed_form_equal_keys_and_zero_query():
    rng = np.random.default_rng(6)
    n, Hkv, d, Hq = 45, 1, 8, 2
    kval = np.broadcast_to(rng.standard_normal((1, Hkv, d)), (n, Hkv, d)).copy()
    v = rng.standard_normal((n, Hkv, d))
    pk, pv, bt = _one_seq_pool(kval, v)
    vb = OP.widen_bf16(W.f32_to_bf16_bits(v.astype(np.float32)))
    mean_v = vb[:, 0].mean(axis=0)
    q = rand_bits(rng, (1, Hq, d))
    out = oracle.decode(q, pk, pv, bt, [n], 0.3)
    assert np.max(np.abs(out[0] - mean_v)) <= 1e-13
    # q = 0 with arbitrary keys: uniform weights as well
    pk2, pv2, bt2 = _one_seq_pool(rng.standard_normal((n, Hkv, d)), v)
    out0 = oracle.decode(np.zeros((1, Hq, d), np.uint16), pk2, pv2, bt2, [n], 0.3)
    assert np.max(np.abs(out0[0] - mean_v)) <= 1e-13


def test_closed_form_single_token_and_empty():
    rng = np.random.default_rng(7)
    q, pk, pv, bt, sl, k, v, cu = small_case(rng, B=2, lens=(1, 9), num_pages=4)
    out = oracle.decode(q, pk, pv, bt, np.array([1, 0], np.int32), 0.5)
    for h in range(q.shape[1]):
        assert np.array_equal(out[0, h], OP.widen_bf16(v[0, h // 2]))
    assert np.all(out[1] == 0.0)


def test_hand_derived_examples():
    with open(os.path.join(GOLDEN, "hand_examples.txt")) as f:
        lines = [l for l in f if l.strip() and not l.startswith("#")]
    env = {"exp": math.exp, "sqrt": math.sqrt}
    assert len(lines) == 3
    for line in lines:
        name, q, ks, vs, exp = [x.strip() for x in line.split("|")]
        qv = np.array([[float(x) for x in q.split(",")]])
        kv = np.array([[float(x) for x in r.split(",")] for r in ks.split(";")])
        vv = np.array([[float(x) for x in r.split(",")] for r in vs.split(";")])
        want = np.array([eval(e, env) for e in exp.split(", ")])
        pk, pv, bt = _one_seq_pool(kv[:, None, :], vv[:, None, :])
        qb = W.f32_to_bf16_bits(qv[None].astype(np.float32))
        out = oracle.decode(qb, pk, pv, bt, [len(kv)], 1 / math.sqrt(2))
        assert np.max(np.abs(out[0, 0] - want)) <= 1e-15, name


# ------------------------------------------------------------------------------------------------
# p-4 physical page permutation, p-5 shared vs duplicated prefix pages, p-8 append round trip
# ------------------------------------------------------------------------------------------------

def test_page_permutation_invariance_bitwise():
    w = W.make_workload("rlvr_d64")
    vals = W.make_values(w)
    pk, pv = build_pool(w, vals)
    ref = oracle.decode(vals.q, pk, pv, w.block_tables, w.decode_len, w.scale)
    perm = np.random.default_rng(3).permutation(w.num_pages)
    pk2, pv2 = np.empty_like(pk), np.empty_like(pv)
    pk2[perm], pv2[perm] = pk, pv
    bt2 = np.where(w.block_tables >= 0, perm[np.maximum(w.block_tables, 0)], -1)
    got = oracle.decode(vals.q, pk2, pv2, bt2, w.decode_len, w.scale)
    assert np.array_equal(ref, got)


def test_shared_vs_duplicated_prefix_bitwise():
    w = W.make_workload("rlvr_d64")
    vals = W.make_values(w)
    pk, pv = build_pool(w, vals)
    ref = oracle.decode(vals.q, pk, pv, w.block_tables, w.decode_len, w.scale)
    # give every non-representative member its own copy of the shared pages
    extra = int(sum(w.shared_pages[g] * (np.sum(w.group_id == g) - 1) for g in range(w.num_groups)))
    pk2 = np.concatenate([pk, np.zeros((extra,) + pk.shape[1:], pk.dtype)])
    pv2 = np.concatenate([pv, np.zeros((extra,) + pv.shape[1:], pv.dtype)])
    bt2 = w.block_tables.copy()
    nxt = w.num_pages
    seen = set()
    for i in range(w.B):
        g = int(w.group_id[i])
        if g < 0:
            continue
        if g not in seen:
            seen.add(g)
            continue
        for j in range(int(w.shared_pages[g])):
            pk2[nxt], pv2[nxt] = pk[bt2[i, j]], pv[bt2[i, j]]
            bt2[i, j] = nxt
            nxt += 1
    assert nxt == len(pk2)
    got = oracle.decode(vals.q, pk2, pv2, bt2, w.decode_len, w.scale)
    assert np.array_equal(ref, got)


def test_append_round_trip_bitwise():
    w = W.make_workload("mixed_s")
    vals = W.make_values(w)
    pk, pv = build_pool(w, vals)
    for i in range(w.B):
        k, v = W.seq_kv_bits(w, vals, i)
        n = int(w.final_len[i])
        pos = np.arange(n)
        pages = w.block_tables[i][pos // 16]
        assert np.array_equal(pk[pages, :, pos % 16, :], k)
        assert np.array_equal(pv[pages, :, pos % 16, :], v)


# ------------------------------------------------------------------------------------------------
# p-6 split at any page boundary + log-sum-exp merge == unsplit
# ------------------------------------------------------------------------------------------------

def _partial(q, k, v, scale):
    """(m, l, acc) of one key range for one head, in fp64 (the quantities a split-KV plan carries)."""
    if k.shape[0] == 0:
        return -np.inf, 0.0, np.zeros(v.shape[1])
    s = scale * (k @ q)
    m = s.max()
    w = np.exp(s - m)
    return m, w.sum(), w @ v


def _merge(parts):
    m = max(p[0] for p in parts)
    if m == -np.inf:
        return np.zeros_like(parts[0][2])
    l = sum(p[1] * math.exp(p[0] - m) for p in parts if p[1] > 0)
    acc = sum(p[2] * math.exp(p[0] - m) for p in parts if p[1] > 0)
    return acc / l


@pytest.mark.parametrize("seed", [0, 1])
def test_lse_merge_associativity(seed):
    rng = np.random.default_rng(seed)
    n, d = 16 * 13 + 5, 32
    k = OP.widen_bf16(rand_bits(rng, (n, d)))
    v = OP.widen_bf16(rand_bits(rng, (n, d)))
    q = OP.widen_bf16(rand_bits(rng, (d,)))
    ref = oracle.attend(q[None], k, v, 0.2)[0]
    for _ in range(5):
        cuts = sorted(set(rng.integers(0, n // 16 + 1, size=4).tolist()))
        bounds = [0] + [16 * c for c in cuts] + [n]
        parts = [_partial(q, k[a:b], v[a:b], 0.2) for a, b in zip(bounds[:-1], bounds[1:])]
        parts.append(_partial(q, k[:0], v[:0], 0.2))  # an empty range is neutral
        assert np.max(np.abs(_merge(parts) - ref)) <= 1e-12


# ------------------------------------------------------------------------------------------------
# p-7 prefill reductions
# ------------------------------------------------------------------------------------------------

def test_prefill_chunk_of_one_equals_decode():
    rng = np.random.default_rng(21)
    q, pk, pv, bt, sl, *_ = small_case(rng, B=3, Hq=4, Hkv=2, d=8, lens=(9, 30, 47), num_pages=12)
    dec = oracle.decode(q, pk, pv, bt, sl, 0.3)
    pre = oracle.prefill(q, pk, pv, bt, sl - 1, np.arange(4, dtype=np.int32), 0.3)
    assert np.max(np.abs(dec - pre)) <= 1e-15


def test_prefill_two_chunks_equal_one():
    w = W.make_workload("agentic_s")
    vals = W.make_values(w)
    i, seq = 1, int(w.prefill_seqs[1])
    ctx, C = int(w.prefill_ctx[i]), int(w.prefill_chunk[i])
    k, v = W.seq_kv_bits(w, vals, seq, ctx + C)
    k, v = OP.widen_bf16(k), OP.widen_bf16(v)
    a = int(w.cu_q()[i])
    qi = vals.qp[a:a + C]
    one = oracle.prefill_seq(qi, k, v, w.scale, ctx)
    h = C // 2
    first = oracle.prefill_seq(qi[:h], k, v, w.scale, ctx)
    second = oracle.prefill_seq(qi[h:], k, v, w.scale, ctx + h)
    assert np.max(np.abs(np.concatenate([first, second]) - one)) <= 1e-13


def test_prefill_ctx0_is_causal_attention():
    rng = np.random.default_rng(8)
    C, Hq, Hkv, d = 37, 4, 1, 16
    q, pk, pv, bt, sl, k, v, cu = small_case(rng, B=1, Hq=Hq, Hkv=Hkv, d=d, lens=(C,), num_pages=5)
    qp = rand_bits(rng, (C, Hq, d))
    ref = oracle.prefill(qp, pk, pv, bt, np.array([0], np.int32), np.array([0, C], np.int32), 0.25)
    kk = np.repeat(OP.widen_bf16(k).transpose(1, 0, 2), Hq, axis=0)
    vv = np.repeat(OP.widen_bf16(v).transpose(1, 0, 2), Hq, axis=0)
    got = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(OP.widen_bf16(qp).transpose(1, 0, 2)), torch.from_numpy(kk), torch.from_numpy(vv),
        is_causal=True, scale=0.25).numpy().transpose(1, 0, 2)
    assert np.max(np.abs(got - ref)) <= 1e-12


# ------------------------------------------------------------------------------------------------
# planted mistakes: each plausible bug in a copy of the oracle must fail a pin above
# ------------------------------------------------------------------------------------------------

def _tiny_brute():
    w = W.make_workload("tiny")
    vals = W.make_values(w)
    pk, pv = build_pool(w, vals)
    return w, vals, pk, pv, py_decode(vals.q, pk, pv, w.block_tables, w.decode_len, w.scale)


@pytest.mark.parametrize("mistake", ["gqa_modulo", "slot_swap", "no_scale", "transposed_v", "drop_last"])
def test_planted_mistakes_are_caught(monkeypatch, mistake):
    w, vals, pk, pv, bf = _tiny_brute()
    if mistake == "gqa_modulo":
        monkeypatch.setattr(OP, "kv_head_of", lambda h, hq, hkv: h % hkv)
    elif mistake == "slot_swap":
        def bad_gather(pool_k, pool_v, row, n):
            pos = np.arange(n)
            pages = np.asarray(row, dtype=np.int64)[pos // 16]
            slots = (pos % 16) ^ 1
            return OP.widen_bf16(pool_k[pages, :, slots, :]), OP.widen_bf16(pool_v[pages, :, slots, :])
        monkeypatch.setattr(OP, "gather", bad_gather)
    elif mistake == "no_scale":
        real = OP.attend
        monkeypatch.setattr(OP, "attend", lambda q, k, v, s: real(q, k, v, 1.0))
    elif mistake == "transposed_v":
        def bad_attend(q, k, v, scale):
            s = scale * (q @ k.T)
            w_ = np.exp(s - s.max(axis=1, keepdims=True))
            return (w_ @ k) / w_.sum(axis=1, keepdims=True)
        monkeypatch.setattr(OP, "attend", bad_attend)
    elif mistake == "drop_last":
        real = OP.attend
        monkeypatch.setattr(OP, "attend", lambda q, k, v, s: real(q, k[:-1], v[:-1], s))
    got = OP.decode(vals.q, pk, pv, w.block_tables, w.decode_len, w.scale)
    assert np.max(np.abs(got - bf)) > 1e-6


def test_planted_causal_off_by_one_is_caught(monkeypatch):
    rng = np.random.default_rng(9)
    q, pk, pv, bt, sl, *_ = small_case(rng, B=1, Hq=2, Hkv=1, d=8, lens=(30,), num_pages=3)
    dec = oracle.decode(q, pk, pv, bt, sl, 0.3)
    real = OP.attend_causal
    monkeypatch.setattr(OP, "attend_causal", lambda q_, k, v, s, fp: real(q_, k, v, s, fp - 1))
    pre = OP.prefill(q, pk, pv, bt, sl - 1, np.array([0, 1], np.int32), 0.3)
    assert np.max(np.abs(dec - pre)) > 1e-6


# ------------------------------------------------------------------------------------------------
# host KV tier (Sec. 5.5): eviction to the host and restore into other physical pages changes nothing
# ------------------------------------------------------------------------------------------------

def test_tier_restore_elsewhere_is_invisible():
    """Offload every used page, wipe them, restore each into an unused page with the block tables
    patched: gathers and decode are bitwise unchanged (attention never sees where a page lives).
    Restoring over the original pages after the wipe gives back the same pool."""
    rng = np.random.default_rng(5)
    q, pk, pv, bt, lens, *_ = small_case(rng, num_pages=32)
    ref = oracle.decode(q, pk, pv, bt, lens, 0.3)
    used = [int(x) for x in np.unique(bt[bt >= 0])]
    free = [p for p in range(32) if p not in used]
    hk, hv = oracle.offload(pk, pv, used)
    assert hk.shape == (len(used),) + pk.shape[1:] and hv.shape == hk.shape
    assert np.array_equal(hk, pk[used]) and np.array_equal(hv, pv[used])
    pk2, pv2, bt2 = pk.copy(), pv.copy(), bt.copy()
    pk2[used] = 0
    pv2[used] = 0
    dst = [int(x) for x in rng.permutation(free)[: len(used)]]
    rows, lps = [], []
    for p in used:  # every page of small_case is referenced by exactly one (row, logical page)
        i, lp = (int(x) for x in np.argwhere(bt == p)[0])
        rows.append(i)
        lps.append(lp)
    oracle.restore(pk2, pv2, dst, hk, hv, bt2, rows, lps)
    for j, p in enumerate(used):
        assert bt2[rows[j], lps[j]] == dst[j] and bt[rows[j], lps[j]] == p
    for i, n in enumerate(lens):
        a = oracle.gather(pk, pv, bt[i], int(n))
        b = oracle.gather(pk2, pv2, bt2[i], int(n))
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert np.array_equal(oracle.decode(q, pk2, pv2, bt2, lens, 0.3), ref)
    pk3, pv3 = pk.copy(), pv.copy()
    pk3[used] = 0
    pv3[used] = 0
    oracle.restore(pk3, pv3, used, hk, hv)
    assert np.array_equal(pk3, pk) and np.array_equal(pv3, pv)
