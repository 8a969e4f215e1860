"""Pins of the FP8 (OCP E4M3) KV quantisation oracle (CPU only): the code table and the rounding against
torch's float8_e4m3fn (a library special case of the same format), the saturation convention, and
attention over an FP8 pool against the pinned bf16 oracle on the same (dequantised) values."""
import numpy as np
import pytest
import torch

import oracle
from oracle import fp8 as F
from paper_2608_11152_amd import workloads as W


def test_code_table_matches_torch():
    codes = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    v = F.code_values()
    same = (codes == v) | (np.isnan(codes) & np.isnan(v))
    assert same.all()
    assert v[0x7E] == 448.0 and v[0x01] == 2.0 ** -9 and v[0x08] == 2.0 ** -6 and np.isnan(v[0x7F])


def test_rounding_matches_torch_in_range():
    rng = np.random.default_rng(31)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * s for s in (1e-3, 0.02, 0.7, 9, 120)])
    mags = F.code_values()[:127]
    mids = ((mags[1:] + mags[:-1]) / 2).astype(np.float32)  # exact ties between neighbours
    x = np.concatenate([x, mids, -mids, np.array([0.0, -0.0, 448, -448, 464, -464], np.float32)])
    x = x[np.abs(x) <= 464]
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(F.encode(x.astype(np.float64)), ref)


def test_saturation_and_round_trip():
    big = np.array([465.0, 480.0, 1e6, np.inf, -500.0, -np.inf])
    assert list(F.encode(big)) == [0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0xFE]
    assert (F.encode(np.array([np.nan])) & 0x7F)[0] == 0x7F
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    assert np.array_equal(F.encode(F.code_values()[codes]), codes)


@pytest.mark.parametrize("scale", [1.0, 0.5, 0.37, 3.0])
def test_quantize_and_dequantize_match_torch(scale):
    rng = np.random.default_rng(32)
    bits = W.f32_to_bf16_bits(rng.standard_normal(50000, dtype=np.float32) * 2)
    x = (bits.astype(np.uint32) << 16).view(np.float32)
    y = x * (np.float32(1.0) / np.float32(scale))
    keep = np.abs(y) <= 464
    ref = torch.from_numpy(y[keep]).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    codes = F.quantize_bf16(bits, scale)
    assert np.array_equal(codes[keep], ref)
    back = F.dequantize_bf16(codes, scale)
    tb = (torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).to(torch.float32) * torch.tensor(np.float32(scale)))
    assert np.array_equal(back, tb.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16))


def test_planted_mistake_ties_away_is_caught():
    mags = F.code_values()[:127]
    mids = (mags[1:] + mags[:-1]) / 2
    away = np.searchsorted(mags, mids, side="left")  # rounding ties up would give the upper code
    even = F.encode(mids)
    assert (away != even).any()


@pytest.mark.parametrize("scale", [1.0, 0.25])
def test_fp8_attention_equals_bf16_oracle_on_dequantised_values(scale):
    """With a power-of-two scale every dequantised value is a bf16 value, so attention over the FP8
    pool must equal, bitwise, the bf16 oracle over a pool holding those values."""
    w = W.make_workload("tiny")
    vals = W.make_values(w)
    ck, cv = F.new_pool(w.num_pages, w.Hkv, w.d)
    bk, bv = oracle.new_pool(w.num_pages, w.Hkv, w.d)
    for ab in w.setup_appends + w.step_appends:
        kv = vals.kv[ab.src_rows]
        F.append(ck, cv, kv[:, 0], kv[:, 1], w.block_tables, ab.start_pos, ab.cu_new, scale, scale)
        kd = F.dequantize_bf16(F.quantize_bf16(kv[:, 0], scale), scale)
        vd = F.dequantize_bf16(F.quantize_bf16(kv[:, 1], scale), scale)
        oracle.append(bk, bv, kd, vd, w.block_tables, ab.start_pos, ab.cu_new)
    a = F.decode(vals.q, ck, cv, w.block_tables, w.decode_len, w.scale, scale, scale)
    b = oracle.decode(vals.q, bk, bv, w.block_tables, w.decode_len, w.scale)
    assert np.array_equal(a, b)


# ------------------------------------------------------------------------------------------------
# Attention over an FP8 pool: pinned against the bf16 oracle (power-of-two scales, where dequantised
# values are bf16 values), against itself at chunk size one, and against pure-Python brute force (every
# code decoded from its bits, nearest-code search with ties to the even mantissa, math.exp softmax) at
# scales that are not powers of two.
# ------------------------------------------------------------------------------------------------

import math  # noqa: E402
import struct  # noqa: E402


def _fl32(x: float) -> float:
    """Round a Python float to binary32 (struct packs with round-to-nearest-even)."""
    return struct.unpack("<f", struct.pack("<f", x))[0]


def _py_bf16(bits: int) -> float:
    return struct.unpack(">f", struct.pack(">I", (int(bits) & 0xFFFF) << 16))[0]


def _py_code_value(c: int) -> float:
    """Value of an E4M3 code from its bits: sign, 4 exponent bits (bias 7), 3 mantissa bits."""
    sign = -1.0 if c & 0x80 else 1.0
    e, m = (c >> 3) & 15, c & 7
    if e == 15 and m == 7:
        return float("nan")
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** -6
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


_PY_FINITE = [(c, _py_code_value(c)) for c in range(127)]  # non-negative finite codes


def _py_quantize(bits: int, scale: float) -> int:
    """Brute force: y = fp32(fp32(x) * fp32(1 / fp32(scale))); the nearest non-negative finite code to |y|
    (ties to the code with an even mantissa, i.e. an even code), then the sign bit."""
    x = _py_bf16(bits)
    y = _fl32(x * _fl32(1.0 / _fl32(scale)))
    a = abs(y)
    best, bd = None, None
    for c, v in _PY_FINITE:
        dist = abs(v - a)
        if bd is None or dist < bd or (dist == bd and c % 2 == 0):
            best, bd = c, dist
    return best | (0x80 if math.copysign(1.0, y) < 0 else 0)


def _py_attend(q, ks, vs, scale):
    s = [scale * sum(a * b for a, b in zip(q, k)) for k in ks]
    m = max(s)
    w = [math.exp(x - m) for x in s]
    tot = sum(w)
    return [sum(w[t] * vs[t][c] for t in range(len(ks))) / tot for c in range(len(vs[0]))]


def _small_fp8_case(rng, lens, Hq=4, Hkv=2, d=8, num_pages=None, ks=1.0, vs=1.0):
    num_pages = num_pages or sum((n + 15) // 16 for n in lens) + 3
    perm = rng.permutation(num_pages)
    maxp = max((n + 15) // 16 for n in lens)
    bt = np.full((len(lens), maxp), -1, np.int32)
    nxt = 0
    for i, n in enumerate(lens):
        k = (n + 15) // 16
        bt[i, :k] = perm[nxt:nxt + k]
        nxt += k
    T = sum(lens)
    kb = W.f32_to_bf16_bits(rng.standard_normal((T, Hkv, d), dtype=np.float32) * 1.7)
    vb = W.f32_to_bf16_bits(rng.standard_normal((T, Hkv, d), dtype=np.float32) * 1.7)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    ck, cv = F.new_pool(num_pages, Hkv, d)
    F.append(ck, cv, kb, vb, bt, np.zeros(len(lens), np.int32), cu, ks, vs)
    return bt, kb, vb, cu, ck, cv


def _py_seq_kv(kb, vb, cu, i, n, ks, vs, g):
    """Brute-force dequantised K, V rows of KV head g for the first n tokens of sequence i."""
    K = [[_py_code_value(_py_quantize(x, ks)) * _fl32(ks) for x in kb[cu[i] + t, g].tolist()] for t in range(n)]
    V = [[_py_code_value(_py_quantize(x, vs)) * _fl32(vs) for x in vb[cu[i] + t, g].tolist()] for t in range(n)]
    return K, V


@pytest.mark.parametrize("ks,vs", [(1.0, 1.0), (0.25, 2.0), (4.0, 0.5)])
def test_fp8_prefill_equals_bf16_oracle_on_dequantised_values(ks, vs):
    """Power-of-two scales: every dequantised value is a bf16 value, so the FP8 prefill must equal,
    bitwise, the bf16 oracle's prefill over a pool holding those values."""
    rng = np.random.default_rng(41)
    lens = (37, 70, 18)
    C = np.array([5, 16, 18])
    ctx = np.array(lens) - C
    bt, kb, vb, cu, ck, cv = _small_fp8_case(rng, lens, ks=ks, vs=vs)
    bk, bv = oracle.new_pool(ck.shape[0], 2, 8)
    kd = F.dequantize_bf16(F.quantize_bf16(kb, ks), ks)
    vd = F.dequantize_bf16(F.quantize_bf16(vb, vs), vs)
    oracle.append(bk, bv, kd, vd, bt, np.zeros(3, np.int32), cu)
    assert np.array_equal(oracle.widen_bf16(kd), F.dequantize(F.quantize_bf16(kb, ks), ks))  # exact in bf16
    qp = W.f32_to_bf16_bits(rng.standard_normal((int(C.sum()), 4, 8), dtype=np.float32))
    cq = np.concatenate([[0], np.cumsum(C)]).astype(np.int32)
    a = F.prefill(qp, ck, cv, bt, ctx, cq, 0.3, ks, vs)
    b = oracle.prefill(qp, bk, bv, bt, ctx, cq, 0.3)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("ks,vs", [(0.37, 1.9), (1.3, 0.6)])
def test_fp8_prefill_chunk_of_one_equals_decode(ks, vs):
    rng = np.random.default_rng(42)
    lens = (9, 30, 47)
    bt, kb, vb, cu, ck, cv = _small_fp8_case(rng, lens, ks=ks, vs=vs)
    q = W.f32_to_bf16_bits(rng.standard_normal((3, 4, 8), dtype=np.float32))
    sl = np.array(lens, np.int32)
    dec = F.decode(q, ck, cv, bt, sl, 0.3, ks, vs)
    pre = F.prefill(q, ck, cv, bt, sl - 1, np.arange(4, dtype=np.int32), 0.3, ks, vs)
    assert np.max(np.abs(dec - pre)) <= 1e-15


@pytest.mark.parametrize("ks,vs", [(0.37, 1.9), (1.3, 0.6), (0.5, 2.0)])
def test_fp8_decode_brute_force(ks, vs):
    rng = np.random.default_rng(43)
    lens = (5, 17, 33)
    Hq, Hkv, d = 4, 2, 8
    bt, kb, vb, cu, ck, cv = _small_fp8_case(rng, lens, ks=ks, vs=vs)
    q = W.f32_to_bf16_bits(rng.standard_normal((3, Hq, d), dtype=np.float32))
    ref = F.decode(q, ck, cv, bt, np.array(lens, np.int32), 0.41, ks, vs)
    for i, n in enumerate(lens):
        for h in range(Hq):
            K, V = _py_seq_kv(kb, vb, cu, i, n, ks, vs, h // (Hq // Hkv))
            got = _py_attend([_py_bf16(x) for x in q[i, h].tolist()], K, V, 0.41)
            assert np.max(np.abs(np.array(got) - ref[i, h])) <= 1e-12


@pytest.mark.parametrize("ks,vs", [(0.37, 1.9), (1.3, 0.6)])
def test_fp8_prefill_brute_force(ks, vs):
    rng = np.random.default_rng(44)
    Hq, Hkv, d = 4, 2, 8
    lens = (29, 23)
    C = np.array([7, 23])  # the second session has no history (ctx = 0)
    ctx = np.array(lens) - C
    bt, kb, vb, cu, ck, cv = _small_fp8_case(rng, lens, ks=ks, vs=vs)
    qp = W.f32_to_bf16_bits(rng.standard_normal((int(C.sum()), Hq, d), dtype=np.float32))
    cq = np.concatenate([[0], np.cumsum(C)]).astype(np.int32)
    ref = F.prefill(qp, ck, cv, bt, ctx, cq, 0.27, ks, vs)
    for i in range(2):
        for j in range(int(C[i])):
            for h in range(Hq):
                K, V = _py_seq_kv(kb, vb, cu, i, int(ctx[i]) + j + 1, ks, vs, h // (Hq // Hkv))
                got = _py_attend([_py_bf16(x) for x in qp[cq[i] + j, h].tolist()], K, V, 0.27)
                assert np.max(np.abs(np.array(got) - ref[cq[i] + j, h])) <= 1e-12


def test_fp8_quantizer_brute_force_at_odd_scales():
    """The vectorised quantiser equals the brute-force nearest-code search at non-power-of-two scales."""
    rng = np.random.default_rng(45)
    bits = W.f32_to_bf16_bits(rng.standard_normal(3000, dtype=np.float32) * 40)
    for s in (0.37, 1.9, 1.3, 0.6, 0.011):
        got = F.quantize_bf16(bits, s)
        assert [int(c) for c in got] == [_py_quantize(int(b), s) for b in bits]


def _planted_case(ks=0.37, vs=1.9):
    rng = np.random.default_rng(46)
    Hq, Hkv, d = 4, 2, 8
    lens = (21, 40)
    C = np.array([6, 9])
    ctx = np.array(lens) - C
    bt, kb, vb, cu, ck, cv = _small_fp8_case(rng, lens, ks=ks, vs=vs)
    qp = W.f32_to_bf16_bits(rng.standard_normal((int(C.sum()), Hq, d), dtype=np.float32))
    cq = np.concatenate([[0], np.cumsum(C)]).astype(np.int32)
    brute = np.zeros((int(C.sum()), Hq, d))
    for i in range(2):
        for j in range(int(C[i])):
            for h in range(Hq):
                K, V = _py_seq_kv(kb, vb, cu, i, int(ctx[i]) + j + 1, ks, vs, h // (Hq // Hkv))
                brute[cq[i] + j, h] = _py_attend([_py_bf16(x) for x in qp[cq[i] + j, h].tolist()], K, V, 0.27)
    return (qp, ck, cv, bt, ctx, cq, ks, vs), brute


@pytest.mark.parametrize("mistake", ["dropped_v_scale", "swapped_scales", "ctx_off_by_one"])
def test_fp8_planted_mistakes_are_caught(monkeypatch, mistake):
    from oracle import paged_attention as OP
    (qp, ck, cv, bt, ctx, cq, ks, vs), brute = _planted_case()
    assert np.max(np.abs(F.prefill(qp, ck, cv, bt, ctx, cq, 0.27, ks, vs) - brute)) <= 1e-12
    real_gather, real_prefill_seq = F.gather, OP.prefill_seq
    if mistake == "dropped_v_scale":
        monkeypatch.setattr(F, "gather", lambda pk, pv, row, n, k_s=1.0, v_s=1.0: real_gather(pk, pv, row, n, k_s, 1.0))
    elif mistake == "swapped_scales":
        monkeypatch.setattr(F, "gather", lambda pk, pv, row, n, k_s=1.0, v_s=1.0: real_gather(pk, pv, row, n, v_s, k_s))
    elif mistake == "ctx_off_by_one":
        monkeypatch.setattr(OP, "prefill_seq", lambda q, k, v, s, c, rows=None: real_prefill_seq(q, k, v, s, c - 1, rows))
    got = F.prefill(qp, ck, cv, bt, ctx, cq, 0.27, ks, vs)
    assert np.max(np.abs(got - brute)) > 1e-6
