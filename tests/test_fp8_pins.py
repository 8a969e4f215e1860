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
