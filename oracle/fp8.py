"""FP8 (OCP E4M3) KV quantisation — TEST INFRASTRUCTURE ONLY (CPU).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may import this
module; the product path never does and shares no code with it.

Format (OCP 8-bit floating point, E4M3 "fn" variant): sign, 4 exponent bits (bias 7), 3 mantissa bits;
exponent 0 holds subnormals m/8 * 2^-6; exponent 15 with mantissa 7 is NaN; there is no infinity, so the
largest finite magnitude is 1.75 * 2^8 = 448.

Quantisation of a KV element (the library's convention; the paper stores KV in the engine's dtype and
says nothing about fp8): y = fp32(x) * fp32(1 / scale) in binary32, then y is rounded to the nearest E4M3
value, ties to the even mantissa; finite |y| beyond 448 saturates to 448; NaN stays NaN.  Dequantisation
is code value * scale.  A scale is a binary32 number (the library's scales are C floats), so a Python
scale is first rounded to binary32.  Attention over an fp8 pool is the plain attention of the
dequantised values.
"""
from __future__ import annotations

import numpy as np


def code_values() -> np.ndarray:
    """Value of every code 0..255 (float64; NaN for the two NaN codes), from the format definition."""
    c = np.arange(256)
    s = (c >> 7) & 1
    e = (c >> 3) & 15
    m = (c & 7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * 2.0 ** (e.astype(np.float64) - 7.0))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return np.where(s == 1, -mag, mag)


_VALS = code_values()
_MAGS = _VALS[:127]  # codes 0..126: the finite non-negative magnitudes, increasing with the code


def encode(y) -> np.ndarray:
    """E4M3 codes of float values y (round to nearest, ties to even mantissa, saturate at 448)."""
    y = np.asarray(y, dtype=np.float64)
    a = np.abs(y)
    hi = np.clip(np.searchsorted(_MAGS, a, side="left"), 0, 126)  # first magnitude >= a
    lo = np.clip(hi - 1, 0, 126)
    d_hi = np.abs(_MAGS[hi] - a)
    d_lo = np.abs(a - _MAGS[lo])
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo)
    code = np.where(a >= 448.0, 126, code)
    code = code | np.where(np.signbit(y), 0x80, 0)
    code = np.where(np.isnan(y), 0x7F | np.where(np.signbit(y), 0x80, 0), code)
    return code.astype(np.uint8)


def quantize_bf16(bits, scale: float) -> np.ndarray:
    """Codes of raw bf16 elements under a per-tensor scale: y = fp32(x) * fp32(1/scale) in binary32."""
    x = (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    inv = np.float32(1.0) / np.float32(scale)
    y = (x * inv).astype(np.float32)
    return encode(y.astype(np.float64))


def dequantize(codes, scale: float) -> np.ndarray:
    """Float64 values code value * scale, the scale taken as the binary32 value the library receives."""
    return _VALS[np.asarray(codes, dtype=np.uint8).astype(np.int64)] * float(np.float32(scale))


def dequantize_bf16(codes, scale: float) -> np.ndarray:
    """Raw bf16 bits of bf16(fp32(code value) * fp32(scale)), both roundings to nearest even."""
    v = (_VALS[np.asarray(codes, dtype=np.uint8).astype(np.int64)].astype(np.float32) * np.float32(scale))
    u = v.astype(np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) & 0xFFFF
    r = np.where(np.isnan(v), 0x7FC0 | ((u >> 16) & 0x8000), r)
    return r.astype(np.uint16)


# --- an FP8 pool in the oracle's own logical layout: codes uint8 [num_pages, Hkv, 16, d] for K and V ---

def new_pool(num_pages: int, num_kv_heads: int, head_dim: int):
    shape = (num_pages, num_kv_heads, 16, head_dim)
    return np.zeros(shape, dtype=np.uint8), np.zeros(shape, dtype=np.uint8)


def append(pool_k, pool_v, k_bits, v_bits, block_tables, start_pos, cu_new, k_scale=1.0, v_scale=1.0):
    """Quantise new tokens (raw bf16 [T, Hkv, d]) and write their codes to their paged slots."""
    kq = quantize_bf16(k_bits, k_scale)
    vq = quantize_bf16(v_bits, v_scale)
    for i in range(len(start_pos)):
        for t in range(int(cu_new[i]), int(cu_new[i + 1])):
            p = int(start_pos[i]) + (t - int(cu_new[i]))
            page = int(block_tables[i][p // 16])
            pool_k[page, :, p % 16, :] = kq[t]
            pool_v[page, :, p % 16, :] = vq[t]


def gather(pool_k, pool_v, table_row, n: int, k_scale=1.0, v_scale=1.0):
    """Dequantised float64 K, V [n, Hkv, d] of one sequence, read through its block table."""
    pos = np.arange(n)
    pages = np.asarray(table_row, dtype=np.int64)[pos // 16]
    return (dequantize(pool_k[pages, :, pos % 16, :], k_scale), dequantize(pool_v[pages, :, pos % 16, :], v_scale))


def decode(q_bits, pool_k, pool_v, block_tables, seq_lens, scale: float, k_scale=1.0, v_scale=1.0):
    """Paged decode attention over the dequantised pool (plain attention of the stored values)."""
    from .paged_attention import decode_seq
    q = np.asarray(q_bits)
    out = np.zeros(q.shape)
    for i in range(q.shape[0]):
        n = int(seq_lens[i])
        if n == 0:
            continue
        k, v = gather(pool_k, pool_v, block_tables[i], n, k_scale, v_scale)
        out[i] = decode_seq(q[i], k, v, scale)
    return out


def prefill(q_bits, pool_k, pool_v, block_tables, ctx_lens, cu_q, scale: float, k_scale=1.0, v_scale=1.0):
    """Chunked prefill over the dequantised pool."""
    from .paged_attention import prefill_seq
    out = np.zeros(np.asarray(q_bits).shape)
    for i in range(len(ctx_lens)):
        a, b = int(cu_q[i]), int(cu_q[i + 1])
        if b == a:
            continue
        ctx = int(ctx_lens[i])
        k, v = gather(pool_k, pool_v, block_tables[i], ctx + (b - a), k_scale, v_scale)
        out[a:b] = prefill_seq(q_bits[a:b], k, v, scale, ctx)
    return out
