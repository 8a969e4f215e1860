"""CPU fp64 oracle for prefix-shared paged-KV attention — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may import or
call this module.  The product path (the HIP library and its Python binding) never does, and shares no
code with it: this file reimplements everything it needs (bf16 widening, paging, attention) in the most
direct form, in float64.

What it computes
----------------
The paper (MISA-T, "Scheduling Mixed RL Rollouts Beyond Prefix Locality") is a routing-layer policy and
prints no attention formula; it fixes the *structure* of the data this oracle runs over:

* KV state lives in fixed-size blocks of a paged pool, retained per session (Sec. 2.3 on PagedAttention
  KV management; Sec. 3.2, the retained blocks k_s(t) of Eq. 2).  A sequence's token at logical position
  t lives in physical page ``block_table[t // 16]`` at slot ``t % 16``.
* Samples of one rollout group share the prompt prefix (Sec. 3.1, group identity g_r), and reuse is
  block-granular (Sec. 4.4: whole prompt blocks are matched by hash).  Sharing changes where bytes live, not
  what attention computes, so this oracle ignores any sharing hint: every sequence is gathered through
  its own block table.
* A later agentic turn prefills only the uncached L - H tokens over the cached history H (Eq. 1,
  Sec. 1), i.e. chunk queries at positions ctx..ctx+C-1 attend to the history plus the chunk's own
  earlier tokens.

The arithmetic is the textbook scaled-dot-product softmax attention with grouped-query heads, which the
paper does not restate.  Readings taken where the paper is silent:
  * softmax scale = caller's ``scale`` (1/sqrt(d) by default);
  * query head h reads KV head floor(h / (Hq / Hkv));
  * the decode query sees every cached token including its own (seq_len counts it);
  * prefill is bottom-right causal: chunk row j (position ctx + j) sees keys [0, ctx + j];
  * an empty sequence yields a zero output;
  * no positional term, mask, window or soft-cap beyond the lengths.
These conventions are not fixed by the paper ("parity unpinned" for the convention itself); every other
property of the functions below is pinned by the CPU tests (brute force, closed forms, invariances).

Data layout used here (the oracle's own, not the GPU library's): a logical pool holds raw bf16 bits as
``uint16 [num_pages, Hkv, 16, d]`` for K and for V.
"""
from __future__ import annotations

import numpy as np

PAGE = 16


def widen_bf16(bits) -> np.ndarray:
    """Raw bf16 bits (uint16) -> exact float64.  bf16 is the upper half of an IEEE-754 binary32."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def new_pool(num_pages: int, num_kv_heads: int, head_dim: int):
    """An empty logical pool: (K, V) raw-bit arrays [num_pages, Hkv, 16, d], zero-filled."""
    shape = (num_pages, num_kv_heads, PAGE, head_dim)
    return np.zeros(shape, dtype=np.uint16), np.zeros(shape, dtype=np.uint16)


def append(pool_k, pool_v, k_bits, v_bits, block_tables, start_pos, cu_new):
    """Write new tokens into their paged slots (Sec. 3.2: a session's retained blocks grow).

    Sequence i appends tokens ``k_bits[cu_new[i]:cu_new[i+1]]`` ([T, Hkv, d] raw bits) at logical
    positions start_pos[i], start_pos[i]+1, ...; position p goes to page block_tables[i][p // 16],
    slot p % 16.  Copies bits, so the result is exact."""
    B = len(start_pos)
    for i in range(B):
        for t in range(int(cu_new[i]), int(cu_new[i + 1])):
            p = int(start_pos[i]) + (t - int(cu_new[i]))
            page = int(block_tables[i][p // PAGE])
            pool_k[page, :, p % PAGE, :] = k_bits[t]
            pool_v[page, :, p % PAGE, :] = v_bits[t]


def gather(pool_k, pool_v, table_row, n: int):
    """Contiguous float64 K, V [n, Hkv, d] of one sequence, read through its block table."""
    pos = np.arange(n)
    pages = np.asarray(table_row, dtype=np.int64)[pos // PAGE]
    slots = pos % PAGE
    return widen_bf16(pool_k[pages, :, slots, :]), widen_bf16(pool_v[pages, :, slots, :])


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float) -> np.ndarray:
    """softmax(scale * q k^T) v for one head: q [R, d], k [n, d], v [n, d] -> [R, d] (float64).

    Subtracting the row max before exponentiating is the usual exact rewrite of softmax.  An empty key
    set gives zeros."""
    if k.shape[0] == 0:
        return np.zeros((q.shape[0], v.shape[1]))
    s = scale * (q @ k.T)
    s = s - s.max(axis=1, keepdims=True)
    w = np.exp(s)
    return (w @ v) / w.sum(axis=1, keepdims=True)


def attend_causal(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float, first_pos: int):
    """Row j of q (absolute position first_pos + j) attends keys [0, first_pos + j] (float64)."""
    R = q.shape[0]
    n = first_pos + R
    s = scale * (q @ k[:n].T)
    mask = np.arange(n)[None, :] > (first_pos + np.arange(R))[:, None]
    s[mask] = -np.inf
    s = s - s.max(axis=1, keepdims=True)
    w = np.exp(s)
    return (w @ v[:n]) / w.sum(axis=1, keepdims=True)


def kv_head_of(h: int, num_q_heads: int, num_kv_heads: int) -> int:
    """Grouped-query mapping: contiguous query heads share one KV head."""
    return h // (num_q_heads // num_kv_heads)


def decode_seq(q_bits_i, k, v, scale):
    """Decode output of one sequence: q [Hq, d] raw bits, contiguous k, v [n, Hkv, d] float64."""
    q = widen_bf16(q_bits_i)
    Hq, Hkv = q.shape[0], k.shape[1]
    out = np.zeros(q.shape)
    for h in range(Hq):
        g = kv_head_of(h, Hq, Hkv)
        out[h] = attend(q[h][None, :], k[:, g, :], v[:, g, :], scale)[0]
    return out


def decode(q_bits, pool_k, pool_v, block_tables, seq_lens, scale: float) -> np.ndarray:
    """Paged decode attention: one query token per sequence over its seq_lens[i] cached tokens.

    q_bits [B, Hq, d] raw bf16; returns float64 [B, Hq, d]."""
    B = len(seq_lens)
    out = np.zeros(np.asarray(q_bits).shape)
    for i in range(B):
        n = int(seq_lens[i])
        k, v = gather(pool_k, pool_v, block_tables[i], n)
        out[i] = decode_seq(q_bits[i], k, v, scale)
    return out


def prefill_seq(q_bits_rows, k, v, scale, ctx: int, rows=None):
    """Chunk prefill of one session: q [C, Hq, d] raw bits at positions ctx..ctx+C-1 over contiguous
    k, v [>= ctx+C, Hkv, d] float64.  ``rows`` optionally restricts to a subset of chunk rows (rows are
    independent, so a subset is computed exactly as in the full result)."""
    q = widen_bf16(q_bits_rows)
    C, Hq, _ = q.shape
    Hkv = k.shape[1]
    rows = np.arange(C) if rows is None else np.asarray(rows)
    out = np.zeros((len(rows), Hq, q.shape[2]))
    for h in range(Hq):
        g = kv_head_of(h, Hq, Hkv)
        for r0 in range(0, len(rows), 64):
            sel = rows[r0:r0 + 64]
            if np.all(np.diff(sel) == 1):
                j0 = int(sel[0])
                out[r0:r0 + len(sel), h] = attend_causal(q[sel, h], k[:, g], v[:, g], scale, ctx + j0)
            else:
                for t, j in enumerate(sel):
                    n = ctx + int(j) + 1
                    out[r0 + t, h] = attend(q[j, h][None, :], k[:n, g], v[:n, g], scale)[0]
    return out


def prefill(q_bits, pool_k, pool_v, block_tables, ctx_lens, cu_q, scale: float) -> np.ndarray:
    """Chunked prefill over a cached prefix for every session: q_bits [sum C_i, Hq, d] raw bf16.

    Session i's chunk rows are q_bits[cu_q[i]:cu_q[i+1]] at positions ctx_lens[i] + j.  Its chunk
    tokens must already be in the pool.  Returns float64 [sum C_i, Hq, d]."""
    out = np.zeros(np.asarray(q_bits).shape)
    for i in range(len(ctx_lens)):
        a, b = int(cu_q[i]), int(cu_q[i + 1])
        if b == a:
            continue
        ctx = int(ctx_lens[i])
        k, v = gather(pool_k, pool_v, block_tables[i], ctx + (b - a))
        out[a:b] = prefill_seq(q_bits[a:b], k, v, scale, ctx)
    return out


def offload(pool_k, pool_v, page_ids):
    """The host tier's copy of pool pages page_ids (Sec. 5.5: a host-memory tier backs up GPU-resident
    KV): their K and V raw bits, [n, Hkv, 16, d] each, in the order given."""
    ids = np.asarray(page_ids, dtype=np.int64)
    return pool_k[ids].copy(), pool_v[ids].copy()


def restore(pool_k, pool_v, page_ids, host_k, host_v, block_tables=None, rows=None, lpages=None):
    """Put host-tier page i back into pool page page_ids[i]; when a block table is given, logical page
    lpages[i] of table row rows[i] then names that page.  Copies bits, so the result is exact."""
    for i, p in enumerate(page_ids):
        pool_k[int(p)] = host_k[i]
        pool_v[int(p)] = host_v[i]
        if block_tables is not None:
            block_tables[int(rows[i]), int(lpages[i])] = int(p)
