"""The replay's engine step on the GPU: every call goes through the library's C-ABI (kv_append,
prefix_chunk_prefill_attn, paged_decode_attn) on one paged pool.  Keys, values and queries are synthetic
N(0, 1) bf16 values from a seeded device generator; the replay models serving, not a trained model."""
from __future__ import annotations

import numpy as np


class LibraryEngine:
    def __init__(self, cfg, device="cuda", seed: int = 0, keep_last: bool = False):
        import torch
        from paper_2608_11152_amd import kvpattn as kp
        self.kp, self.torch = kp, torch
        self.cfg = cfg
        self.pool = kp.Pool(1, cfg.pool_pages, cfg.Hkv, cfg.d)
        self.gen = torch.Generator(device=device)
        self.gen.manual_seed(seed)
        self.device = device
        self.keep_last = keep_last
        self.last_decode = None
        self.calls = {"kv_append": 0, "prefix_chunk_prefill_attn": 0, "paged_decode_attn": 0}

    def _randn(self, *shape):
        t = self.torch
        return t.randn(shape, generator=self.gen, device=self.device, dtype=t.float32).to(t.bfloat16)

    def _table(self, rp, sessions, lens):
        return self.torch.from_numpy(rp.table_rows(sessions, lens)).to(self.device)

    def prefill(self, rp, batch):
        """batch: (session, H, L): append tokens [H, L) of each session, then prefill them over [0, H)."""
        kp, cfg = self.kp, self.cfg
        sessions = [s for s, _, _ in batch]
        lens = [L for _, _, L in batch]
        ctx = np.array([H for _, H, _ in batch], np.int32)
        cu = np.concatenate([[0], np.cumsum([L - H for _, H, L in batch])]).astype(np.int32)
        bt = self._table(rp, sessions, lens)
        T = int(cu[-1])
        if T == 0:
            return
        k, v = self._randn(T, cfg.Hkv, cfg.d), self._randn(T, cfg.Hkv, cfg.d)
        kp.kv_append(self.pool, 0, k, v, bt, ctx, cu)
        q = self._randn(T, cfg.Hq, cfg.d)
        kp.prefix_chunk_prefill_attn(q, self.pool, 0, bt, ctx, cu, out_dtype=self.torch.bfloat16)
        self.calls["kv_append"] += 1
        self.calls["prefix_chunk_prefill_attn"] += 1

    def decode(self, rp, dec):
        """dec: (session, first new position, new tokens): append them, then one decode query per session
        over all its tokens, with the groups' shared prompt pages as the group-prefix hint."""
        kp, cfg = self.kp, self.cfg
        sessions = [s for s, _, _ in dec]
        lens = np.array([a + n for _, a, n in dec], np.int32)
        start = np.array([a for _, a, _ in dec], np.int32)
        cu = np.concatenate([[0], np.cumsum([n for _, _, n in dec])]).astype(np.int32)
        bt = self._table(rp, sessions, lens)
        T = int(cu[-1])
        k, v = self._randn(T, cfg.Hkv, cfg.d), self._randn(T, cfg.Hkv, cfg.d)
        kp.kv_append(self.pool, 0, k, v, bt, start, cu)
        gid, shared = rp.group_hint(sessions)
        gp = kp.group_prefix(gid, shared) if len(shared) else None
        q = self._randn(len(dec), cfg.Hq, cfg.d)
        out = kp.paged_decode_attn(q, self.pool, 0, bt, lens, group_prefix=gp)
        self.calls["kv_append"] += 1
        self.calls["paged_decode_attn"] += 1
        if self.keep_last:
            self.last_decode = (q, out, bt, lens)

    def close(self):
        self.pool.close()
