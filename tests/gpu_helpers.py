"""Shared helpers for the GPU parity tests: run a workload's appends through the C-ABI and the same
appends through the CPU oracle, from the same seeded inputs."""
import sys

import numpy as np

import oracle
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

# Tolerance for bf16 inputs with fp32 accumulation (max-abs and mean-abs against the fp64 oracle).
MAX_ABS = 1e-2
MEAN_ABS = 1e-3


def note(msg):
    """Name the case being run before each GPU step, flushed, so a failure can be located."""
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


def to_dev_bits(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)


def gp_of(w):
    return kp.group_prefix(w.group_id, w.shared_pages) if w.num_groups else None


class GpuCase:
    """A workload with every append done on the GPU pool (and, lazily, the oracle's pool)."""

    def __init__(self, w, vals=None, block_tables=None, num_pages=None):
        import torch
        self.w = w
        self.vals = vals if vals is not None else W.make_values(w)
        self.bt_host = w.block_tables if block_tables is None else block_tables
        self.num_pages = w.num_pages if num_pages is None else num_pages
        self.pool = kp.Pool(1, self.num_pages, w.Hkv, w.d)
        self.bt = torch.from_numpy(np.ascontiguousarray(self.bt_host)).cuda()
        kv = self.vals.kv
        self.kv_dev = to_dev_bits(kv) if isinstance(kv, np.ndarray) else kv
        self.gp = gp_of(w)
        for ab in w.setup_appends + w.step_appends:
            rows = torch.from_numpy(ab.src_rows).cuda()
            k = self.kv_dev[rows, 0].contiguous()
            v = self.kv_dev[rows, 1].contiguous()
            kp.kv_append(self.pool, 0, k, v, self.bt, ab.start_pos, ab.cu_new,
                         group_prefix=self.gp if ab.use_group_prefix else None)
        torch.cuda.synchronize()
        self._opool = None

    def oracle_pool(self):
        if self._opool is None:
            pk, pv = oracle.new_pool(self.num_pages, self.w.Hkv, self.w.d)
            for ab in self.w.setup_appends + self.w.step_appends:
                kv = self.vals.kv[ab.src_rows]
                oracle.append(pk, pv, kv[:, 0], kv[:, 1], self.bt_host, ab.start_pos, ab.cu_new)
            self._opool = (pk, pv)
        return self._opool

    def decode(self, out_dtype=None, group_prefix="auto"):
        import torch
        q = to_dev_bits(self.vals.q) if isinstance(self.vals.q, np.ndarray) else self.vals.q
        gp = self.gp if group_prefix == "auto" else group_prefix
        out = kp.paged_decode_attn(q, self.pool, 0, self.bt, self.w.decode_len, group_prefix=gp,
                                   scale=self.w.scale, out_dtype=out_dtype or torch.float32)
        torch.cuda.synchronize()
        return out

    def oracle_decode(self):
        pk, pv = self.oracle_pool()
        return oracle.decode(self.vals.q, pk, pv, self.bt_host, self.w.decode_len, self.w.scale)

    def prefill(self, out_dtype=None):
        import torch
        w = self.w
        s0, s1 = int(w.prefill_seqs[0]), int(w.prefill_seqs[-1]) + 1
        q = to_dev_bits(self.vals.qp) if isinstance(self.vals.qp, np.ndarray) else self.vals.qp
        out = kp.prefix_chunk_prefill_attn(q, self.pool, 0, self.bt[s0:s1], w.prefill_ctx, w.cu_q(),
                                           scale=w.scale, out_dtype=out_dtype or torch.float32)
        torch.cuda.synchronize()
        return out

    def oracle_prefill(self):
        w = self.w
        pk, pv = self.oracle_pool()
        s0, s1 = int(w.prefill_seqs[0]), int(w.prefill_seqs[-1]) + 1
        return oracle.prefill(self.vals.qp, pk, pv, self.bt_host[s0:s1], w.prefill_ctx, w.cu_q(), w.scale)


def assert_close(got, ref, what, max_abs=MAX_ABS, mean_abs=MEAN_ABS):
    import torch
    g = got.float().cpu().numpy().astype(np.float64) if isinstance(got, torch.Tensor) else got
    err = np.abs(g - ref)
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    mx, mn = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    note(f"{what}: max_abs={mx:.3e} mean_abs={mn:.3e}")
    assert mx <= max_abs and mn <= mean_abs, f"{what}: max_abs={mx:.3e} mean_abs={mn:.3e}"


def oracle_by_kv_head(fn, q_bits, k_bits, v_bits, scale, *args, **kw):
    """Call an oracle routine (oracle.decode_seq or oracle.prefill_seq) once per KV head on contiguous
    copies of that head's K/V, with the query heads that read it (head h reads KV head h // (Hq / Hkv),
    reading c-2).  The arithmetic per head is the single call's; only the strided gathers are avoided,
    which makes the full-size comparisons several times faster.  q_bits [..., Hq, d] raw bf16;
    k_bits, v_bits [n, Hkv, d] raw bf16 (or float64 values)."""
    Hq, Hkv = q_bits.shape[-2], k_bits.shape[1]
    G = Hq // Hkv
    outs = []
    for g in range(Hkv):
        kg, vg = np.ascontiguousarray(k_bits[:, g:g + 1]), np.ascontiguousarray(v_bits[:, g:g + 1])
        if kg.dtype == np.uint16:
            kg, vg = oracle.widen_bf16(kg), oracle.widen_bf16(vg)
        outs.append(fn(np.ascontiguousarray(q_bits[..., g * G:(g + 1) * G, :]), kg, vg, scale, *args, **kw))
    return np.concatenate(outs, axis=-2)
