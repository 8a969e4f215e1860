"""GPU tests of FP8 (OCP E4M3) KV pools: kv_append's codes bit-exact against the oracle's quantiser in
the documented byte layout, kv_gather's dequantised values bit-exact, and decode / prefill over FP8
pages within tolerance of the oracle's attention over the dequantised values."""
import numpy as np
import pytest

from gpu_helpers import assert_close, gp_of, note, to_dev_bits
from oracle import fp8 as F
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

pytestmark = pytest.mark.gpu


class Fp8Case:
    def __init__(self, name, k_scale=1.0, v_scale=1.0, **over):
        import torch
        self.w = w = W.make_workload(name, **over)
        self.vals = W.make_values(w)
        self.ks, self.vs = k_scale, v_scale
        self.pool = kp.Pool(1, w.num_pages, w.Hkv, w.d, dtype=kp.KVP_FP8_E4M3)
        self.pool.set_scales(0, k_scale, v_scale)
        self.bt = torch.from_numpy(np.ascontiguousarray(w.block_tables)).cuda()
        kv = to_dev_bits(self.vals.kv)
        self.gp = gp_of(w)
        self.ck, self.cv = F.new_pool(w.num_pages, w.Hkv, w.d)
        for ab in w.setup_appends + w.step_appends:
            rows = torch.from_numpy(ab.src_rows).cuda()
            kp.kv_append(self.pool, 0, kv[rows, 0].contiguous(), kv[rows, 1].contiguous(), self.bt, ab.start_pos,
                         ab.cu_new, group_prefix=self.gp if ab.use_group_prefix else None)
            x = self.vals.kv[ab.src_rows]
            F.append(self.ck, self.cv, x[:, 0], x[:, 1], w.block_tables, ab.start_pos, ab.cu_new, k_scale, v_scale)
        torch.cuda.synchronize()


def _k_pos(t, c):
    return (((c // 64) * 4 + (c % 32) // 8) * 16 + t) * 16 + ((c // 32) % 2) * 8 + c % 8


def _v_pos(t, c, D):
    s = (t & ~12) | ((t & 4) << 1) | ((t & 8) >> 1)
    return 16 * D + ((((c // 32) * 2 + s // 8) * 16 + c % 16) * 16 + ((c // 16) % 2) * 8 + s % 8)


@pytest.mark.parametrize("name,ks,vs", [("tiny", 1.0, 1.0), ("mixed_s", 0.37, 1.9), ("rlvr_d64", 0.5, 0.5)])
def test_fp8_append_codes_in_documented_layout(name, ks, vs):
    note(f"fp8 append layout {name} scales {ks} {vs}")
    c = Fp8Case(name, ks, vs)
    w = c.w
    raw = c.pool.layer_bytes(0).cpu().numpy().reshape(w.num_pages, w.Hkv, 2 * 16 * w.d)
    t = np.arange(16)[:, None]
    cc = np.arange(w.d)[None, :]
    ik, iv = _k_pos(t, cc), _v_pos(t, cc, w.d)
    pages = np.unique(w.block_tables[w.block_tables >= 0])
    for page in pages:
        for h in range(w.Hkv):
            assert np.array_equal(raw[page, h][ik], c.ck[page, h]), ("K", page, h)
            assert np.array_equal(raw[page, h][iv], c.cv[page, h]), ("V", page, h)
    assert c.pool.device_error() == kp.KVP_OK


@pytest.mark.parametrize("name,ks,vs", [("mixed_s", 0.37, 1.9), ("rlvr_d64", 1.0, 1.0)])
def test_fp8_gather_dequantised_bitexact(name, ks, vs):
    import torch
    note(f"fp8 gather {name}")
    c = Fp8Case(name, ks, vs)
    w = c.w
    k, v = kp.kv_gather(c.pool, 0, c.bt, w.final_len)
    torch.cuda.synchronize()
    kb = k.view(torch.int16).cpu().numpy().view(np.uint16)
    vb = v.view(torch.int16).cpu().numpy().view(np.uint16)
    off = 0
    for i in range(w.B):
        n = int(w.final_len[i])
        pos = np.arange(n)
        pg = w.block_tables[i][pos // 16]
        ek = F.dequantize_bf16(c.ck[pg, :, pos % 16, :], ks)
        ev = F.dequantize_bf16(c.cv[pg, :, pos % 16, :], vs)
        assert np.array_equal(kb[off:off + n], ek), f"K of sequence {i}"
        assert np.array_equal(vb[off:off + n], ev), f"V of sequence {i}"
        off += n


def test_fp8_pool_settings():
    pool = kp.Pool(2, 16, 2, 64, dtype=kp.KVP_FP8_E4M3)
    assert pool.kv_dtype() == kp.KVP_FP8_E4M3
    assert kp.kv_pool_page_bytes(pool) == 2 * 2 * 16 * 64
    _, nbytes = pool.layer_ptr(1)
    assert nbytes == 16 * 2 * 2 * 16 * 64
    for bad in ((0.0, 1.0), (1.0, -1.0), (float("inf"), 1.0), (float("nan"), 1.0)):
        with pytest.raises(kp.KvpError) as ei:
            pool.set_scales(0, *bad)
        assert ei.value.code == kp.KVP_EINVAL
    with pytest.raises(kp.KvpError) as ei:
        pool.set_scales(2, 1.0, 1.0)
    assert ei.value.code == kp.KVP_EINVAL
    bf = kp.Pool(1, 16, 2, 64)
    assert bf.kv_dtype() == kp.KVP_BF16
    with pytest.raises(kp.KvpError) as ei:
        bf.set_scales(0, 1.0, 1.0)
    assert ei.value.code == kp.KVP_EUNSUPPORTED


def _decode(c, gp="auto", out_dtype=None):
    import torch
    w = c.w
    q = to_dev_bits(c.vals.q)
    out = kp.paged_decode_attn(q, c.pool, 0, c.bt, w.decode_len, group_prefix=c.gp if gp == "auto" else gp,
                               scale=w.scale, out_dtype=out_dtype or torch.float32)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("name,ks,vs", [("tiny", 1.0, 1.0), ("rlvr_s", 0.37, 1.9), ("rlhf_s", 1.0, 1.0),
                                         ("agentic_s", 0.5, 2.0), ("mixed_s", 1.0, 0.8), ("rlvr_d64", 1.3, 0.6)])
def test_fp8_decode_parity(name, ks, vs):
    note(f"fp8 decode {name} scales {ks} {vs}")
    c = Fp8Case(name, ks, vs)
    w = c.w
    ref = F.decode(c.vals.q, c.ck, c.cv, w.block_tables, w.decode_len, w.scale, ks, vs)
    assert_close(_decode(c), ref, f"fp8 decode {name}")
    if c.gp is not None:
        assert_close(_decode(c, gp=None), ref, f"fp8 decode {name} without the group hint")
    assert c.pool.device_error() == kp.KVP_OK


def test_fp8_decode_bf16_out_and_determinism():
    import torch
    c = Fp8Case("mixed_s", 0.7, 1.1)
    note("fp8 decode bf16 out, determinism")
    a = _decode(c, out_dtype=torch.bfloat16)
    b = _decode(c, out_dtype=torch.bfloat16)
    assert torch.equal(a, b)
    ref = F.decode(c.vals.q, c.ck, c.cv, c.w.block_tables, c.w.decode_len, c.w.scale, 0.7, 1.1)
    assert_close(a, ref, "fp8 decode bf16 out")


def _prefill(c, out_dtype=None):
    import torch
    w = c.w
    s0, s1 = int(w.prefill_seqs[0]), int(w.prefill_seqs[-1]) + 1
    out = kp.prefix_chunk_prefill_attn(to_dev_bits(c.vals.qp), c.pool, 0, c.bt[s0:s1], w.prefill_ctx, w.cu_q(),
                                       scale=w.scale, out_dtype=out_dtype or torch.float32)
    torch.cuda.synchronize()
    return out


def _oracle_prefill(c):
    w = c.w
    s0, s1 = int(w.prefill_seqs[0]), int(w.prefill_seqs[-1]) + 1
    return F.prefill(c.vals.qp, c.ck, c.cv, w.block_tables[s0:s1], w.prefill_ctx, w.cu_q(), w.scale, c.ks, c.vs)


@pytest.mark.parametrize("name,ks,vs,over", [("agentic_s", 1.0, 1.0, {}), ("mixed_s", 0.45, 1.7, {}),
                                              ("agentic_s", 0.8, 0.9, {"d": 64})])
def test_fp8_prefill_parity(name, ks, vs, over):
    note(f"fp8 prefill {name} {over} scales {ks} {vs}")
    c = Fp8Case(name, ks, vs, **over)
    assert_close(_prefill(c), _oracle_prefill(c), f"fp8 prefill {name} {over}")
    assert c.pool.device_error() == kp.KVP_OK
