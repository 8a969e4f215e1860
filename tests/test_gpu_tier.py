"""GPU tests of the host KV tier (kv_offload / kv_restore, Sec. 5.5 of the paper): bit-exact page round
trips through pinned host memory, restore into other physical pages with a block-table patch (decode
unchanged bitwise and within tolerance of the oracle), and the host-side argument checks."""
import numpy as np
import pytest

from gpu_helpers import GpuCase, assert_close, note
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

pytestmark = pytest.mark.gpu


def _used_pages(w):
    """Every page the workload's appends wrote (up to each sequence's final length)."""
    used = []
    for i in range(w.B):
        n = (int(max(w.decode_len[i], w.final_len[i])) + 15) // 16
        used.extend(int(x) for x in w.block_tables[i][:n])
    return sorted(set(used))


def _page_bytes_of(raw, ids, pb):
    """Bytes of pool pages `ids` from an int16 view of the raw layer."""
    import torch
    r = raw.view(torch.uint8)
    return torch.cat([r[i * pb:(i + 1) * pb] for i in ids]).cpu()


def test_offload_restore_round_trip_bitwise():
    import torch
    w = W.make_workload("mixed_s")
    note("tier round trip mixed_s")
    c = GpuCase(w)
    ref_out = c.decode()
    pb = kp.kv_pool_page_bytes(c.pool)
    assert pb == w.Hkv * 64 * w.d
    raw0 = c.pool.layer_raw().clone()
    used = _used_pages(w)
    host = torch.empty(len(used) * pb, dtype=torch.uint8, pin_memory=True)
    kp.kv_offload(c.pool, 0, used, host)
    torch.cuda.synchronize()
    assert torch.equal(host, _page_bytes_of(raw0, used, pb)), "offloaded bytes differ from the pool pages"
    c.pool.reset()
    torch.cuda.synchronize()
    assert int(c.pool.layer_raw().abs().sum().item()) == 0
    kp.kv_restore(c.pool, 0, host, used)
    torch.cuda.synchronize()
    assert torch.equal(c.pool.layer_raw(), raw0), "restored pool differs from the original"
    out = c.decode()
    assert torch.equal(out, ref_out), "decode after restore is not bitwise equal"
    assert c.pool.device_error() == kp.KVP_OK


def test_restore_elsewhere_with_table_patch():
    """Restore every page into a different free page and patch the device block tables: decode is
    bitwise equal to decode over the original placement and within tolerance of the oracle."""
    import torch
    w = W.make_workload("tiny", pool_pages=256)
    note("tier restore elsewhere tiny")
    c = GpuCase(w)
    ref_out = c.decode()
    pb = kp.kv_pool_page_bytes(c.pool)
    used = _used_pages(w)
    rows, lps = [], []
    for p in used:
        i, lp = (int(x) for x in np.argwhere(w.block_tables == p)[0])
        rows.append(i)
        lps.append(lp)
    host = torch.empty(len(used) * pb, dtype=torch.uint8, pin_memory=True)
    kp.kv_offload(c.pool, 0, used, host)
    c.pool.reset()
    free = [p for p in range(w.num_pages) if p not in set(used)]
    dst = [int(x) for x in np.random.default_rng(9).permutation(free)[: len(used)]]
    bt2 = c.bt.clone()
    kp.kv_restore(c.pool, 0, host, dst, block_tables=bt2, rows=rows, lpages=lps)
    torch.cuda.synchronize()
    expect = w.block_tables.copy()
    for j in range(len(used)):
        expect[rows[j], lps[j]] = dst[j]
    assert np.array_equal(bt2.cpu().numpy(), expect), "block-table patch differs"
    q = c.vals.q if not isinstance(c.vals.q, np.ndarray) else None
    from gpu_helpers import to_dev_bits
    qd = to_dev_bits(c.vals.q) if isinstance(c.vals.q, np.ndarray) else c.vals.q
    out = kp.paged_decode_attn(qd, c.pool, 0, bt2, w.decode_len, scale=w.scale, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out), "decode over restored pages is not bitwise equal"
    assert_close(out, c.oracle_decode(), "tier restore elsewhere vs oracle")
    assert c.pool.device_error() == kp.KVP_OK


def test_tier_host_errors():
    import torch
    w = W.make_workload("tiny", pool_pages=64)
    note("tier host errors")
    c = GpuCase(w)
    pb = kp.kv_pool_page_bytes(c.pool)
    pinned = torch.empty(4 * pb, dtype=torch.uint8, pin_memory=True)
    pageable = torch.empty(4 * pb, dtype=torch.uint8)
    dev = torch.empty(4 * pb, dtype=torch.uint8, device="cuda")
    raw0 = c.pool.layer_raw().clone()
    cases = [
        (lambda: kp.kv_offload(c.pool, 0, [0, 1], pageable), kp.KVP_EINVAL),
        (lambda: kp.kv_offload(c.pool, 0, [0, 1], dev), kp.KVP_EINVAL),
        (lambda: kp.kv_offload(c.pool, 0, [0, 64], pinned), kp.KVP_ERANGE),
        (lambda: kp.kv_offload(c.pool, 0, [-1], pinned), kp.KVP_ERANGE),
        (lambda: kp.kv_restore(c.pool, 0, pinned, [3, 3]), kp.KVP_EINVAL),
        (lambda: kp.kv_restore(c.pool, 0, pinned, [70]), kp.KVP_ERANGE),
        (lambda: kp.kv_restore(c.pool, 0, pageable, [1]), kp.KVP_EINVAL),
        (lambda: kp.kv_restore(c.pool, 0, pinned, [1], block_tables=c.bt.clone(), rows=[w.B], lpages=[0]),
         kp.KVP_EINVAL),
        (lambda: kp.kv_restore(c.pool, 0, pinned, [1], block_tables=c.bt.clone(), rows=[0],
                               lpages=[c.bt.shape[1]]), kp.KVP_ERANGE),
        (lambda: kp.kv_offload(c.pool, 1, [0], pinned), kp.KVP_EINVAL),
    ]
    for fn, code in cases:
        with pytest.raises(kp.KvpError) as ei:
            fn()
        assert ei.value.code == code, str(ei.value)
    torch.cuda.synchronize()
    assert torch.equal(c.pool.layer_raw(), raw0), "a refused call changed the pool"
    kp.kv_offload(c.pool, 0, [], pinned)  # empty batch is a no-op
    kp.kv_restore(c.pool, 0, pinned, [])
