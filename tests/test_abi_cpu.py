"""C-ABI boundary checks that need no GPU: the library loads and exports every declared symbol, the host
planner covers every (sequence, page) exactly once and is a pure function of lengths and groups, and the
host validators return the documented error codes."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "kvpattn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_bound_names():
    assert declared_functions() == sorted(kp.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(kp.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_strerror_and_version():
    assert "range" in kp.kvp_strerror(kp.KVP_ERANGE)
    assert kp.kvp_strerror(12345) == "unknown error"
    assert "gfx950" in kp.kvp_version()


def _coverage(seq_lens, gid=None, shared=None, Hq=32, Hkv=4):
    gp = kp.group_prefix(gid, shared) if gid is not None else None
    items, parts, ch = kp.kvp_plan_decode(seq_lens, Hq, Hkv, gp)
    B = len(seq_lens)
    G = Hq // Hkv
    cover = [np.zeros((int(n) + 15) // 16, np.int32) for n in seq_lens]
    slots = [set() for _ in range(B)]
    direct = [0] * B
    for kind, row, lo, hi, tok_end, first, nmem, slot in items.tolist():
        assert 0 < hi - lo <= max(ch, 16)
        if kind == 0:
            assert first == row and nmem == 1 and tok_end == seq_lens[row]
            cover[row][lo:hi] += 1
            if slot < 0:
                direct[row] += 1
            else:
                slots[row].add(slot)
        else:
            g = gid[row]
            assert tok_end == shared[g] * 16 and hi <= shared[g]
            mem = [i for i in range(B) if gid[i] == g and seq_lens[i] > 0]
            k = mem.index(first)
            assert nmem * G <= 64 and mem[k:k + nmem] == mem[k:k + nmem]
            for i in mem[k:k + nmem]:
                cover[i][lo:hi] += 1
                slots[i].add(slot)
    for i in range(B):
        assert np.all(cover[i] == 1), (i, cover[i])
        if direct[i]:
            assert direct[i] == 1 and not slots[i]
        else:
            assert slots[i] == set(range(len(slots[i])))
    return items, parts, ch


@pytest.mark.parametrize("name", ["tiny", "rlvr_s", "rlhf_s", "mixed_s", "rlvr_d64", "rlvr", "mixed"])
def test_plan_covers_every_page_once(name):
    w = W.make_workload(name)
    gid = w.group_id if w.num_groups else None
    _coverage(w.decode_len, gid, w.shared_pages if gid is not None else None, w.Hq, w.Hkv)


def _plan_constant(name):
    import re
    hdr = open(os.path.join(ROOT, "paper_2608_11152_amd", "csrc", "kvp_plan.h")).read()
    return int(re.search(rf"constexpr int {name} = (\d+);", hdr).group(1))


@pytest.mark.parametrize("name", ["mixed", "rlhf", "agentic"])
def test_plan_segments_are_balanced(name):
    """Wave-path chunks are cut into segments of equal cost (pages plus a fixed start cost per chunk)
    whatever the length skew.  Packed in order into budgets of pages_per_split + that cost (in-order
    greedy packing uses the fewest budgets), the chunks fill one round of waves, and no chunk is larger
    than pages_per_split."""
    w = W.make_workload(name)
    gp = kp.group_prefix(w.group_id, w.shared_pages) if w.num_groups else None
    items, parts, seg = kp.kvp_plan_decode(w.decode_len, w.Hq, w.Hkv, gp)
    wave = items[(items[:, 0] == 0) | (items[:, 6] * (w.Hq // w.Hkv) <= 16)]
    K, waves = _plan_constant("kChunkStartPages"), _plan_constant("kDecodeWaves")
    pages = (wave[:, 3] - wave[:, 2]).tolist()
    # a shared-prefix chunk gives each of its members a partial; a sequence splits only at segment ends
    assert max(pages) <= seg and parts < int(items[:, 6].sum()) + w.B
    cap, fill, n_seg = seg + K, 0, 1
    for p in pages:
        if fill > 0 and fill + K + p > cap:
            n_seg, fill = n_seg + 1, 0
        fill += K + p
    assert n_seg * w.Hkv <= waves, (n_seg, w.Hkv, waves)


def test_plan_prefix_counted_once_per_group():
    w = W.make_workload("rlvr")
    items, _, _ = kp.kvp_plan_decode(w.decode_len, w.Hq, w.Hkv, kp.group_prefix(w.group_id, w.shared_pages))
    pref = items[items[:, 0] == 1]
    per_group = {}
    for kind, row, lo, hi, *_ in pref.tolist():
        per_group[w.group_id[row]] = per_group.get(w.group_id[row], 0) + hi - lo
    for g, n in per_group.items():
        assert n == w.shared_pages[g]  # 8 samples x 8 heads = 64 columns: one subgroup reads each page once


def test_plan_edge_lengths():
    _coverage([0, 1, 15, 16, 17, 31, 32, 33, 5000, 0], Hq=8, Hkv=2)
    gid = np.array([0, 0, 0, 1, 1, -1, 0], np.int32)
    shared = np.array([2, 0], np.int32)
    _coverage([40, 32, 0, 7, 9, 100, 33], gid, shared, Hq=8, Hkv=1)  # G = 8, member with len == prefix


def test_plan_is_deterministic_and_independent_of_pages():
    w = W.make_workload("mixed")
    gp = kp.group_prefix(w.group_id, w.shared_pages)
    a = kp.kvp_plan_decode(w.decode_len, w.Hq, w.Hkv, gp)
    b = kp.kvp_plan_decode(w.decode_len.copy(), w.Hq, w.Hkv, kp.group_prefix(w.group_id, w.shared_pages))
    assert np.array_equal(a[0], b[0]) and a[1:] == b[1:]
    w2 = W.make_workload("mixed", seed=w.seed)  # same lengths; the permutation is not an input of the plan
    assert np.array_equal(kp.kvp_plan_decode(w2.decode_len, w.Hq, w.Hkv, gp)[0], a[0])


def test_plan_large_group_splits_into_subgroups():
    # 24 members x 8 heads = 192 columns -> three subgroups of 8; each reads the prefix once
    B = 24
    items, _, _ = kp.kvp_plan_decode([100] * B, 32, 4, kp.group_prefix([0] * B, [5]))
    pref = items[items[:, 0] == 1]
    assert len(pref) == 3 and set(pref[:, 6].tolist()) == {8}


def test_plan_wide_group_goes_to_waves_only_when_prefix_is_small():
    """A group wider than one wave (8 members x 8 heads) is read per 16-column subgroup on the wave path
    when that adds at most 1% pages to the call; otherwise it stays one LDS-staged item per page range."""
    G, B = 8, 8
    long_private = [2 * 16 + 4000] * B  # 2 shared pages, ~250 private pages each: 6 extra pages of ~2000
    items, _, _ = _coverage(long_private, np.zeros(B, np.int32), np.array([2], np.int32), Hq=32, Hkv=4)
    pref = items[items[:, 0] == 1]
    assert len(pref) > 0 and np.all(pref[:, 6] * G <= 16)
    assert sorted(set(pref[:, 6].tolist())) == [2]  # four subgroups of two members, each reads the prefix
    assert int((pref[:, 3] - pref[:, 2]).sum()) == 4 * 2
    long_prefix = [40 * 16 + 100] * B  # 40 shared pages against ~7 private pages each
    items, _, _ = _coverage(long_prefix, np.zeros(B, np.int32), np.array([40], np.int32), Hq=32, Hkv=4)
    pref = items[items[:, 0] == 1]
    assert np.all(pref[:, 6] == B) and int((pref[:, 3] - pref[:, 2]).sum()) == 40


def test_plan_validation_codes():
    with pytest.raises(kp.KvpError) as e:
        kp.kvp_plan_decode([10], 12, 4)  # G = 3
    assert e.value.code == kp.KVP_EUNSUPPORTED
    with pytest.raises(kp.KvpError) as e:
        kp.kvp_plan_decode([10, 20], 8, 2, kp.group_prefix([0, 1], [1]))  # group id out of range
    assert e.value.code == kp.KVP_EGROUP
    with pytest.raises(kp.KvpError) as e:
        kp.kvp_plan_decode([10, 40], 8, 2, kp.group_prefix([0, 0], [1]))  # member shorter than prefix
    assert e.value.code == kp.KVP_EGROUP
    with pytest.raises(kp.KvpError) as e:
        kp.kvp_plan_decode([-1], 8, 2)
    assert e.value.code == kp.KVP_EINVAL


def test_check_tables_codes():
    w = W.make_workload("rlvr_d64")
    gp = kp.group_prefix(w.group_id, w.shared_pages)
    assert kp.kvp_check_tables(w.block_tables, w.final_len, w.num_pages, gp) == kp.KVP_OK
    bt = w.block_tables.copy()
    bt[3, 0] = w.num_pages  # out of the pool
    assert kp.kvp_check_tables(bt, w.final_len, w.num_pages, gp) == kp.KVP_ERANGE
    bt = w.block_tables.copy()
    member = int(np.flatnonzero(w.group_id == 0)[1])
    bt[member, 0] = bt[member, int(w.shared_pages[0])]  # a member whose "shared" page differs
    assert kp.kvp_check_tables(bt, w.final_len, w.num_pages, gp) == kp.KVP_EGROUP
    long = w.final_len.copy()
    long[0] = w.maxp * 16 + 1
    assert kp.kvp_check_tables(w.block_tables, long, w.num_pages, None) == kp.KVP_ERANGE


def test_pool_create_rejects_unsupported_shapes_without_a_device():
    h = ctypes.c_void_p()
    L = kp.lib()
    assert L.kv_pool_create(ctypes.byref(h), 1, 16, 16, 2, 96, 0) == kp.KVP_EUNSUPPORTED
    assert L.kv_pool_create(ctypes.byref(h), 1, 16, 32, 2, 128, 0) == kp.KVP_EUNSUPPORTED
    assert L.kv_pool_create(ctypes.byref(h), 1, 16, 16, 2, 128, 1) == kp.KVP_EUNSUPPORTED
    assert L.kv_pool_create(ctypes.byref(h), 0, 16, 16, 2, 128, 0) == kp.KVP_EINVAL
    assert L.kv_pool_create(None, 1, 16, 16, 2, 128, 0) == kp.KVP_EINVAL
    assert L.kv_pool_destroy(None) == kp.KVP_OK


def test_binding_refuses_host_tensors():
    """Device arguments are bare pointers to the library: the binding refuses host tensors up front (this
    runs without a GPU; nothing reaches the library)."""
    import torch
    q = torch.zeros((2, 8, 64), dtype=torch.bfloat16)
    bt = torch.zeros((2, 4), dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU tensor"):
        kp.paged_decode_attn(q, None, 0, bt, [16, 16])
    with pytest.raises(ValueError, match="GPU tensor"):
        kp.prefix_chunk_prefill_attn(q, None, 0, bt, [0, 0], [0, 1, 2])
    with pytest.raises(ValueError, match="cu_new"):
        kp.kv_append(None, 0, q, q, bt, [0, 0], [0, 1])
    with pytest.raises(ValueError, match="GPU tensor"):
        kp.kv_append(None, 0, q, q, bt, [0, 0], [0, 1, 2])


def test_missing_library_fails_loudly():
    """There is no CPU fallback: without the built library every entry point raises."""
    code = ("import paper_2608_11152_amd.kvpattn as kp; kp.LIB_PATH = '/nonexistent/libkvpattn.so'\n"
            "try:\n    kp.kvp_version()\nexcept RuntimeError as e:\n    print('raised', e)\n")
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=root, timeout=120)
    assert r.returncode == 0 and "raised" in r.stdout and "missing" in r.stdout


def test_product_code_never_imports_the_oracle():
    """The oracle is test infrastructure: nothing in the package or the C sources imports, links or reads it."""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    pkg = os.path.join(root, "paper_2608_11152_amd")
    pat = re.compile(r"^\s*(import\s+oracle|from\s+oracle\b)|#include\s+\"?.*oracle", re.M)
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert not pat.search(text), os.path.join(dirpath, f)


def test_product_code_never_imports_the_controller_replay():
    """The MISA-T controller replay (misa_t/) is a harness around the library: the package never imports
    it, and neither does the benchmark."""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    pat = re.compile(r"^\s*(import\s+misa_t|from\s+misa_t\b)", re.M)
    paths = [os.path.join(root, "bench.py")]
    for dirpath, _, files in os.walk(os.path.join(root, "paper_2608_11152_amd")):
        paths += [os.path.join(dirpath, f) for f in files if f.endswith(".py")]
    for p in paths:
        assert not pat.search(open(p).read()), p
