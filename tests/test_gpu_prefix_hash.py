"""GPU tests of prompt-block hashing and prefix lookup (Sec. 4.4 of the paper): block hashes bit-exact
against the oracle, group shared pages derived on the device equal to the oracle's (and to the
workload's whole prompt pages), and the device prefix table's lookups equal the oracle table's."""
import numpy as np
import pytest

from gpu_helpers import note
from oracle import prefix_hash as PH
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

pytestmark = pytest.mark.gpu


def _dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _u64(t):
    return t.cpu().numpy().view(np.uint64)


def _oracle_hashes(tokens, cu, seed=0):
    out = []
    for i in range(len(cu) - 1):
        out.extend(PH.block_hashes(tokens[cu[i]:cu[i + 1]], seed))
    return np.array(out, dtype=np.uint64)


@pytest.mark.parametrize("name", ["mixed_s", "agentic_s", "rlvr_s"])
def test_block_hashes_bitexact(name):
    import torch
    w = W.make_workload(name)
    t, cu = W.make_tokens(w)
    note(f"block hashes {name}: {len(cu) - 1} seqs, {int(cu[-1])} tokens")
    for seed in (0, 0x1234_5678_9ABC_DEF1):
        got = kp.kvp_block_hashes(_dev(t), cu, seed=seed)
        torch.cuda.synchronize()
        ref = _oracle_hashes(t, cu, seed)
        assert np.array_equal(_u64(got), ref), f"{name} seed {seed:#x}"


def test_block_hashes_edge_lengths():
    import torch
    rng = np.random.default_rng(21)
    lens = [0, 1, 15, 16, 17, 31, 32, 1023, 1024, 1025, 64 * 16, 64 * 16 + 16, 130 * 16 + 7, 0, 48]
    t = rng.integers(-2**31, 2**31 - 1, size=sum(lens), dtype=np.int64).astype(np.int32)  # negative ids too
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    note("block hashes edge lengths")
    got = kp.kvp_block_hashes(_dev(t), cu, seed=7)
    torch.cuda.synchronize()
    assert np.array_equal(_u64(got), _oracle_hashes(t, cu, 7))
    empty = kp.kvp_block_hashes(_dev(t[:15]), np.array([0, 15], np.int32))
    assert empty.numel() == 0


@pytest.mark.parametrize("name", ["mixed_s", "rlvr_s", "rlhf_s"])
def test_group_shared_pages_device(name):
    w = W.make_workload(name)
    t, cu = W.make_tokens(w)
    note(f"group shared pages {name}")
    h = kp.kvp_block_hashes(_dev(t), cu)
    got = kp.kvp_group_shared_pages(h, cu, w.group_id, w.num_groups)
    assert np.array_equal(got, w.shared_pages)


def test_group_shared_pages_random_groups():
    rng = np.random.default_rng(22)
    seqs, gid = [], []
    G = 7
    for g in range(G):
        m = [0, 1, 1, 2, 3, 5, 8][g]  # group 0 has no members
        common = list(rng.integers(0, 50000, size=int(rng.integers(0, 300))))
        for _ in range(m):
            seqs.append(common + list(rng.integers(0, 50000, size=int(rng.integers(0, 90)))))
            gid.append(g)
    for _ in range(3):  # ungrouped
        seqs.append(list(rng.integers(0, 50000, size=int(rng.integers(0, 200)))))
        gid.append(-1)
    order = rng.permutation(len(seqs))
    seqs = [seqs[i] for i in order]
    gid = np.array([gid[i] for i in order], np.int32)
    t = np.array([x for s in seqs for x in s], np.int32)
    cu = np.concatenate([[0], np.cumsum([len(s) for s in seqs])]).astype(np.int32)
    note("group shared pages random")
    h = kp.kvp_block_hashes(_dev(t), cu)
    got = kp.kvp_group_shared_pages(h, cu, gid, G)
    hs = [PH.block_hashes(s) for s in seqs]
    ref = [PH.group_shared_pages([hs[i] for i in range(len(seqs)) if gid[i] == g]) for g in range(G)]
    assert list(got) == ref


def test_prefix_table_lookup_insert_erase_clear():
    import torch
    w = W.make_workload("mixed_s")
    t_all, cu_all = W.make_tokens(w)
    hist = W.step_start(w)
    t_hist, cu_hist = W.make_tokens(w, lens=hist)
    note("prefix table mixed_s")
    T = kp.PrefixTable(12)
    O = PH.PrefixTable()
    # the cached history of every sequence: its full pages and the physical pages holding them
    h_hist = kp.kvp_block_hashes(_dev(t_hist), cu_hist)
    off = kp.block_hash_offsets(cu_hist)
    ids = np.concatenate([w.block_tables[i][: int(off[i + 1] - off[i])] for i in range(w.B)]).astype(np.int32)
    T.insert(h_hist, _dev(ids))
    O.insert(_oracle_hashes(t_hist, cu_hist).tolist(), ids.tolist())
    # requests carry the full token lists (history + the step's new tokens)
    h_all = kp.kvp_block_hashes(_dev(t_all), cu_all)
    ho = _oracle_hashes(t_all, cu_all)
    offa = kp.block_hash_offsets(cu_all)

    def check(tag):
        m, pg = T.lookup(h_all, cu_all)
        torch.cuda.synchronize()
        m, pg = m.cpu().numpy(), pg.cpu().numpy()
        for i in range(w.B):
            rm, rp = O.lookup(ho[offa[i]:offa[i + 1]].tolist())
            assert m[i] == rm, f"{tag}: seq {i} matched {m[i]} vs {rm}"
            assert list(pg[offa[i]:offa[i + 1]]) == rp, f"{tag}: seq {i} pages"
        return m

    m = check("after insert")
    assert np.array_equal(m, hist // 16), "the cached history is the reusable prefix"
    # evict the second half of every history's pages
    er_h, er_p = [], []
    for i in range(w.B):
        n = int(off[i + 1] - off[i])
        er_h.append(np.arange(off[i] + n // 2, off[i + 1]))
    sel = np.concatenate(er_h).astype(np.int64)
    T.erase(h_hist[_dev(sel)], _dev(ids[sel]))
    O.erase(_oracle_hashes(t_hist, cu_hist)[sel].tolist(), ids[sel].tolist())
    check("after erase")
    T.clear()
    m, _ = T.lookup(h_all, cu_all)
    assert int(m.sum().item()) == 0
    assert T.error() == kp.KVP_OK


def test_prefix_table_full_reports_enomem():
    import torch
    T = kp.PrefixTable(4)  # 16 slots
    note("prefix table full")
    h = torch.arange(1, 41, dtype=torch.int64, device="cuda") * 0x9E3779B97F4A7C15 % (2**62)
    p = torch.arange(40, dtype=torch.int32, device="cuda")
    T.insert(h, p)
    assert T.error() == kp.KVP_ENOMEM
    m, pg = T.lookup(h[:16], np.array([0, 256], np.int32))
    torch.cuda.synchronize()
    assert 0 <= int(m[0].item()) <= 16


def test_prefix_host_errors():
    import torch
    t = _dev(np.arange(64, dtype=np.int32))
    out = torch.empty(8, dtype=torch.int64, device="cuda")
    cases = [
        (lambda: kp.lib().kvp_block_hashes(kp._dptr(t), kp._ptr(np.array([1, 32], np.int32)), 1, 0, kp._dptr(out), None), kp.KVP_EINVAL),
        (lambda: kp.lib().kvp_block_hashes(kp._dptr(t), kp._ptr(np.array([0, 32, 16], np.int32)), 2, 0, kp._dptr(out), None), kp.KVP_EINVAL),
        (lambda: kp.lib().kvp_group_shared_pages(kp._dptr(out), kp._ptr(np.array([0, 32], np.int32)), 1,
                                                  kp._ptr(np.array([3], np.int32)), 2, kp._dptr(out), None), kp.KVP_EGROUP),
    ]
    for fn, code in cases:
        assert fn() == code
    with pytest.raises(kp.KvpError) as ei:
        kp.PrefixTable(3)
    assert ei.value.code == kp.KVP_EINVAL
