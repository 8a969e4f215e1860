"""Pins of the prompt-block hashing oracle (CPU only): the SplitMix64 reference outputs, the prefix
property of the hash chain, and the two quantities the hashes are used for — a rollout group's shared
whole pages and a request's reusable prefix — against brute force over the token ids."""
import os

import numpy as np
import pytest

from oracle import prefix_hash as PH
from paper_2608_11152_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_reference_outputs():
    with open(os.path.join(GOLDEN, "splitmix64_seed0.txt")) as f:
        ref = [int(line, 16) for line in f.read().splitlines() if line.strip() and not line.startswith("#")]
    got = [PH.mix((n * PH.GAMMA) & PH.M64) for n in range(len(ref))]
    assert got == ref


def _toks(rng, n):
    return [int(x) for x in rng.integers(0, 151936, size=n)]


def test_prefix_property_and_sensitivity():
    rng = np.random.default_rng(11)
    for _ in range(20):
        n = int(rng.integers(16, 400))
        a = _toks(rng, n)
        ha = PH.block_hashes(a)
        assert len(ha) == n // 16
        # any extension leaves earlier hashes unchanged
        b = a + _toks(rng, int(rng.integers(0, 50)))
        assert PH.block_hashes(b)[: len(ha)] == ha
        # one changed token: earlier pages equal, its page and every later page differ
        p = int(rng.integers(0, n))
        c = list(a)
        c[p] = (c[p] + 1 + int(rng.integers(0, 1000))) % 151936
        hc = PH.block_hashes(c)
        for k in range(len(ha)):
            if k < p // 16:
                assert hc[k] == ha[k]
            else:
                assert hc[k] != ha[k]
        # the seed names the hash family
        if ha:
            assert PH.block_hashes(a, seed=1)[0] != ha[0]


def test_token_pairs_are_ordered():
    """Swapping two tokens of a page changes its hash (the fold is not a symmetric function)."""
    rng = np.random.default_rng(12)
    for _ in range(20):
        a = _toks(rng, 16)
        i, j = (int(x) for x in rng.choice(16, size=2, replace=False))
        if a[i] == a[j]:
            continue
        b = list(a)
        b[i], b[j] = b[j], b[i]
        assert PH.block_hashes(a) != PH.block_hashes(b)


def _lcp_pages(seqs):
    """Brute force: the number of leading full pages on which every sequence has the same tokens."""
    n = min(len(s) for s in seqs) // 16
    for k in range(n):
        if any(s[16 * k:16 * (k + 1)] != seqs[0][16 * k:16 * (k + 1)] for s in seqs[1:]):
            return k
    return n


def test_group_shared_pages_equals_token_lcp():
    rng = np.random.default_rng(13)
    for _ in range(30):
        m = int(rng.integers(1, 6))
        common = _toks(rng, int(rng.integers(0, 200)))
        seqs = [common + _toks(rng, int(rng.integers(0, 120))) for _ in range(m)]
        if rng.random() < 0.3 and m > 1:  # members that also share part of their private tail
            seqs[1] = seqs[0][: len(seqs[0]) - 3] + _toks(rng, 5)
        hashes = [PH.block_hashes(s) for s in seqs]
        assert PH.group_shared_pages(hashes) == _lcp_pages(seqs)
    assert PH.group_shared_pages([]) == 0


def test_workload_groups_share_their_whole_prompt_pages():
    """The synthetic rollout groups carry identical prompts: the derived shared pages are floor(P/16)."""
    for name in ("mixed_s", "rlvr_s", "rlhf_s"):
        w = W.make_workload(name)
        t, cu = W.make_tokens(w)
        hs = [PH.block_hashes(t[cu[i]:cu[i + 1]]) for i in range(w.B)]
        for g in range(w.num_groups):
            mem = [hs[i] for i in range(w.B) if w.group_id[i] == g]
            assert PH.group_shared_pages(mem) == int(w.shared_pages[g]) == int(w.prompt_len[g]) // 16


def test_lookup_equals_brute_force():
    rng = np.random.default_rng(14)
    cached = []
    base = [_toks(rng, int(rng.integers(32, 300))) for _ in range(4)]
    for b in base:  # cached sequences: some extend others, so prefixes repeat across entries
        cached.append(b)
        cached.append(b[: int(rng.integers(0, len(b)))] + _toks(rng, int(rng.integers(0, 80))))
    pages = [[int(x) for x in rng.integers(0, 10_000, size=len(s) // 16)] for s in cached]
    T = PH.PrefixTable()
    for s, p in zip(cached, pages):
        T.insert(PH.block_hashes(s), p)
    queries = [c[: int(rng.integers(0, len(c) + 1))] + _toks(rng, int(rng.integers(0, 60))) for c in cached]
    queries += [_toks(rng, 64)]
    for q in queries:
        hq = PH.block_hashes(q)
        m, got_pages = T.lookup(hq)
        best = max(_lcp_pages([q, c]) for c in cached)
        assert m == best
        for k in range(m):  # the page kept for a block is the largest page id inserted for it
            cands = [pages[j][k] for j, c in enumerate(cached) if _lcp_pages([q, c]) > k]
            assert got_pages[k] == max(cands)
        assert got_pages[m:] == [-1] * (len(hq) - m)
    # erasing one holder of a block leaves the mapping if another (larger) page holds it
    s0 = cached[0]
    h0 = PH.block_hashes(s0)
    T.erase(h0[:1], [pages[0][0]])
    m, _ = T.lookup(h0)
    holders = [pages[j][0] for j, c in enumerate(cached) if _lcp_pages([s0, c]) > 0]
    assert (m > 0) == (max(holders) != pages[0][0])


def test_planted_mistake_chain_without_parent_is_caught():
    """A hash that forgets the parent (hash(k) = mix(local(k))) names a page, not a prefix: two
    sequences that differ only before page k would collide at page k.  The sensitivity pin sees it."""
    def bad_hashes(tokens):
        return [PH.mix(PH.local_hash(tokens[16 * k:16 * (k + 1)])) for k in range(len(tokens) // 16)]
    rng = np.random.default_rng(15)
    a = _toks(rng, 64)
    b = list(a)
    b[3] += 1
    assert bad_hashes(a)[1:] == bad_hashes(b)[1:]          # the mistake: later pages collide
    assert PH.block_hashes(a)[1:] != PH.block_hashes(b)[1:]  # the oracle keeps them apart
