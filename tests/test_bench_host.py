"""Host-side arithmetic of bench.py (no GPU): the algorithmic byte counts the reported bandwidth is
divided by, and the one-GPU guard."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2608_11152_amd import workloads as W  # noqa: E402


def test_decode_bytes_tiny_by_hand():
    # lengths 17, 64, 100, 256; 2 KV heads, d = 64, 8 query heads, bf16, no sharing
    w = W.make_workload("tiny")
    kv = (17 + 64 + 100 + 256) * 2 * 64 * 2 * 2
    qo = 4 * 8 * 64 * 2 * 2
    pages = 2 + 4 + 7 + 16
    assert bench.decode_algorithmic_bytes(w) == kv + qo + 4 * pages


def test_decode_bytes_count_shared_pages_once():
    """Each group's shared prompt pages (tokens and block-table entries) count once, not once per member."""
    w = W.make_workload("rlvr_s")
    dec = w.decode_len > 0
    members = [int(((w.group_id == g) & dec).sum()) for g in range(w.num_groups)]
    saved_pages = sum(max(0, m - 1) * int(w.shared_pages[g]) for g, m in enumerate(members))
    assert saved_pages > 0
    tokens = int(w.decode_len.sum()) - 16 * saved_pages
    pages = sum((int(n) + 15) // 16 for n in w.decode_len) - saved_pages
    expected = tokens * w.Hkv * w.d * 2 * 2 + int(dec.sum()) * w.Hq * w.d * 2 * 2 + 4 * pages
    assert bench.decode_algorithmic_bytes(w) == expected


def test_fp8_bytes_are_half_the_kv():
    w = W.make_workload("rlhf_s")
    b16, b8 = bench.decode_algorithmic_bytes(w), bench.decode_algorithmic_bytes(w, kv_elem_bytes=1)
    assert b16 - b8 == w.unique_decode_tokens() * w.Hkv * w.d * 2


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0 and "one GPU" in r.stdout
