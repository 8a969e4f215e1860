"""Benchmark of the prefix-shared paged-KV attention path on one MI355X.

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload mixed] [--no-cpu-baseline]

Workload (default): the mixed rollout step — 40 sessions (2 RLVR groups x 8 samples, 6 RLHF groups x 2,
12 agentic sessions with 32k-128k cached history) in a 1.5M-token pool of randomly permuted pages.
One step = kv_append of every session's new tokens (40 decode tokens + 8 agentic 2048-token chunks),
paged_decode_attn for all 40 sessions (shared prompt pages read once per group, split-KV + LSE merge),
then prefix_chunk_prefill_attn for the 8 chunks over their cached histories.  Inputs are synthetic
(seeded N(0,1) bf16 values), resident in HBM before timing starts.  Each step first overwrites a 512 MB
buffer so that no KV read can hit the 256 MB Infinity Cache left warm by the previous step (in a serving
engine the rest of the model runs between two attention calls).

Prints one JSON line.  `value` is the metric: effective decode KV bandwidth (algorithmic bytes of the
paged_decode_attn call / its GPU time).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "paged decode-attn effective KV GB/s (% HBM peak) + decode tokens/s, mixed batch"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
HOST_LINK_PEAK_GBS = 64.0  # PCIe Gen5 x16, one direction

WORKLOAD_TEXT = {
    "mixed": "mixed step: 40 sessions (16 RLVR in 2 groups x 8, 12 RLHF in 6 groups x 2, 12 agentic), "
             "1.5M-token pool of permuted 16-token pages, decode for all 40 + 2048-token prefill chunks "
             "for 8 agentic sessions; GQA 32/4, d=128, bf16",
    "rlvr": "RLVR decode: 64 groups x 8 samples, shared prompt U[128,1024], private U[1k,16k]; GQA 32/4, d=128",
    "rlhf": "RLHF decode: 128 groups x 2 samples, lognormal prompt/response (median 1k); GQA 32/4, d=128",
    "agentic": "agentic turn: 32 sessions, history U[32k,128k], 2048-token chunk prefill + 1 decode; "
               "GQA 32/4, d=128",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mixed", choices=sorted(WORKLOAD_TEXT))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="budget of the oracle baseline sample")
    ap.add_argument("--no-flush", action="store_true", help="do not evict the Infinity Cache between steps")
    ap.add_argument("--no-fp8", action="store_true", help="skip the FP8-KV leg (same step over an FP8 pool)")
    ap.add_argument("--no-mixed-step", action="store_true",
                    help="skip the leg that times the step's attention as one mixed_step_attn launch")
    ap.add_argument("--no-prefill-split", action="store_true",
                    help="skip the split-history prefill leg (keeps a profile's prefill and merge kernels to the step)")
    return ap.parse_args()


def decode_algorithmic_bytes(w, kv_elem_bytes: int = 2) -> int:
    """KV bytes of every cached token decode reads, each group's shared pages counted once, plus Q, O
    (bf16) and the block-table entries referenced."""
    kv = w.unique_decode_tokens() * w.Hkv * w.d * 2 * kv_elem_bytes
    dec = w.decode_len > 0
    qo = int(dec.sum()) * w.Hq * w.d * 2 * 2
    pages = 0
    for i in range(w.B):
        n = int(w.decode_len[i])
        if n:
            g = int(w.group_id[i])
            pages += (n + 15) // 16 - (int(w.shared_pages[g]) if g >= 0 else 0)
    for g in range(w.num_groups):
        if np.any((w.group_id == g) & dec):
            pages += int(w.shared_pages[g])
    return kv + qo + 4 * pages


def prefill_algorithmic_bytes(w) -> int:
    """Unique bytes the prefill must touch: each session's KV up to its last chunk token, Q and O."""
    toks = int((w.prefill_ctx + w.prefill_chunk).sum())
    return toks * w.Hkv * w.d * 4 + int(w.prefill_chunk.sum()) * w.Hq * w.d * 4


PROFILE_OF = {"mixed": "decode_prefill_mixed_step.md", "rlvr": "decode_rlvr_64x8.md",
              "rlhf": "decode_rlhf_128x2.md", "agentic": "decode_prefill_agentic_32x128k.md"}
KERNEL_SOURCES = ("decode.hip", "decode_dev.h", "prefill.hip", "prefill_dev.h", "prefill_body.inc", "plan.cpp", "api.cpp", "kvp_layout.h",
                  "kvp_kernels.h", "kvp_plan.h")


def profiled_traffic(workload: str) -> dict:
    """Per-launch HBM bytes (FETCH_SIZE x2 + WRITE_SIZE, see the profile summary) for this workload:
    {"decode", "prefill", "decode_fp8", "prefill_fp8"} -> bytes, each None when the summary lacks it.
    All None when no summary exists or the kernel sources changed since the counters were taken."""
    import hashlib
    keys = {"traffic-decode-bytes": "decode", "traffic-prefill-bytes": "prefill",
            "traffic-decode-fp8-bytes": "decode_fp8", "traffic-prefill-fp8-bytes": "prefill_fp8"}
    res = {v: None for v in keys.values()}
    path = os.path.join(ROOT, "profiles", PROFILE_OF.get(workload, "-"))
    if not os.path.exists(path):
        return res
    fields = {}
    for line in open(path):
        if ":" in line and line.split(":")[0].strip() in (("kernel-source-sha256",) + tuple(keys)):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2608_11152_amd", "csrc", f), "rb").read())
    if fields.get("kernel-source-sha256") != h.hexdigest():
        return res
    for k, name in keys.items():
        if fields.get(k):
            res[name] = int(float(fields[k]))
    return res


def library_gemm_tflops(dev, stream, n: int = 16384, reps: int = 5) -> float:
    """bf16 dense GEMM rate of the vendor library (torch.matmul -> hipBLASLt) on N(0,1) operands.

    The chip's clock under dense bf16 matrix load depends on the operand data (random operands draw more
    power than constants), so this is the practical MFMA ceiling next to which the prefill rate is read.
    """
    import torch
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    a = torch.randn(n, n, generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    b = torch.randn(n, n, generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    for _ in range(3):
        c = a @ b
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        c = a @ b
    e1.record(stream)
    torch.cuda.synchronize()
    del a, b, c
    return round(2.0 * n ** 3 * reps / (e0.elapsed_time(e1) / 1e3) / 1e12, 1)


def kv_tier_leg(kp, pool, w, stream, reps: int = 3) -> dict:
    """Host KV tier: offload, then restore, every page of the workload's longest sequence through pinned
    host memory (kv_offload / kv_restore, one launch each), beside plain contiguous copies of the same
    byte count between pinned host memory and HBM as the host link's practical rate."""
    import torch
    i = int(np.argmax(w.final_len))
    ids = [int(x) for x in w.block_tables[i][: (int(w.final_len[i]) + 15) // 16]]
    pb = kp.kv_pool_page_bytes(pool)
    nbytes = len(ids) * pb
    host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    dev = torch.empty(nbytes, dtype=torch.uint8, device="cuda")

    def timed(fn):
        fn()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / 1e3)
        return round(nbytes / float(np.median(ts)) / 1e9, 2)

    off = timed(lambda: kp.kv_offload(pool, 0, ids, host))
    res = timed(lambda: kp.kv_restore(pool, 0, host, ids))
    h2d = timed(lambda: dev.copy_(host, non_blocking=True))
    d2h = timed(lambda: host.copy_(dev, non_blocking=True))
    del host, dev
    return {"pages": len(ids), "bytes": nbytes, "offload_gbs": off, "restore_gbs": res, "h2d_copy_gbs": h2d,
            "d2h_copy_gbs": d2h,
            "roofline": {"bound": "host link", "achieved": res, "peak": HOST_LINK_PEAK_GBS, "unit": "GB/s",
                         "frac": round(res / HOST_LINK_PEAK_GBS, 4), "kernel": "kv_restore"}}


def prefix_hash_leg(kp, W, w, stream, reps: int = 5) -> dict:
    """Prompt-block hashing and prefix lookup over the workload's synthetic token ids: hash every full
    page of every sequence, derive the groups' shared pages, register each sequence's cached history in
    a device prefix table, and look up the full sequences (their reusable prefix H)."""
    import torch
    tokens, cu = W.make_tokens(w)
    th, cuh = W.make_tokens(w, lens=W.step_start(w))
    t_dev, th_dev = torch.from_numpy(tokens).cuda(), torch.from_numpy(th).cuda()
    off_h = kp.block_hash_offsets(cuh)
    ids = np.concatenate([w.block_tables[i][: int(off_h[i + 1] - off_h[i])] for i in range(w.B)]).astype(np.int32)
    ids_dev = torch.from_numpy(ids).cuda()
    pages = int(kp.block_hash_offsets(cu)[-1])
    h_all = torch.empty(max(1, pages), dtype=torch.int64, device="cuda")
    table = kp.PrefixTable(max(10, int(np.ceil(np.log2(max(2, 2 * len(ids)))))))
    h_hist = kp.kvp_block_hashes(th_dev, cuh)
    table.insert(h_hist, ids_dev)

    def timed(fn):
        fn()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    t_hash = timed(lambda: kp.kvp_block_hashes(t_dev, cu, out=h_all))
    t_look = timed(lambda: table.lookup(h_all, cu))
    matched, _ = table.lookup(h_all, cu)
    shared = kp.kvp_group_shared_pages(h_all, cu, w.group_id, w.num_groups) if w.num_groups else np.zeros(0)
    ok = bool(np.array_equal(shared, w.shared_pages)) and bool(
        np.array_equal(matched.cpu().numpy(), W.step_start(w) // 16))
    table.close()
    return {"tokens": int(cu[-1]), "pages": pages, "hash_ms": round(t_hash, 4),
            "hash_tokens_per_s": round(int(cu[-1]) / (t_hash / 1e3), 1), "lookup_ms": round(t_look, 4),
            "lookup_pages_per_s": round(pages / (t_look / 1e3), 1), "reused_tokens": int(matched.sum().item()) * 16,
            "derived_prefixes_match": ok}


def fp8_kv_leg(kp, w, vals, gp, bt, step_batches, flush, stream, steps: int, warmup: int, bf16_decode_s: float,
               has_prefill: bool, s0: int, s1: int, cu_q) -> dict:
    """The same step over an FP8 (E4M3) pool of the same workload: kv_append quantises, decode and prefill
    read one byte per KV element.  Scales stay 1 (the N(0,1) values sit well inside E4M3's range)."""
    import torch
    pool = kp.Pool(1, w.num_pages, w.Hkv, w.d, dtype=kp.KVP_FP8_E4M3)
    for ab in w.setup_appends:
        rows = torch.from_numpy(ab.src_rows).to(bt.device)
        kp.kv_append(pool, 0, vals.kv[rows, 0].contiguous(), vals.kv[rows, 1].contiguous(), bt, ab.start_pos,
                     ab.cu_new, group_prefix=gp if ab.use_group_prefix else None)
    ws = torch.empty(max(1, kp.paged_decode_workspace_size(pool, w.decode_len, w.Hq, gp)), dtype=torch.uint8,
                     device=bt.device)
    out = torch.empty((w.B, w.Hq, w.d), dtype=torch.bfloat16, device=bt.device)
    if has_prefill:
        pf_ws = torch.empty(max(1, kp.prefix_chunk_prefill_workspace_size(pool, w.prefill_ctx, cu_q, w.Hq)),
                            dtype=torch.uint8, device=bt.device)
        pf_out = torch.empty((int(cu_q[-1]), w.Hq, w.d), dtype=torch.bfloat16, device=bt.device)
    t_dec, t_pf = [], []
    for it in range(warmup + steps):
        flush.fill_(1)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        for k, v, ab in step_batches:
            kp.kv_append(pool, 0, k, v, bt, ab.start_pos, ab.cu_new, group_prefix=gp if ab.use_group_prefix else None)
        ev[0].record(stream)
        kp.paged_decode_attn(vals.q, pool, 0, bt, w.decode_len, group_prefix=gp, scale=w.scale, out=out, ws=ws)
        ev[1].record(stream)
        if has_prefill:
            kp.prefix_chunk_prefill_attn(vals.qp, pool, 0, bt[s0:s1], w.prefill_ctx, cu_q, scale=w.scale,
                                         out=pf_out, ws=pf_ws)
        ev[2].record(stream)
        torch.cuda.synchronize()
        if it >= warmup:
            t_dec.append(ev[0].elapsed_time(ev[1]))
            t_pf.append(ev[1].elapsed_time(ev[2]))
    if pool.device_error() != kp.KVP_OK:
        raise RuntimeError("device error in the FP8 leg")
    pool.close()
    dec_s = float(np.median(t_dec)) / 1e3
    nbytes = decode_algorithmic_bytes(w, kv_elem_bytes=1)
    n_dec = int((w.decode_len > 0).sum())
    res = {"kv_dtype": "fp8 e4m3 (bf16 matrix-core operands, fp32 accumulation)",
           "decode_ms": round(dec_s * 1e3, 4), "decode_gbs": round(nbytes / dec_s / 1e9, 2),
           "decode_hbm_peak_frac": round(nbytes / dec_s / 1e9 / HBM_PEAK_GBS, 4),
           "decode_tokens_per_s": round(n_dec / dec_s, 1), "decode_speedup_vs_bf16": round(bf16_decode_s / dec_s, 3),
           "algorithmic_bytes_per_launch": nbytes}
    if has_prefill:
        pf_s = float(np.median(t_pf)) / 1e3
        res["prefill_ms"] = round(pf_s * 1e3, 4)
        res["prefill_tflops"] = round(w.prefill_flops() / pf_s / 1e12, 2)
    return res


def prefill_split_leg(kp, dev, stream, ctx: int = 131072, chunks=(64, 256), reps: int = 10) -> dict:
    """One agentic session with a long cached history and a short new chunk (Eq. 1's L - H small against
    H): too few query tiles to fill the GPU, so the planner splits each tile's history into key ranges
    (partials merged per query row).  GQA 32/4, d = 128, bf16 pages, synthetic N(0, 1) values."""
    import torch
    Hq, Hkv, d = 32, 4, 128
    n = ctx + max(chunks)
    npg = (n + 15) // 16
    g = torch.Generator(device=dev)
    g.manual_seed(1234)
    perm = torch.randperm(npg + 7, generator=g, device=dev)[:npg].to(torch.int32)[None, :].contiguous()
    pool = kp.Pool(1, npg + 7, Hkv, d)
    kv = torch.randn((n, 2, Hkv, d), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    kp.kv_append(pool, 0, kv[:, 0].contiguous(), kv[:, 1].contiguous(), perm, [0], [0, n])
    del kv
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    res = {"ctx": ctx}
    for C in chunks:
        q = torch.randn((C, Hq, d), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
        ws = torch.empty(kp.prefix_chunk_prefill_workspace_size(pool, [ctx], [0, C], Hq), dtype=torch.uint8,
                         device=dev)
        out = torch.empty((C, Hq, d), dtype=torch.bfloat16, device=dev)
        ts = []
        for it in range(reps + 3):
            # Two passes over the flush buffer (about 150 us of device work) queued ahead of the start
            # event: the host call is submitted while they run, so the events time the device work only
            # (the host's own time is reported beside it).
            flush.fill_(1)
            flush.fill_(2)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            kp.prefix_chunk_prefill_attn(q, pool, 0, perm, [ctx], [0, C], out=out, ws=ws)
            e1.record(stream)
            torch.cuda.synchronize()
            if it >= 3:
                ts.append(e0.elapsed_time(e1) / 1e3)
        torch.cuda.synchronize()
        hs = []
        for _ in range(5):
            h0 = time.perf_counter()
            kp.prefix_chunk_prefill_attn(q, pool, 0, perm, [ctx], [0, C], out=out, ws=ws)
            hs.append((time.perf_counter() - h0) * 1e3)
        torch.cuda.synchronize()
        t = float(np.median(ts))
        flops = 4 * d * Hq * (C * ctx + C * (C + 1) // 2)
        kv_bytes = (ctx + C) * Hkv * d * 2 * 2
        res[f"C{C}"] = {"ms": round(t * 1e3, 4), "host_call_ms": round(float(np.median(hs)), 4),
                        "tflops": round(flops / t / 1e12, 2),
                        "mfma_frac": round(flops / t / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                        "kv_gbs": round(kv_bytes / t / 1e9, 1), "algorithmic_flops": flops, "kv_bytes": kv_bytes}
    if pool.device_error() != kp.KVP_OK:
        raise RuntimeError("device error in the split-prefill leg")
    pool.close()
    del flush
    return res


def mixed_step_leg(kp, pool, w, vals, gp, bt, flush, stream, s0: int, s1: int, cu_q, reps: int = 10) -> dict:
    """The step's attention (decode of every sequence and prefill of the chunks) as one mixed_step_attn
    launch, against the two separate calls, on the same pool and inputs: runs interleaved, each after the
    cache flush, timed with HIP events on the launch stream.  The outputs are compared bitwise."""
    import torch
    dev = vals.q.device
    od = torch.empty((w.B, w.Hq, w.d), dtype=torch.bfloat16, device=dev)
    op = torch.empty((int(cu_q[-1]), w.Hq, w.d), dtype=torch.bfloat16, device=dev)
    rd, rp = torch.empty_like(od), torch.empty_like(op)
    ws = torch.empty(max(1, kp.mixed_step_workspace_size(pool, w.decode_len, w.prefill_ctx, cu_q, w.Hq, gp)),
                     dtype=torch.uint8, device=dev)
    dws = torch.empty(max(1, kp.paged_decode_workspace_size(pool, w.decode_len, w.Hq, gp)), dtype=torch.uint8,
                      device=dev)
    pws = torch.empty(max(1, kp.prefix_chunk_prefill_workspace_size(pool, w.prefill_ctx, cu_q, w.Hq)),
                      dtype=torch.uint8, device=dev)
    btp = bt[s0:s1]

    def fused():
        kp.mixed_step_attn(pool, 0, vals.q, bt, w.decode_len, vals.qp, btp, w.prefill_ctx, cu_q, group_prefix=gp,
                           scale=w.scale, out_dec=od, out_pf=op, ws=ws)

    def separate():
        kp.paged_decode_attn(vals.q, pool, 0, bt, w.decode_len, group_prefix=gp, scale=w.scale, out=rd, ws=dws)
        kp.prefix_chunk_prefill_attn(vals.qp, pool, 0, btp, w.prefill_ctx, cu_q, scale=w.scale, out=rp, ws=pws)

    t = {"fused": [], "separate": []}
    for it in range(reps + 1):
        for name, fn in (("separate", separate), ("fused", fused)):
            flush.fill_(1)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            if it >= 1:
                t[name].append(e0.elapsed_time(e1))
    if pool.device_error() != kp.KVP_OK:
        raise RuntimeError("device error in the mixed-step leg")
    same = bool(torch.equal(od, rd) and torch.equal(op, rp))
    f, sep = float(np.median(t["fused"])), float(np.median(t["separate"]))
    return {"fused_ms": round(f, 4), "separate_ms": round(sep, 4), "speedup": round(sep / f, 4),
            "fused_ms_p10_p90": [round(float(np.percentile(t["fused"], q)), 4) for q in (10, 90)],
            "separate_ms_p10_p90": [round(float(np.percentile(t["separate"], q)), 4) for q in (10, 90)],
            "outputs_bitwise_equal": same, "reps": reps}


def cpu_baseline(w, vals, budget_s: float):
    """Time the CPU fp64 oracle (as it stands) on a bounded sample of the same decode workload."""
    import oracle
    from paper_2608_11152_amd import workloads as W
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        blas_threads = None
    order = [i for i in range(w.B) if w.decode_len[i] > 0]
    order.sort(key=lambda i: int(w.decode_len[i]))  # shortest first: many sessions within the budget
    q_all = W.to_numpy_bits(vals.q)
    done_bytes, done_tok, secs, passes = 0, 0, 0.0, 0
    kv_cache = {}
    while secs < budget_s:  # whole passes over the decode batch until the time budget is used
        for i in order:
            n = int(w.decode_len[i])
            if i not in kv_cache:
                kv_cache[i] = W.seq_kv_bits(w, vals, i, n)
            k, v = kv_cache[i]
            t0 = time.perf_counter()
            oracle.decode_seq(q_all[i], oracle.widen_bf16(k), oracle.widen_bf16(v), w.scale)
            secs += time.perf_counter() - t0
            done_bytes += n * w.Hkv * w.d * 4
            done_tok += 1
            if secs >= budget_s and passes == 0 and len(kv_cache) < len(order):
                break
        passes += 1
    # Put the rate on the byte basis of `value`: the oracle reads every sequence's KV (a shared prompt once
    # per sample), so its time for the whole batch is the sample time scaled by the batch's logical bytes
    # over the sample's; `value` divides the batch's algorithmic (unique) bytes by that time.
    batch_logical = sum(int(w.decode_len[i]) for i in order) * w.Hkv * w.d * 4
    batch_s = secs * batch_logical / done_bytes
    unique = decode_algorithmic_bytes(w)
    return {
        "value": round(unique / batch_s / 1e9, 4), "unit": "GB/s", "cores": blas_threads or os.cpu_count(),
        "kind": "oracle",
        "bytes": "value = the batch's algorithmic decode bytes (as in the GPU value: unique KV with a group's "
                 "shared pages once, Q, O, page-table entries) / the oracle's time for the whole batch, "
                 "extrapolated from the sample by logical KV bytes; logical_gbs = the sample's logical KV "
                 "bytes (every sample's own KV) / its time",
        "logical_gbs": round(done_bytes / secs / 1e9, 4),
        "sample": f"numpy fp64 oracle decode (oracle.decode_seq) of the workload's {len(order)} decode sessions, "
                  f"{passes} pass(es), {done_tok} sequence decodes, {done_bytes / 1e9:.2f} GB of logical KV "
                  f"(contiguous per-sequence K/V, page gather excluded), {secs:.1f} s of CPU time; "
                  f"decode tokens/s = {done_tok / secs:.3f}; os.cpu_count()={os.cpu_count()}, "
                  f"affinity={len(os.sched_getaffinity(0))}, blas_threads={blas_threads}",
        "decode_tokens_per_s": round(done_tok / secs, 4),
    }


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "the library runs on one GPU; sharding across GPUs is not implemented, so "
                                   "--gpus must be 1", "n_gpus": args.gpus}))
        sys.exit(2)
    import torch

    from paper_2608_11152_amd import kvpattn as kp
    from paper_2608_11152_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = W.make_workload(args.workload)
    vals = W.make_values(w, values="torch", device=dev)
    gp = kp.group_prefix(w.group_id, w.shared_pages) if w.num_groups else None
    pool = kp.Pool(1, w.num_pages, w.Hkv, w.d)
    bt = torch.from_numpy(w.block_tables).to(dev)

    def append_batch(ab):
        rows = torch.from_numpy(ab.src_rows).to(dev)
        return (vals.kv[rows, 0].contiguous(), vals.kv[rows, 1].contiguous(), ab)

    for ab in w.setup_appends:
        k, v, _ = append_batch(ab)
        kp.kv_append(pool, 0, k, v, bt, ab.start_pos, ab.cu_new, group_prefix=gp if ab.use_group_prefix else None)
        del k, v
    step_batches = [append_batch(ab) for ab in w.step_appends]
    has_prefill = len(w.prefill_seqs) > 0
    dec_ws = torch.empty(kp.paged_decode_workspace_size(pool, w.decode_len, w.Hq, gp), dtype=torch.uint8, device=dev)
    dec_out = torch.empty((w.B, w.Hq, w.d), dtype=torch.bfloat16, device=dev)
    if has_prefill:
        s0, s1 = int(w.prefill_seqs[0]), int(w.prefill_seqs[-1]) + 1
        cu_q = w.cu_q()
        pf_ws = torch.empty(max(1, kp.prefix_chunk_prefill_workspace_size(pool, w.prefill_ctx, cu_q, w.Hq)),
                            dtype=torch.uint8, device=dev)
        pf_out = torch.empty((int(cu_q[-1]), w.Hq, w.d), dtype=torch.bfloat16, device=dev)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    def step(ev=None):
        if not args.no_flush:
            flush.fill_(1)
        if ev:
            ev[0].record(stream)
        for k, v, ab in step_batches:
            kp.kv_append(pool, 0, k, v, bt, ab.start_pos, ab.cu_new, group_prefix=gp if ab.use_group_prefix else None)
        if ev:
            ev[1].record(stream)
        kp.paged_decode_attn(vals.q, pool, 0, bt, w.decode_len, group_prefix=gp, scale=w.scale, out=dec_out,
                             ws=dec_ws)
        if ev:
            ev[2].record(stream)
        if has_prefill:
            kp.prefix_chunk_prefill_attn(vals.qp, pool, 0, bt[s0:s1], w.prefill_ctx, cu_q, scale=w.scale,
                                         out=pf_out, ws=pf_ws)
        if ev:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    err = pool.device_error()
    if err != kp.KVP_OK:
        raise RuntimeError(f"device error {err} during the benchmark")
    # Host time of each call (validation, planning, packing, launch), from 5 back-to-back calls after a
    # synchronisation: inside the timed loop the host runs ahead until the library's ring of 8 pinned
    # staging slots is full and then waits there for earlier steps, so a call's time there measures the
    # GPU, not the host.
    def host_time(fn):
        torch.cuda.synchronize()
        ts = []
        for _ in range(5):
            h0 = time.perf_counter()
            fn()
            ts.append((time.perf_counter() - h0) * 1e3)
        torch.cuda.synchronize()
        return ts
    host_dec = host_time(lambda: kp.paged_decode_attn(vals.q, pool, 0, bt, w.decode_len, group_prefix=gp,
                                                      scale=w.scale, out=dec_out, ws=dec_ws))
    host_pf = host_time(lambda: kp.prefix_chunk_prefill_attn(vals.qp, pool, 0, bt[s0:s1], w.prefill_ctx, cu_q,
                                                             scale=w.scale, out=pf_out, ws=pf_ws)) if has_prefill else [0.0]
    host_ms = [(host_dec[i], host_pf[min(i, len(host_pf) - 1)]) for i in range(len(host_dec))]
    t_app = np.array([e[0].elapsed_time(e[1]) for e in evs])
    t_dec = np.array([e[1].elapsed_time(e[2]) for e in evs])
    t_pf = np.array([e[2].elapsed_time(e[3]) for e in evs])

    # Plain device copy of 1 GiB (2 GiB of HBM traffic): the bandwidth a streaming kernel reaches here.
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(5):
        dst.copy_(src)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * (1 << 30) / (c0.elapsed_time(c1) / 1e3) / 1e9
    del src, dst
    gemm_tflops = library_gemm_tflops(dev, stream) if has_prefill else None

    traffic = profiled_traffic(args.workload)
    traffic_dec, traffic_pf = traffic["decode"], traffic["prefill"]
    dec_bytes = decode_algorithmic_bytes(w)
    dec_s = float(np.median(t_dec)) / 1e3
    dec_gbs = dec_bytes / dec_s / 1e9
    n_dec = int((w.decode_len > 0).sum())
    res = {
        "metric": METRIC,
        "value": round(dec_gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": WORKLOAD_TEXT[args.workload], "sessions": w.B, "decode_sessions": n_dec,
                   "prefill_chunks": int(len(w.prefill_seqs)), "pool_pages": w.num_pages,
                   "unique_decode_tokens": w.unique_decode_tokens(),
                   "logical_decode_tokens": w.logical_decode_tokens(), "seed": w.seed},
        "decode_hbm_peak_frac": round(dec_gbs / HBM_PEAK_GBS, 4),
        "decode_tokens_per_s": round(n_dec / dec_s, 1),
        "decode_ms": {"median": round(float(np.median(t_dec)), 4), "mean": round(float(np.mean(t_dec)), 4),
                      "p10": round(float(np.percentile(t_dec, 10)), 4),
                      "p90": round(float(np.percentile(t_dec, 90)), 4)},
        "append_ms": round(float(np.median(t_app)), 4),
        "host_call_ms": {"paged_decode_attn": round(float(np.median([h[0] for h in host_ms])), 4),
                         "prefix_chunk_prefill_attn": round(float(np.median([h[1] for h in host_ms])), 4)},
        "hbm_copy_gbs": round(copy_gbs, 1),
        "roofline": {"bound": "hbm", "achieved": round(dec_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(dec_gbs / HBM_PEAK_GBS, 4), "traffic": traffic_dec,
                     "kernel": "paged_decode_attn (shared-prefix + split-KV partial kernels and LSE merge)",
                     "algorithmic_bytes_per_launch": dec_bytes},
    }
    if has_prefill:
        pf_s = float(np.median(t_pf)) / 1e3
        flops = w.prefill_flops()
        res["prefill_ms"] = {"median": round(float(np.median(t_pf)), 4), "mean": round(float(np.mean(t_pf)), 4),
                             "p10": round(float(np.percentile(t_pf, 10)), 4),
                             "p90": round(float(np.percentile(t_pf, 90)), 4)}
        res["prefill_tflops"] = round(flops / pf_s / 1e12, 2)
        res["roofline_prefill"] = {"bound": "mfma", "achieved": round(flops / pf_s / 1e12, 2),
                                   "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                   "frac": round(flops / pf_s / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4),
                                   "traffic": traffic_pf,
                                   "kernel": "prefix_chunk_prefill_attn", "algorithmic_flops_per_launch": flops,
                                   "algorithmic_bytes_per_launch": prefill_algorithmic_bytes(w),
                                   "library_gemm_tflops": gemm_tflops,
                                   "frac_of_library_gemm": round(flops / pf_s / 1e12 / gemm_tflops, 4)}
    if not args.no_fp8:
        res["fp8_kv"] = fp8_kv_leg(kp, w, vals, gp, bt, step_batches, flush, stream, min(args.steps, 10), 2, dec_s,
                                   has_prefill, s0 if has_prefill else 0, s1 if has_prefill else 0,
                                   cu_q if has_prefill else None)
        res["fp8_kv"]["decode_traffic"] = traffic["decode_fp8"]
        if has_prefill:
            res["fp8_kv"]["prefill_traffic"] = traffic["prefill_fp8"]
    if has_prefill and not args.no_mixed_step:
        res["mixed_step"] = mixed_step_leg(kp, pool, w, vals, gp, bt, flush, stream, s0, s1, cu_q)
    if not args.no_prefill_split:
        res["prefill_split"] = prefill_split_leg(kp, dev, stream)
    res["kv_tier"] = kv_tier_leg(kp, pool, w, stream)
    res["prefix_hash"] = prefix_hash_leg(kp, W, w, stream)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, vals, args.cpu_seconds)
    print(json.dumps(res), flush=True)
    pool.close()


if __name__ == "__main__":
    main()
