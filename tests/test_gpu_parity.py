"""GPU parity of the HIP path (through the C-ABI) against the CPU fp64 oracle, on reduced-size versions of
every workload class (several tiles, ragged tails), plus the bit-exact properties of the paged layout."""
import numpy as np
import pytest

import oracle
from paper_2608_11152_amd import kvpattn as kp
from paper_2608_11152_amd import workloads as W

from gpu_helpers import GpuCase, assert_close, note, to_dev_bits

pytestmark = pytest.mark.gpu

DECODE_CASES = ["tiny", "rlvr_s", "rlhf_s", "agentic_s", "mixed_s", "rlvr_d64"]


@pytest.fixture(scope="module")
def cases():
    return {}


def get_case(cases, name):
    if name not in cases:
        note(f"setup {name}")
        cases[name] = GpuCase(W.make_workload(name))
    return cases[name]


# ------------------------------------------------------------------------------------------------
# kv_append: bit-exact round trip and the documented pool layout
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny", "mixed_s", "rlvr_d64"])
def test_append_round_trip_bitwise(cases, name):
    c = get_case(cases, name)
    w = c.w
    note(f"kv_gather {name}")
    k, v = kp.kv_gather(c.pool, 0, c.bt, w.final_len)
    import torch
    torch.cuda.synchronize()
    kb = k.view(torch.int16).cpu().numpy().view(np.uint16)
    vb = v.view(torch.int16).cpu().numpy().view(np.uint16)
    off = 0
    for i in range(w.B):
        n = int(w.final_len[i])
        ek, ev = W.seq_kv_bits(w, c.vals, i)
        assert np.array_equal(kb[off:off + n], ek), f"K of sequence {i}"
        assert np.array_equal(vb[off:off + n], ev), f"V of sequence {i}"
        off += n
    assert c.pool.device_error() == kp.KVP_OK


def _layout_index(D, t, c, which):
    """Element offset inside a (page, head) block as documented in include/kvpattn.h."""
    if which == 0:
        return ((c // 8) * 16 + t) * 8 + c % 8
    s = (t & ~12) | ((t & 4) << 1) | ((t & 8) >> 1)
    return 16 * D + (((c // 16) * 2 + s // 8) * 16 + c % 16) * 8 + s % 8


@pytest.mark.parametrize("name", ["tiny", "rlvr_d64"])
def test_pool_raw_layout_matches_header(cases, name):
    c = get_case(cases, name)
    w = c.w
    raw = c.pool.layer_raw(0).cpu().numpy().view(np.uint16).reshape(c.num_pages, w.Hkv, 2 * 16 * w.d)
    pk, pv = c.oracle_pool()
    D = w.d
    t = np.arange(16)[:, None]
    cc = np.arange(D)[None, :]
    ik = _layout_index(D, t, cc, 0)
    iv = _layout_index(D, t, cc, 1)
    for page in np.unique(w.block_tables[w.block_tables >= 0])[:40]:
        for h in range(w.Hkv):
            assert np.array_equal(raw[page, h][ik], pk[page, h]), (page, h)
            assert np.array_equal(raw[page, h][iv], pv[page, h]), (page, h)


# ------------------------------------------------------------------------------------------------
# decode parity
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name", DECODE_CASES)
def test_decode_parity_f32(cases, name):
    c = get_case(cases, name)
    note(f"decode {name} f32")
    got = c.decode()
    assert_close(got, c.oracle_decode(), f"decode {name}")
    assert c.pool.device_error() == kp.KVP_OK


@pytest.mark.parametrize("name", ["tiny", "rlvr_s", "mixed_s"])
def test_decode_parity_bf16_out(cases, name):
    import torch
    c = get_case(cases, name)
    note(f"decode {name} bf16")
    got = c.decode(out_dtype=torch.bfloat16)
    assert_close(got, c.oracle_decode(), f"decode {name} bf16-out")


@pytest.mark.parametrize("name", ["rlvr_s", "rlhf_s", "mixed_s", "rlvr_d64"])
def test_decode_shared_prefix_hint_vs_none(cases, name):
    """The group-prefix hint reads shared pages once per group; the result must match the ungrouped run."""
    c = get_case(cases, name)
    note(f"decode {name} with / without group hint")
    a = c.decode()
    b = c.decode(group_prefix=None)
    ref = c.oracle_decode()
    assert_close(a, ref, f"{name} grouped")
    assert_close(b, ref, f"{name} ungrouped")
    assert_close(a, b.cpu().numpy().astype(np.float64), f"{name} grouped vs ungrouped")


def test_decode_page_permutation_bitwise():
    """Same logical content under a different physical page assignment: bitwise identical outputs."""
    import torch
    w = W.make_workload("mixed_s")
    vals = W.make_values(w)
    a = GpuCase(w, vals)
    perm = np.random.default_rng(77).permutation(w.num_pages)
    bt2 = np.where(w.block_tables >= 0, perm[np.maximum(w.block_tables, 0)], -1).astype(np.int32)
    b = GpuCase(w, vals, block_tables=bt2)
    note("decode permutation")
    oa, ob = a.decode(), b.decode()
    assert torch.equal(oa, ob)
    pa, pb = a.prefill(), b.prefill()
    assert torch.equal(pa, pb)


def test_decode_deterministic(cases):
    import torch
    c = get_case(cases, "rlvr_s")
    note("decode determinism")
    assert torch.equal(c.decode(), c.decode())


def test_many_calls_in_flight_on_two_streams(cases):
    """Two dozen decode and prefill calls queued on two streams with no host synchronisation in between,
    more than the library's pinned metadata slots (a slot is reused only after the GPU work that read it
    has completed). Each call has its own lengths, so a slot handed out too early would show: every
    output must equal the same call made alone."""
    import torch
    c = get_case(cases, "mixed_s")
    w = c.w
    q, qp = to_dev_bits(c.vals.q), to_dev_bits(c.vals.qp)
    s0, s1 = int(w.prefill_seqs[0]), int(w.prefill_seqs[-1]) + 1
    floor = np.zeros(w.B, np.int64)
    if w.num_groups:
        grouped = w.group_id >= 0
        floor[grouped] = w.shared_pages[w.group_id[grouped]] * 16
    variants = []
    for k in range(4):
        lens = np.maximum(w.decode_len - 5 * k, np.minimum(w.decode_len, floor + 1)).astype(np.int32)
        variants.append(("decode", lens, c.gp if k % 2 == 0 else None))
    variants.append(("prefill", None, None))

    def call(v, stream):
        kind, lens, gp = v
        if kind == "prefill":
            return kp.prefix_chunk_prefill_attn(qp, c.pool, 0, c.bt[s0:s1], w.prefill_ctx, w.cu_q(), scale=w.scale,
                                                stream=stream)
        return kp.paged_decode_attn(q, c.pool, 0, c.bt, lens, group_prefix=gp, scale=w.scale, stream=stream)

    note("many calls in flight: references")
    refs = [call(v, None) for v in variants]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    note("many calls in flight: 24 calls on two streams")
    outs = []
    for k in range(24):
        s = streams[k % 2]
        with torch.cuda.stream(s):
            outs.append((k % len(variants), call(variants[k % len(variants)], s)))
    torch.cuda.synchronize()
    for v, out in outs:
        assert torch.equal(out, refs[v]), f"call of variant {v} differs from the same call made alone"


def test_default_buffers_belong_to_the_call_stream(cases, monkeypatch):
    """Calls on a side stream given as an argument (no stream context): the workspace and output the
    binding allocates must belong to that stream, so memory allocated on the current stream afterwards
    (while the side stream's kernels may still be pending) never aliases them, and the outputs equal the
    same calls on the current stream."""
    import torch
    c = get_case(cases, "mixed_s")
    w = c.w
    q, qp = to_dev_bits(c.vals.q), to_dev_bits(c.vals.qp)
    s0, s1 = int(w.prefill_seqs[0]), int(w.prefill_seqs[-1]) + 1
    ref_d = kp.paged_decode_attn(q, c.pool, 0, c.bt, w.decode_len, group_prefix=c.gp, scale=w.scale)
    ref_p = kp.prefix_chunk_prefill_attn(qp, c.pool, 0, c.bt[s0:s1], w.prefill_ctx, w.cu_q(), scale=w.scale)
    torch.cuda.synchronize()
    made = []
    real = kp._alloc_on

    def spy(stream, shape, dtype, device):
        t = real(stream, shape, dtype, device)
        made.append((t.data_ptr(), t.numel() * t.element_size()))
        return t

    monkeypatch.setattr(kp, "_alloc_on", spy)
    side = torch.cuda.Stream()
    note("side-stream calls with binding-allocated buffers")
    with torch.cuda.stream(side):
        torch.cuda._sleep(20_000_000)  # keep the side stream busy so its kernels are still pending below
    out_d = kp.paged_decode_attn(q, c.pool, 0, c.bt, w.decode_len, group_prefix=c.gp, scale=w.scale, stream=side)
    out_p = kp.prefix_chunk_prefill_attn(qp, c.pool, 0, c.bt[s0:s1], w.prefill_ctx, w.cu_q(), scale=w.scale,
                                         stream=side)
    junk = [torch.full((n,), 255, dtype=torch.uint8, device="cuda") for _, n in made]
    for t in junk:
        lo, hi = t.data_ptr(), t.data_ptr() + t.numel()
        assert all(hi <= p0 or p0 + n <= lo for p0, n in made), "current-stream memory aliases a pending buffer"
    side.synchronize()
    torch.cuda.synchronize()
    assert torch.equal(out_d, ref_d) and torch.equal(out_p, ref_p)
    del junk


def test_decode_duplicated_prefix_pages_match_shared(cases):
    """Members given private copies of the prompt pages (no sharing) give the shared-page result."""
    w = W.make_workload("rlvr_d64")
    vals = W.make_values(w)
    shared = GpuCase(w, vals)
    # Build a workload where every member owns copies of the prompt pages.
    wd = W.make_workload("rlvr_d64")
    extra = int(sum(w.shared_pages[g] * (np.sum(w.group_id == g) - 1) for g in range(w.num_groups)))
    bt = w.block_tables.copy()
    nxt = w.num_pages
    seen = set()
    for i in range(w.B):
        g = int(w.group_id[i])
        if g in seen:
            for j in range(int(w.shared_pages[g])):
                bt[i, j] = nxt
                nxt += 1
        seen.add(g)
    assert nxt == w.num_pages + extra
    wd.block_tables = bt
    wd.shared_pages = np.zeros_like(w.shared_pages)
    # every sequence appends its whole prefix into its own pages
    import copy
    ab = copy.deepcopy(w.setup_appends[1])
    cnt = np.diff(ab.cu_new)
    rows = []
    for i in range(w.B):
        rows.append(w.token_rows[i][: int(ab.start_pos[i]) + int(cnt[i])])
    ab.start_pos = np.zeros(w.B, np.int32)
    ab.cu_new = np.concatenate([[0], np.cumsum([len(r) for r in rows])]).astype(np.int32)
    ab.src_rows = np.concatenate(rows)
    wd.setup_appends = [ab]
    dup = GpuCase(wd, vals, num_pages=nxt)
    note("decode duplicated prefix")
    a, b = shared.decode(), dup.decode(group_prefix=None)
    assert_close(b, shared.oracle_decode(), "duplicated prefix vs oracle")
    assert_close(a, b.cpu().numpy().astype(np.float64), "shared vs duplicated")


# ------------------------------------------------------------------------------------------------
# prefill parity
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["agentic_s", "mixed_s"])
def test_prefill_parity(cases, name):
    c = get_case(cases, name)
    note(f"prefill {name}")
    got = c.prefill()
    assert_close(got, c.oracle_prefill(), f"prefill {name}")
    assert c.pool.device_error() == kp.KVP_OK


def test_prefill_bf16_out(cases):
    import torch
    c = get_case(cases, "agentic_s")
    note("prefill bf16")
    assert_close(c.prefill(out_dtype=torch.bfloat16), c.oracle_prefill(), "prefill agentic_s bf16-out")


@pytest.mark.parametrize("ctx,C,G", [(0, 37, 8), (0, 1, 8), (5, 1, 8), (16, 16, 4), (33, 130, 2), (1000, 3, 16),
                                     (47, 64, 1)])
def test_prefill_shapes(ctx, C, G):
    """Causal ctx = 0, single-row chunks, page-aligned and ragged contexts, every GQA ratio."""
    import torch
    Hkv, d = 2, 128 if G != 16 else 64
    Hq = G * Hkv
    rng = np.random.default_rng(ctx * 1000 + C + G)
    n = ctx + C
    npg = (n + 15) // 16
    num_pages = npg + 5
    bt = rng.permutation(num_pages)[:npg].astype(np.int32)[None, :]
    kvb = W.f32_to_bf16_bits(rng.standard_normal((n, 2, Hkv, d), dtype=np.float32))
    qb = W.f32_to_bf16_bits(rng.standard_normal((C, Hq, d), dtype=np.float32))
    pool = kp.Pool(1, num_pages, Hkv, d)
    btd = torch.from_numpy(bt).cuda()
    kvd = to_dev_bits(kvb)
    note(f"prefill shape ctx={ctx} C={C} G={G}")
    kp.kv_append(pool, 0, kvd[:, 0].contiguous(), kvd[:, 1].contiguous(), btd, [0], [0, n])
    out = kp.prefix_chunk_prefill_attn(to_dev_bits(qb), pool, 0, btd, [ctx], [0, C], scale=0.09)
    torch.cuda.synchronize()
    ref = oracle.prefill_seq(qb, oracle.widen_bf16(kvb[:, 0]), oracle.widen_bf16(kvb[:, 1]), 0.09, ctx)
    assert_close(out, ref, f"prefill ctx={ctx} C={C} G={G}")
    # a chunk of one row is a decode step over ctx + 1 tokens
    if C == 1:
        dec = kp.paged_decode_attn(to_dev_bits(qb), pool, 0, btd, [n], scale=0.09)
        torch.cuda.synchronize()
        # same bf16 weights and weight sums; only fp32 summation order differs (a rare bf16 rounding flip of
        # one weight moves an output by ~2^-9 of that weight's share)
        assert_close(dec, out.cpu().numpy().astype(np.float64), "decode == prefill of one row", 2e-4, 1e-5)


# ------------------------------------------------------------------------------------------------
# edge cases and errors
# ------------------------------------------------------------------------------------------------

@pytest.mark.parametrize("pattern", ["rising", "falling", "wide"])
def test_softmax_dynamic_range(pattern):
    """Scores far from N(0, 1): rising along the sequence (the running max moves by more than 8 (log2) in
    almost every 64-key stage, so the kernels rescale every stage), falling (the max is at key 0 and later
    weights fall to 2^-100), and wide (scores of std ~50 in log2 units, weights nearly one-hot)."""
    import torch
    G, Hkv, d, ctx, C = 8, 2, 128, 700, 70
    Hq, n = G * Hkv, ctx + C
    rng = np.random.default_rng({"rising": 1, "falling": 2, "wide": 3}[pattern])
    u = rng.standard_normal(d).astype(np.float32)
    if pattern == "wide":
        k = 6.0 * rng.standard_normal((n, Hkv, d)).astype(np.float32)
        q = 6.0 * rng.standard_normal((C, Hq, d)).astype(np.float32)
    else:
        a = np.linspace(-6.0, 6.0, n, dtype=np.float32)
        if pattern == "falling":
            a = a[::-1].copy()
        k = a[:, None, None] * u[None, None, :] + 0.3 * rng.standard_normal((n, Hkv, d)).astype(np.float32)
        q = u[None, None, :] + 0.3 * rng.standard_normal((C, Hq, d)).astype(np.float32)
    v = rng.standard_normal((n, Hkv, d)).astype(np.float32)
    kvb = W.f32_to_bf16_bits(np.stack([k, v], axis=1))
    qb = W.f32_to_bf16_bits(q)
    npg = (n + 15) // 16
    num_pages = npg + 3
    bt = rng.permutation(num_pages)[:npg].astype(np.int32)[None, :]
    pool = kp.Pool(1, num_pages, Hkv, d)
    btd = torch.from_numpy(bt).cuda()
    kvd = to_dev_bits(kvb)
    note(f"softmax dynamic range {pattern}")
    kp.kv_append(pool, 0, kvd[:, 0].contiguous(), kvd[:, 1].contiguous(), btd, [0], [0, n])
    out = kp.prefix_chunk_prefill_attn(to_dev_bits(qb), pool, 0, btd, [ctx], [0, C], scale=0.09)
    dec = kp.paged_decode_attn(to_dev_bits(qb[C - 1:]), pool, 0, btd, [n], scale=0.09)
    torch.cuda.synchronize()
    kf, vf = oracle.widen_bf16(kvb[:, 0]), oracle.widen_bf16(kvb[:, 1])
    ref = oracle.prefill_seq(qb, kf, vf, 0.09, ctx)
    assert np.all(np.isfinite(ref))
    assert_close(out, ref, f"prefill {pattern}")
    assert_close(dec, ref[C - 1:], f"decode {pattern}")


@pytest.mark.parametrize("G,d", [(1, 128), (2, 64), (4, 128), (16, 64), (16, 128)])
def test_decode_edge_lengths(G, d):
    """Empty, single-token, page-aligned and ragged sequences, long sequences split many ways."""
    import torch
    lens = [0, 1, 2, 15, 16, 17, 31, 32, 33, 250, 4097, 0, 9000]
    Hkv = 2
    Hq = G * Hkv
    rng = np.random.default_rng(G * 7 + d)
    pages = [(n + 15) // 16 for n in lens]
    maxp = max(pages)
    num_pages = sum(pages) + 3
    perm = rng.permutation(num_pages).astype(np.int32)
    bt = np.full((len(lens), maxp), -1, np.int32)
    o = 0
    for i, p in enumerate(pages):
        bt[i, :p] = perm[o:o + p]
        o += p
    T = sum(lens)
    kvb = W.f32_to_bf16_bits(rng.standard_normal((T, 2, Hkv, d), dtype=np.float32))
    qb = W.f32_to_bf16_bits(rng.standard_normal((len(lens), Hq, d), dtype=np.float32))
    pool = kp.Pool(1, num_pages, Hkv, d)
    btd = torch.from_numpy(bt).cuda()
    kvd = to_dev_bits(kvb)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    note(f"decode edge lengths G={G} d={d}")
    kp.kv_append(pool, 0, kvd[:, 0].contiguous(), kvd[:, 1].contiguous(), btd, np.zeros(len(lens), np.int32), cu)
    out = kp.paged_decode_attn(to_dev_bits(qb), pool, 0, btd, lens, scale=0.1)
    torch.cuda.synchronize()
    pk, pv = oracle.new_pool(num_pages, Hkv, d)
    oracle.append(pk, pv, kvb[:, 0], kvb[:, 1], bt, np.zeros(len(lens), np.int32), cu)
    ref = oracle.decode(qb, pk, pv, bt, lens, 0.1)
    assert_close(out, ref, f"edge lengths G={G} d={d}")
    assert np.all(out[0].cpu().numpy() == 0) and np.all(out[11].cpu().numpy() == 0)


@pytest.mark.parametrize("lens", [[32773], [32773, 0, 16001]])
def test_decode_few_long_sequences_many_partials(lens):
    """A call of a few long sequences is cut into short (8-page) segments to fill the GPU: one 32k-token
    sequence alone becomes hundreds of partials per KV head, all folded by the merge."""
    import torch
    Hq, Hkv, d = 32, 4, 128
    _, parts, seg = kp.kvp_plan_decode(np.array(lens, np.int32), Hq, Hkv)
    assert seg == 8 and parts >= 200, (parts, seg)
    rng = np.random.default_rng(sum(lens))
    pages = [(n + 15) // 16 for n in lens]
    num_pages = sum(pages) + 3
    perm = rng.permutation(num_pages).astype(np.int32)
    bt = np.full((len(lens), max(pages)), -1, np.int32)
    o = 0
    for i, pg in enumerate(pages):
        bt[i, :pg] = perm[o:o + pg]
        o += pg
    T = sum(lens)
    kvb = W.f32_to_bf16_bits(rng.standard_normal((T, 2, Hkv, d), dtype=np.float32))
    qb = W.f32_to_bf16_bits(rng.standard_normal((len(lens), Hq, d), dtype=np.float32))
    pool = kp.Pool(1, num_pages, Hkv, d)
    btd = torch.from_numpy(bt).cuda()
    kvd = to_dev_bits(kvb)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    note(f"decode few long sequences {lens}: {parts} partials")
    kp.kv_append(pool, 0, kvd[:, 0].contiguous(), kvd[:, 1].contiguous(), btd, np.zeros(len(lens), np.int32), cu)
    out = kp.paged_decode_attn(to_dev_bits(qb), pool, 0, btd, lens, scale=0.0884)
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    pk, pv = oracle.new_pool(num_pages, Hkv, d)
    oracle.append(pk, pv, kvb[:, 0], kvb[:, 1], bt, np.zeros(len(lens), np.int32), cu)
    ref = oracle.decode(qb, pk, pv, bt, lens, 0.0884)
    assert_close(out, ref, f"few long sequences {lens}")
    pool.close()


def test_host_errors_enqueue_nothing(cases):
    import torch
    c = get_case(cases, "tiny")
    w = c.w
    q = to_dev_bits(c.vals.q)
    sentinel = torch.full((w.B, w.Hq, w.d), 7.0, device="cuda")
    too_long = w.decode_len.copy()
    too_long[1] = w.maxp * 16 + 1
    with pytest.raises(kp.KvpError) as e:
        kp.paged_decode_attn(q, c.pool, 0, c.bt, too_long, out=sentinel)
    assert e.value.code == kp.KVP_ERANGE
    # a call whose sequences fit one wave segment (8 pages in all) has no partials and needs no
    # workspace; a workload with partials needs one
    assert kp.paged_decode_workspace_size(c.pool, np.array([16, 30, 60, 1], np.int32), w.Hq) == 0
    cr = get_case(cases, "rlvr_s")
    need = kp.paged_decode_workspace_size(cr.pool, cr.w.decode_len, cr.w.Hq, cr.gp)
    assert need > 8
    ws = torch.empty(need - 8, dtype=torch.uint8, device="cuda")
    sentinel_r = torch.full((cr.w.B, cr.w.Hq, cr.w.d), 7.0, device="cuda")
    with pytest.raises(kp.KvpError) as e:
        kp.paged_decode_attn(to_dev_bits(cr.vals.q), cr.pool, 0, cr.bt, cr.w.decode_len, group_prefix=cr.gp,
                             out=sentinel_r, ws=ws)
    assert e.value.code == kp.KVP_EWORKSPACE
    assert torch.all(sentinel_r == 7.0)
    with pytest.raises(kp.KvpError) as e:
        kp.paged_decode_attn(q, c.pool, 0, c.bt, w.decode_len, out=sentinel, scale=-1.0)
    assert e.value.code == kp.KVP_EINVAL
    with pytest.raises(kp.KvpError) as e:
        kp.paged_decode_attn(q, c.pool, 3, c.bt, w.decode_len, out=sentinel)
    assert e.value.code == kp.KVP_EINVAL
    torch.cuda.synchronize()
    assert torch.all(sentinel == 7.0)
    # kv_append into a shared page is refused when the group hint is given
    g = W.make_workload("rlvr_d64")
    cg = get_case(cases, "rlvr_d64")
    kv = cg.kv_dev[:1]
    member = int(np.flatnonzero(g.group_id == 0)[1])
    sp = np.zeros(g.B, np.int32)
    cu = np.zeros(g.B + 1, np.int32)
    cu[member + 1:] = 1
    with pytest.raises(kp.KvpError) as e:
        kp.kv_append(cg.pool, 0, kv[:, 0].contiguous(), kv[:, 1].contiguous(), cg.bt, sp, cu,
                     group_prefix=kp.group_prefix(g.group_id, g.shared_pages))
    assert e.value.code == kp.KVP_ESHARED


def test_binding_checks_tensors_before_launch(cases):
    """The C-ABI takes bare device pointers, so the binding checks what they are assumed to hold (dtype,
    rank, density, row counts) and raises before anything is enqueued."""
    import torch
    c = get_case(cases, "tiny")
    w = c.w
    q = to_dev_bits(c.vals.q)
    lens = w.decode_len
    sentinel = torch.full((w.B, w.Hq, w.d), 7.0, device="cuda")
    bad_calls = {
        "q with one sequence fewer": lambda: kp.paged_decode_attn(q[:-1].contiguous(), c.pool, 0, c.bt, lens,
                                                                 out=sentinel),
        "q in float32": lambda: kp.paged_decode_attn(q.float(), c.pool, 0, c.bt, lens, out=sentinel),
        "strided q": lambda: kp.paged_decode_attn(q.transpose(0, 1).contiguous().transpose(0, 1), c.pool, 0,
                                                  c.bt, lens, out=sentinel),
        "block tables of int64": lambda: kp.paged_decode_attn(q, c.pool, 0, c.bt.long(), lens, out=sentinel),
        "block tables missing a row": lambda: kp.paged_decode_attn(q, c.pool, 0, c.bt[:-1], lens, out=sentinel),
        "column slice of the block tables": lambda: kp.paged_decode_attn(q, c.pool, 0, c.bt[:, :-1], lens,
                                                                         out=sentinel),
        "out of the wrong shape": lambda: kp.paged_decode_attn(q, c.pool, 0, c.bt, lens, out=sentinel[:, :-1]),
        "out in float16": lambda: kp.paged_decode_attn(q, c.pool, 0, c.bt, lens, out=sentinel.half()),
        "host q": lambda: kp.paged_decode_attn(q.cpu(), c.pool, 0, c.bt, lens, out=sentinel),
        "q with another head_dim than the pool": lambda: kp.paged_decode_attn(
            torch.zeros((w.B, w.Hq, 2 * w.d), dtype=torch.bfloat16, device="cuda"), c.pool, 0, c.bt, lens,
            out=sentinel),
        "q heads not a multiple of the KV heads": lambda: kp.paged_decode_attn(
            torch.zeros((w.B, w.Hq + 1, w.d), dtype=torch.bfloat16, device="cuda"), c.pool, 0, c.bt, lens,
            out=sentinel),
    }
    for what, call in bad_calls.items():
        note(f"binding check: {what}")
        with pytest.raises(ValueError):
            call()
    kv = c.kv_dev
    sp = np.zeros(w.B, np.int32)
    cu = np.arange(w.B + 1, dtype=np.int32)
    k1, v1 = kv[: w.B - 1, 0].contiguous(), kv[: w.B - 1, 1].contiguous()
    note("binding check: kv_append with fewer token rows than cu_new")
    with pytest.raises(ValueError):
        kp.kv_append(c.pool, 0, k1, v1, c.bt, sp, cu)
    note("binding check: kv_append with a wrong head count")
    with pytest.raises(ValueError):
        kp.kv_append(c.pool, 0, kv[: w.B, 0, :1].contiguous(), kv[: w.B, 1, :1].contiguous(), c.bt, sp, cu)
    cq = np.array([0, 3], np.int32)
    qp = torch.zeros((4, w.Hq, w.d), dtype=torch.bfloat16, device="cuda")
    note("binding check: prefill q rows differ from cu_q")
    with pytest.raises(ValueError):
        kp.prefix_chunk_prefill_attn(qp, c.pool, 0, c.bt, np.array([0], np.int32), cq)
    sent_p = torch.full((3, w.Hq, w.d), 7.0, device="cuda")
    for what, qbad in {"another head_dim": torch.zeros((3, w.Hq, 2 * w.d), dtype=torch.bfloat16, device="cuda"),
                       "heads not a multiple of the KV heads": torch.zeros((3, w.Hq + 1, w.d), dtype=torch.bfloat16,
                                                                           device="cuda")}.items():
        note(f"binding check: prefill q with {what}")
        with pytest.raises(ValueError):
            kp.prefix_chunk_prefill_attn(qbad, c.pool, 0, c.bt, np.array([0], np.int32), cq, out=sent_p)
    torch.cuda.synchronize()
    assert torch.all(sentinel == 7.0) and torch.all(sent_p == 7.0)


def test_bad_page_id_is_skipped_and_reported():
    """An out-of-pool page id in a device block table is never dereferenced: the kernels skip the page and
    record KVP_ERANGE; outputs stay finite and equal attention over the remaining pages."""
    import torch
    w = W.make_workload("tiny")
    c = GpuCase(w)
    bt_bad = w.block_tables.copy()
    bt_bad[3, 5] = w.num_pages + 1000
    btd = torch.from_numpy(bt_bad).cuda()
    note("decode with a bad page id")
    out = kp.paged_decode_attn(to_dev_bits(c.vals.q), c.pool, 0, btd, w.decode_len, scale=w.scale)
    torch.cuda.synchronize()
    assert c.pool.device_error() == kp.KVP_ERANGE
    assert c.pool.device_error() == kp.KVP_OK  # read-and-clear
    o = out.cpu().numpy()
    assert np.all(np.isfinite(o))
    ref = c.oracle_decode()
    assert_close(out[:3], ref[:3], "unaffected sequences")
    # sequence 3 without page 5: attention over its other tokens
    pk, pv = c.oracle_pool()
    k, v = oracle.gather(pk, pv, w.block_tables[3], int(w.decode_len[3]))
    keep = np.ones(len(k), bool)
    keep[5 * 16:6 * 16] = False
    exp = oracle.decode_seq(c.vals.q[3], k[keep], v[keep], w.scale)
    assert_close(out[3:4], exp[None], "sequence with the skipped page")


def test_pool_reset_zeroes(cases):
    import torch
    w = W.make_workload("tiny")
    c = GpuCase(w)
    c.pool.reset()
    torch.cuda.synchronize()
    assert bool(torch.all(c.pool.layer_raw(0) == 0))


@pytest.mark.parametrize("G,members,d", [(8, 3, 128), (16, 2, 128), (4, 12, 64), (8, 12, 128), (1, 80, 64),
                                         (2, 5, 128), (16, 5, 64)])
def test_decode_group_shapes(G, members, d):
    """Shared-prefix groups of every tiling: 2 and 3 column tiles on the LDS path, subgroups (> 64
    columns, with a remainder small enough for the wave path), G = 1 and G = 16, odd member counts."""
    rng = np.random.default_rng(G * 100 + members + d)
    P = int(rng.integers(40, 300))           # prompt tokens; shared whole pages = P // 16
    priv = rng.integers(1, 500, size=members)
    _run_group_case(G, members, d, P, priv, rng, "group shapes")


@pytest.mark.parametrize("G,members,d", [(8, 8, 128), (4, 12, 64), (16, 3, 128), (2, 40, 128)])
def test_decode_wide_group_on_wave_path(G, members, d):
    """A wide group whose prompt is a small share of the call's pages is planned as 16-column wave items
    (the prompt pages read once per subgroup, the call launched wave-only): same results."""
    rng = np.random.default_rng(700 + G * 10 + members)
    P = int(rng.integers(32, 60))
    priv = rng.integers(3000, 4000, size=members)
    gp = kp.group_prefix(np.zeros(members, np.int32), np.array([P // 16], np.int32))
    items, _, _ = kp.kvp_plan_decode((P + priv).astype(np.int32), G * 2, 2, gp)
    assert np.all(items[:, 6] * G <= 16), "expected a wave-only plan"
    _run_group_case(G, members, d, P, priv, rng, "wide group on waves")


def _run_group_case(G, members, d, P, priv, rng, tag):
    import torch
    Hkv = 2
    Hq = G * Hkv
    S = P // 16
    lens = (P + priv).astype(np.int32)
    pages = [(int(n) + 15) // 16 for n in lens]
    num_pages = S + sum(p - S for p in pages) + 7
    perm = rng.permutation(num_pages).astype(np.int32)
    maxp = max(pages)
    bt = np.full((members, maxp), -1, np.int32)
    nxt = S
    for i in range(members):
        bt[i, :S] = perm[:S]
        k = pages[i] - S
        bt[i, S:S + k] = perm[nxt:nxt + k]
        nxt += k
    prompt = W.f32_to_bf16_bits(rng.standard_normal((P, 2, Hkv, d), dtype=np.float32))
    own = [W.f32_to_bf16_bits(rng.standard_normal((int(priv[i]), 2, Hkv, d), dtype=np.float32))
           for i in range(members)]
    qb = W.f32_to_bf16_bits(rng.standard_normal((members, Hq, d), dtype=np.float32))
    pool = kp.Pool(1, num_pages, Hkv, d)
    btd = torch.from_numpy(bt).cuda()
    note(f"{tag} G={G} members={members} d={d} P={P}")
    # the first member writes the shared prompt pages, then every member writes its tail + private tokens
    cnt0 = np.zeros(members, np.int64)
    cnt0[0] = S * 16
    kv0 = to_dev_bits(prompt[:S * 16])
    kp.kv_append(pool, 0, kv0[:, 0].contiguous(), kv0[:, 1].contiguous(), btd, np.zeros(members, np.int32),
                 np.concatenate([[0], np.cumsum(cnt0)]).astype(np.int32))
    rest = [np.concatenate([prompt[S * 16:], own[i]]) for i in range(members)]
    kv1 = to_dev_bits(np.concatenate(rest))
    cu1 = np.concatenate([[0], np.cumsum([len(r) for r in rest])]).astype(np.int32)
    gp = kp.group_prefix(np.zeros(members, np.int32), np.array([S], np.int32))
    kp.kv_append(pool, 0, kv1[:, 0].contiguous(), kv1[:, 1].contiguous(), btd, np.full(members, S * 16, np.int32),
                 cu1, group_prefix=gp)
    out = kp.paged_decode_attn(to_dev_bits(qb), pool, 0, btd, lens, group_prefix=gp, scale=0.11)
    out_ng = kp.paged_decode_attn(to_dev_bits(qb), pool, 0, btd, lens, scale=0.11)
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    ref = np.stack([oracle.decode_seq(qb[i], oracle.widen_bf16(np.concatenate([prompt, own[i]])[:, 0]),
                                      oracle.widen_bf16(np.concatenate([prompt, own[i]])[:, 1]), 0.11)
                    for i in range(members)])
    assert_close(out, ref, f"group G={G} x{members} d={d}")
    assert_close(out_ng, ref, f"ungrouped G={G} x{members} d={d}")


@pytest.mark.parametrize("seed", list(range(11, 51)))
def test_randomized_batches(seed):
    """Seeded random batches: groups of 1-12 members with prompts of 0-40 pages (sometimes under one
    page, so nothing is shared), ungrouped and empty sequences, private tails of 0-3000 tokens, every
    GQA ratio and both head dims; decode with and without the group hint, and chunked prefill of a few
    sequences over their own history, against the oracle."""
    import torch
    rng = np.random.default_rng(seed)
    G = int(rng.choice([1, 2, 4, 8, 16]))
    d = int(rng.choice([64, 128]))
    Hkv = int(rng.choice([1, 2, 4]))
    Hq = G * Hkv
    n_groups = int(rng.integers(1, 5))
    sizes = rng.integers(1, 13, size=n_groups)
    n_free = int(rng.integers(0, 5))
    B = int(sizes.sum()) + n_free
    group_id = np.concatenate([np.full(int(s), g, np.int32) for g, s in enumerate(sizes)] +
                              [np.full(n_free, -1, np.int32)])
    P = rng.integers(0, 641, size=n_groups)          # prompt tokens per group
    shared = (P // 16).astype(np.int32)
    priv = rng.integers(0, 3001, size=B)
    priv[rng.random(B) < 0.1] = 0                    # some members have no private tokens (or none at all)
    lens = np.array([(P[group_id[i]] if group_id[i] >= 0 else 0) + priv[i] for i in range(B)], np.int32)
    pages = [(int(n) + 15) // 16 for n in lens]
    num_pages = int(shared.sum()) + sum(pages) + 5
    perm = rng.permutation(num_pages).astype(np.int32)
    maxp = max(1, max(pages))
    bt = np.full((B, maxp), -1, np.int32)
    nxt = 0
    gpages = []
    for g in range(n_groups):
        gpages.append(perm[nxt:nxt + shared[g]])
        nxt += shared[g]
    toks = []
    prompts = [W.f32_to_bf16_bits(rng.standard_normal((int(P[g]), 2, Hkv, d), dtype=np.float32))
               for g in range(n_groups)]
    for i in range(B):
        g = group_id[i]
        S = int(shared[g]) if g >= 0 and lens[i] > 0 else 0
        bt[i, :S] = gpages[g][:S] if S else bt[i, :S]
        k = pages[i] - S
        bt[i, S:S + k] = perm[nxt:nxt + k]
        nxt += k
        own = W.f32_to_bf16_bits(rng.standard_normal((int(priv[i]), 2, Hkv, d), dtype=np.float32))
        full = np.concatenate([prompts[g], own]) if g >= 0 else own
        toks.append(full[:lens[i]])
    pool = kp.Pool(1, num_pages, Hkv, d)
    btd = torch.from_numpy(bt).cuda()
    note(f"randomized batch seed={seed} G={G} d={d} Hkv={Hkv} B={B} groups={n_groups}")
    # shared prompt pages are written once, by each group's first decoding member
    first = {}
    for i in range(B):
        g = group_id[i]
        if g >= 0 and lens[i] > 0 and g not in first:
            first[g] = i
    cnt0 = np.zeros(B, np.int64)
    src0 = []
    for g, i in first.items():
        cnt0[i] = shared[g] * 16
        src0.append(toks[i][:shared[g] * 16])
    gp = kp.group_prefix(group_id, shared)
    if cnt0.sum():
        order = sorted(first.values())
        kv0 = to_dev_bits(np.concatenate([toks[i][:cnt0[i]] for i in order]))
        kp.kv_append(pool, 0, kv0[:, 0].contiguous(), kv0[:, 1].contiguous(), btd, np.zeros(B, np.int32),
                     np.concatenate([[0], np.cumsum(cnt0)]).astype(np.int32))
    start = np.array([shared[group_id[i]] * 16 if group_id[i] >= 0 and lens[i] > 0 else 0 for i in range(B)],
                     np.int32)
    rest = [toks[i][start[i]:] for i in range(B)]
    cu = np.concatenate([[0], np.cumsum([len(r) for r in rest])]).astype(np.int32)
    if cu[-1]:
        kv1 = to_dev_bits(np.concatenate([r for r in rest if len(r)]))
        kp.kv_append(pool, 0, kv1[:, 0].contiguous(), kv1[:, 1].contiguous(), btd, start, cu, group_prefix=gp)
    qb = W.f32_to_bf16_bits(rng.standard_normal((B, Hq, d), dtype=np.float32))
    out = kp.paged_decode_attn(to_dev_bits(qb), pool, 0, btd, lens, group_prefix=gp, scale=0.1)
    out_ng = kp.paged_decode_attn(to_dev_bits(qb), pool, 0, btd, lens, scale=0.1)
    torch.cuda.synchronize()
    assert pool.device_error() == kp.KVP_OK
    ref = np.stack([oracle.decode_seq(qb[i], oracle.widen_bf16(toks[i][:, 0]), oracle.widen_bf16(toks[i][:, 1]), 0.1)
                    if lens[i] else np.zeros((Hq, d)) for i in range(B)])
    assert_close(out, ref, f"randomized decode seed={seed}")
    assert_close(out_ng, ref, f"randomized decode (no hint) seed={seed}")
    # chunked prefill: the last C tokens of a few sequences as the chunk over the rest as history
    sel = [i for i in range(B) if lens[i] >= 2][:3]
    if not sel:
        return
    C = [int(rng.integers(1, min(int(lens[i]), 300) + 1)) for i in sel]
    ctx = [int(lens[i]) - c for i, c in zip(sel, C)]
    cu_q = np.concatenate([[0], np.cumsum(C)]).astype(np.int32)
    qp = W.f32_to_bf16_bits(rng.standard_normal((int(cu_q[-1]), Hq, d), dtype=np.float32))
    btp = torch.from_numpy(np.ascontiguousarray(bt[sel])).cuda()
    outp = kp.prefix_chunk_prefill_attn(to_dev_bits(qp), pool, 0, btp, ctx, cu_q, scale=0.1)
    torch.cuda.synchronize()
    refp = np.concatenate([oracle.prefill_seq(qp[cu_q[j]:cu_q[j + 1]], oracle.widen_bf16(toks[i][:, 0]),
                                              oracle.widen_bf16(toks[i][:, 1]), 0.1, ctx[j])
                           for j, i in enumerate(sel)])
    assert_close(outp, refp, f"randomized prefill seed={seed}")
