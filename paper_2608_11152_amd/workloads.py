"""Seeded synthetic workloads for prefix-shared paged-KV attention over mixed RL rollout sessions.

This module only builds inputs: session lengths, rollout groups, page allocation through a permuted
pool, per-token query/key/value values and the order in which tokens are appended.  It contains none of
the attention arithmetic, so both the CPU oracle and the GPU path consume exactly the same inputs.

Workload structure follows the paper's serving model:
  * sessions hold KV in fixed-size blocks of a shared pool (Sec. 3.2, retained blocks k_s(t));
  * a prompt fans out into grouped samples that share the prompt prefix (Sec. 3.1, group id g_r);
  * prefix reuse is block-granular: a request reuses the leading whole prompt blocks whose hashes are
    cached (Sec. 4.4), so only whole prompt pages are shared and the partial last prompt page is copied into
    each sample's first private page;
  * a later agentic turn prefills only its new tokens over the cached history (Eq. 1, L_r - H_r);
  * the three classes have the length profiles of Tables 1-2 (RLVR: short prompt, long decode;
    RLHF: medium prompt and response; agentic: long cached history, short turn).

The paper's own trace is not available, so these seeded distributions stand in for it.

Value distribution: q, k, v ~ N(0, 1) drawn in fp32 and rounded to bf16 (round-to-nearest-even).
Small workloads draw them with numpy's PCG64 on the host; full-size workloads can draw them with
torch's generator on the device (``values="torch"``).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

PAGE = 16

# Lognormal spread used for the RLHF lengths: the 256 / 4096 clips of a median-1024 prompt sit at the
# 5th / 95th percentiles, i.e. sigma = ln 4 / z_0.95.
LOGNORMAL_SIGMA = math.log(4.0) / 1.6448536269514722


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round-to-nearest-even) and return the raw uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen raw bf16 bits to fp32 exactly."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass
class AppendBatch:
    """One kv_append call: sequence i appends tokens src[cu_new[i]:cu_new[i+1]] at start_pos[i]...

    ``src_rows`` indexes the workload's token-value table (row r = one token, all KV heads)."""
    start_pos: np.ndarray  # int32 [B]
    cu_new: np.ndarray  # int32 [B+1]
    src_rows: np.ndarray  # int64 [cu_new[-1]]
    use_group_prefix: bool  # whether the call passes the group-prefix hint (appends outside shared pages)


@dataclass
class Workload:
    name: str
    Hq: int
    Hkv: int
    d: int
    num_pages: int
    seq_kind: list  # per sequence: "rlvr" | "rlhf" | "agentic" | "plain"
    group_id: np.ndarray  # int32 [B], -1 = ungrouped
    shared_pages: np.ndarray  # int32 [num_groups]: whole prompt pages shared by the group
    prompt_len: np.ndarray  # int32 [num_groups]
    block_tables: np.ndarray  # int32 [B, maxp], -1 padding
    final_len: np.ndarray  # int32 [B]: tokens held by each sequence after the step's appends
    decode_len: np.ndarray  # int32 [B]: seq_lens passed to decode (0 = sequence does not decode)
    prefill_seqs: np.ndarray  # int32 [Bp]: sequences that prefill a chunk this step (contiguous rows)
    prefill_ctx: np.ndarray  # int32 [Bp]: cached tokens before the chunk
    prefill_chunk: np.ndarray  # int32 [Bp]: chunk length
    token_rows: list  # per sequence: int64 [final_len] rows of the value table in position order
    num_token_rows: int
    setup_appends: list = field(default_factory=list)  # AppendBatch list, done before timing
    step_appends: list = field(default_factory=list)  # AppendBatch list, part of each step
    decode_before_prefill_append: bool = False
    seed: int = 0

    @property
    def B(self) -> int:
        return len(self.seq_kind)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def maxp(self) -> int:
        return self.block_tables.shape[1]

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def num_groups(self) -> int:
        return len(self.shared_pages)

    def cu_q(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.prefill_chunk)]).astype(np.int32)

    def unique_decode_tokens(self) -> int:
        """Cached tokens that decode reads, counting each group's shared pages once."""
        tot = 0
        for i in range(self.B):
            n = int(self.decode_len[i])
            g = int(self.group_id[i])
            tot += n - (int(self.shared_pages[g]) * PAGE if g >= 0 and n > 0 else 0)
        for g in range(self.num_groups):
            if np.any((self.group_id == g) & (self.decode_len > 0)):
                tot += int(self.shared_pages[g]) * PAGE
        return tot

    def logical_decode_tokens(self) -> int:
        return int(self.decode_len.sum())

    def prefill_flops(self) -> float:
        """Algorithmic flops of the chunked prefill: 4*d*Hq per (query, visible key) pair."""
        pairs = 0
        for c, n in zip(self.prefill_ctx.tolist(), self.prefill_chunk.tolist()):
            pairs += n * c + n * (n + 1) // 2
        return 4.0 * self.d * self.Hq * pairs


# ----------------------------------------------------------------------------------------------
# session length draws
# ----------------------------------------------------------------------------------------------

def _lognormal_len(rng, n, median, lo, hi):
    x = np.exp(math.log(median) + LOGNORMAL_SIGMA * rng.standard_normal(n))
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


@dataclass
class _Spec:
    name: str
    Hq: int = 32
    Hkv: int = 4
    d: int = 128
    rlvr_groups: int = 0
    rlvr_samples: int = 8
    rlvr_prompt: tuple = (128, 1024)
    rlvr_private: tuple = (1024, 16384)
    rlhf_groups: int = 0
    rlhf_samples: int = 2
    rlhf_prompt: tuple = (1024, 256, 4096)  # median, lo, hi
    rlhf_response: tuple = (1024, 128, 4096)
    agentic: int = 0
    agentic_hist: tuple = (32768, 131072)
    agentic_prefill: int = 0  # how many agentic sessions prefill a chunk this step
    chunk: int = 2048
    agentic_decode_first: bool = True  # mixed step: decode token precedes the chunk
    agentic_decode: bool = True
    plain_lens: tuple = ()
    pool_pages: int = 0  # fixed pool size (0 = needed + 5%)
    pool_slack: float = 0.05


SPECS = {
    # 4 sequences, 8/2 heads, d=64, lengths {17,64,100,256}, no sharing, 64-page permuted pool.
    "tiny": _Spec("tiny", Hq=8, Hkv=2, d=64, plain_lens=(17, 64, 100, 256), pool_pages=64),
    # 64 prompt groups x 8 samples; prompt U[128,1024] shared; private decode U[1k,16k].
    "rlvr": _Spec("rlvr", rlvr_groups=64),
    # 128 groups x 2 samples; prompt and response lognormal (median 1k) clipped.
    "rlhf": _Spec("rlhf", rlhf_groups=128),
    # 32 sessions, history U[32k,128k]; 2048-token chunk prefill, then one decode step.
    "agentic": _Spec("agentic", agentic=32, agentic_prefill=32, agentic_decode_first=False),
    # 40 sessions (16 RLVR, 12 RLHF, 12 agentic); 1.5M-token pool; 8 agentic sessions prefill.
    "mixed": _Spec("mixed", rlvr_groups=2, rlhf_groups=6, agentic=12, agentic_prefill=8,
                   pool_pages=1_500_000 // PAGE),
    # Reduced-size variants: same structure, sizes the CPU oracle finishes in seconds.
    "rlvr_s": _Spec("rlvr_s", rlvr_groups=4, rlvr_private=(40, 1500)),
    "rlhf_s": _Spec("rlhf_s", rlhf_groups=8, rlhf_prompt=(300, 40, 1200), rlhf_response=(300, 1, 1200)),
    "agentic_s": _Spec("agentic_s", agentic=3, agentic_hist=(600, 3000), agentic_prefill=3, chunk=300,
                       agentic_decode_first=False),
    "mixed_s": _Spec("mixed_s", rlvr_groups=1, rlvr_private=(30, 900), rlhf_groups=2,
                     rlhf_prompt=(200, 20, 600), rlhf_response=(200, 1, 600), agentic=3,
                     agentic_hist=(500, 2500), agentic_prefill=2, chunk=200),
    # GQA 8/2 with d=64 and sharing, to cover the second head size on the grouped path.
    "rlvr_d64": _Spec("rlvr_d64", Hq=8, Hkv=2, d=64, rlvr_groups=3, rlvr_samples=4,
                      rlvr_prompt=(16, 200), rlvr_private=(1, 700)),
}

CONFIG_SEEDS = {"tiny": 1001, "rlvr": 1002, "rlhf": 1003, "agentic": 1004, "mixed": 1005}


def make_workload(name: str, seed: int | None = None, **overrides) -> Workload:
    """Build the structure (lengths, groups, block tables, append schedule) of a named workload."""
    spec = SPECS[name]
    if overrides:
        spec = _Spec(**{**spec.__dict__, **overrides})
    if seed is None:
        seed = CONFIG_SEEDS.get(name, 2000 + sorted(SPECS).index(name))
    rng = np.random.default_rng(seed)

    kinds, gid, final_len, decode_len = [], [], [], []
    prompt_len, shared = [], []
    own_len = []  # tokens each sequence holds beyond its group's prompt
    seq_hist, seq_chunk, seq_decode_first = [], [], []

    # --- grouped classes: RLVR then RLHF -------------------------------------------------------
    if spec.rlvr_groups:
        P = rng.integers(spec.rlvr_prompt[0], spec.rlvr_prompt[1], size=spec.rlvr_groups, endpoint=True)
        D = rng.integers(spec.rlvr_private[0], spec.rlvr_private[1],
                         size=spec.rlvr_groups * spec.rlvr_samples, endpoint=True)
        for g in range(spec.rlvr_groups):
            gi = len(prompt_len)
            prompt_len.append(int(P[g]))
            shared.append(int(P[g]) // PAGE)
            for s in range(spec.rlvr_samples):
                kinds.append("rlvr"); gid.append(gi)
                own_len.append(int(D[g * spec.rlvr_samples + s]))
    if spec.rlhf_groups:
        P = _lognormal_len(rng, spec.rlhf_groups, *spec.rlhf_prompt)
        R = _lognormal_len(rng, spec.rlhf_groups * spec.rlhf_samples, *spec.rlhf_response)
        for g in range(spec.rlhf_groups):
            gi = len(prompt_len)
            prompt_len.append(int(P[g]))
            shared.append(int(P[g]) // PAGE)
            for s in range(spec.rlhf_samples):
                kinds.append("rlhf"); gid.append(gi)
                own_len.append(int(R[g * spec.rlhf_samples + s]))
    for i in range(len(kinds)):
        n = prompt_len[gid[i]] + own_len[i]
        final_len.append(n); decode_len.append(n)
        seq_hist.append(n - 1); seq_chunk.append(0); seq_decode_first.append(True)

    # --- agentic sessions ----------------------------------------------------------------------
    if spec.agentic:
        H = rng.integers(spec.agentic_hist[0], spec.agentic_hist[1], size=spec.agentic, endpoint=True)
        for a in range(spec.agentic):
            h = int(H[a])
            c = spec.chunk if a < spec.agentic_prefill else 0
            kinds.append("agentic"); gid.append(-1); own_len.append(0)
            final_len.append(h + c + (1 if spec.agentic_decode else 0))
            if spec.agentic_decode:
                decode_len.append(h + 1 if (spec.agentic_decode_first or c == 0) else h + c + 1)
            else:
                decode_len.append(0)
            seq_hist.append(h); seq_chunk.append(c); seq_decode_first.append(spec.agentic_decode_first)
    # --- plain ungrouped decode sequences ------------------------------------------------------
    for n in spec.plain_lens:
        kinds.append("plain"); gid.append(-1); own_len.append(0)
        final_len.append(int(n)); decode_len.append(int(n))
        seq_hist.append(int(n) - 1); seq_chunk.append(0); seq_decode_first.append(True)

    B = len(kinds)
    gid = np.asarray(gid, dtype=np.int32)
    shared = np.asarray(shared, dtype=np.int32)
    prompt_len = np.asarray(prompt_len, dtype=np.int32)
    final_len = np.asarray(final_len, dtype=np.int64)

    # --- pages: shared prompt pages first, then each sequence's private pages in order ------------
    pages_per_seq = (final_len + PAGE - 1) // PAGE
    need = int(shared.sum()) + int(sum(int(pages_per_seq[i]) - (int(shared[gid[i]]) if gid[i] >= 0 else 0)
                                       for i in range(B)))
    num_pages = spec.pool_pages or int(math.ceil(need * (1.0 + spec.pool_slack)))
    if need > num_pages:
        raise ValueError(f"{name}: workload needs {need} pages, pool holds {num_pages}")
    perm = rng.permutation(num_pages).astype(np.int32)
    nxt = 0
    group_pages = []
    for g in range(len(shared)):
        group_pages.append(perm[nxt:nxt + shared[g]]); nxt += int(shared[g])
    maxp = int(pages_per_seq.max())
    bt = np.full((B, maxp), -1, dtype=np.int32)
    for i in range(B):
        s = int(shared[gid[i]]) if gid[i] >= 0 else 0
        if s:
            bt[i, :s] = group_pages[gid[i]]
        k = int(pages_per_seq[i]) - s
        bt[i, s:s + k] = perm[nxt:nxt + k]; nxt += k

    # --- token value rows: group prompts first, then each sequence's own tokens ------------------
    prompt_base = np.concatenate([[0], np.cumsum(prompt_len)]).astype(np.int64)
    row = int(prompt_base[-1])
    token_rows = []
    for i in range(B):
        if gid[i] >= 0:
            P = int(prompt_len[gid[i]])
            own = int(final_len[i]) - P
            rows = np.concatenate([prompt_base[gid[i]] + np.arange(P), row + np.arange(own)])
            row += own
        else:
            rows = row + np.arange(int(final_len[i])); row += int(final_len[i])
        token_rows.append(rows.astype(np.int64))
    num_rows = row

    # --- append schedule -------------------------------------------------------------------------
    rep = {}
    for i in range(B):
        if gid[i] >= 0 and gid[i] not in rep:
            rep[int(gid[i])] = i
    setup = []
    # (1) each group's representative writes the shared prompt pages (no group hint: pages being filled)
    if rep:
        start = np.zeros(B, np.int32); cnt = np.zeros(B, np.int64); rows = []
        for g, i in sorted(rep.items(), key=lambda t: t[1]):
            cnt[i] = int(shared[g]) * PAGE
        for i in range(B):
            rows.append(token_rows[i][:cnt[i]])
        setup.append(AppendBatch(start, _cu(cnt), np.concatenate(rows), False))
    # (2) every sequence writes its private history (prompt tail copy + own tokens) up to the step
    start = np.zeros(B, np.int32); cnt = np.zeros(B, np.int64); rows = []
    hist = np.asarray(seq_hist, dtype=np.int64)
    for i in range(B):
        s0 = int(shared[gid[i]]) * PAGE if gid[i] >= 0 else 0
        start[i] = s0; cnt[i] = max(0, int(hist[i]) - s0)
        rows.append(token_rows[i][s0:s0 + cnt[i]])
    setup.append(AppendBatch(start, _cu(cnt), np.concatenate(rows), True))

    # step appends: every sequence's step tokens (prefill chunk and/or decode token) form one run
    # [hist, final_len), appended before either attention of the step reads them.
    chunk = np.asarray(seq_chunk, dtype=np.int64)
    dfirst = np.asarray(seq_decode_first, dtype=bool)
    dec = np.asarray(decode_len, dtype=np.int64) > 0
    start = hist.astype(np.int32)
    cnt = final_len - hist
    rows = [token_rows[i][int(hist[i]):int(final_len[i])] for i in range(B)]
    step = [AppendBatch(start, _cu(cnt), np.concatenate(rows), True)] if cnt.sum() else []

    pre = [i for i in range(B) if chunk[i] > 0]
    if pre and pre != list(range(pre[0], pre[0] + len(pre))):
        raise AssertionError("prefill sessions must occupy contiguous rows")
    pctx = np.asarray([int(hist[i]) + (1 if (dfirst[i] and dec[i]) else 0) for i in pre], dtype=np.int32)

    return Workload(
        name=name, Hq=spec.Hq, Hkv=spec.Hkv, d=spec.d, num_pages=num_pages, seq_kind=kinds,
        group_id=gid, shared_pages=shared, prompt_len=prompt_len, block_tables=bt,
        final_len=final_len.astype(np.int32), decode_len=np.asarray(decode_len, dtype=np.int32),
        prefill_seqs=np.asarray(pre, dtype=np.int32), prefill_ctx=pctx,
        prefill_chunk=np.asarray([int(chunk[i]) for i in pre], dtype=np.int32),
        token_rows=token_rows, num_token_rows=num_rows, setup_appends=setup, step_appends=step,
        decode_before_prefill_append=bool(spec.agentic_decode_first), seed=seed)


def _cu(cnt: np.ndarray) -> np.ndarray:
    return np.concatenate([[0], np.cumsum(cnt)]).astype(np.int32)


# ----------------------------------------------------------------------------------------------
# values
# ----------------------------------------------------------------------------------------------

@dataclass
class Values:
    """bf16 values as raw uint16 bits (numpy) or bf16 tensors (torch).

    kv:   [num_token_rows, 2, Hkv, d]  (index 0 = K, 1 = V) per token row
    q:    [B, Hq, d]                   decode queries
    qp:   [sum(prefill_chunk), Hq, d]  prefill queries (chunk rows in session order)
    """
    kv: object
    q: object
    qp: object


def make_values(w: Workload, values: str = "numpy", device=None) -> Values:
    """Draw q/k/v ~ N(0,1) rounded to bf16 from the workload's seed."""
    nq = int(w.prefill_chunk.sum())
    if values == "numpy":
        rng = np.random.default_rng(w.seed + 7919)
        q = f32_to_bf16_bits(rng.standard_normal((w.B, w.Hq, w.d), dtype=np.float32))
        qp = f32_to_bf16_bits(rng.standard_normal((nq, w.Hq, w.d), dtype=np.float32))
        kv = f32_to_bf16_bits(rng.standard_normal((w.num_token_rows, 2, w.Hkv, w.d), dtype=np.float32))
        return Values(kv=kv, q=q, qp=qp)
    if values == "torch":
        import torch
        g = torch.Generator(device=device)
        g.manual_seed(w.seed + 7919)

        def draw(shape):
            out = torch.empty(shape, dtype=torch.bfloat16, device=device)
            flat = out.view(-1)
            step = 1 << 26
            for s in range(0, flat.numel(), step):
                e = min(flat.numel(), s + step)
                flat[s:e] = torch.randn(e - s, generator=g, device=device, dtype=torch.float32)
            return out

        q = draw((w.B, w.Hq, w.d))
        qp = draw((nq, w.Hq, w.d))
        kv = draw((w.num_token_rows, 2, w.Hkv, w.d))
        return Values(kv=kv, q=q, qp=qp)
    raise ValueError(values)


def make_tokens(w: Workload, vocab: int = 151936, lens=None):
    """Synthetic token ids for every sequence, in position order, drawn per value-table row, so group
    members carry identical prompt tokens and every other token is independent.  Returns (tokens int32
    [sum(lens)], cu_tokens int32 [B + 1]) for the first lens[i] tokens of sequence i (default: all)."""
    rng = np.random.default_rng(w.seed + 104729)
    ids = rng.integers(0, vocab, size=w.num_token_rows, dtype=np.int64).astype(np.int32)
    lens = w.final_len if lens is None else np.asarray(lens)
    parts = [ids[w.token_rows[i][: int(lens[i])]] for i in range(w.B)]
    cu = np.concatenate([[0], np.cumsum([len(x) for x in parts])]).astype(np.int32)
    tokens = np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)
    return tokens, cu


def step_start(w: Workload) -> np.ndarray:
    """Tokens each sequence holds before the step's appends (its cached history)."""
    start = np.asarray(w.final_len, dtype=np.int64).copy()
    for ab in w.step_appends:
        for i in range(len(ab.start_pos)):
            if ab.cu_new[i + 1] > ab.cu_new[i]:
                start[i] = min(start[i], int(ab.start_pos[i]))
    return start


def seq_kv_bits(w: Workload, vals: Values, i: int, n: int | None = None):
    """Logical (K, V) of sequence i in position order, as raw bf16 bits [n, Hkv, d] (host numpy)."""
    rows = w.token_rows[i][: (w.final_len[i] if n is None else n)]
    kv = vals.kv
    if isinstance(kv, np.ndarray):
        sel = kv[rows]
    else:
        import torch
        sel = kv[torch.as_tensor(rows, device=kv.device)].view(torch.int16).cpu().numpy().view(np.uint16)
    return sel[:, 0], sel[:, 1]


def to_numpy_bits(t) -> np.ndarray:
    """bf16 torch tensor or uint16 array -> uint16 numpy bits (host)."""
    if isinstance(t, np.ndarray):
        return t
    import torch
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)
