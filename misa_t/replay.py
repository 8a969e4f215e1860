"""Step-by-step replay of mixed rollout serving on one inference instance under an admission policy.

A synthetic trainer releases rollout units toward a target class mixture rho (Sec. 3.1): RLVR prompts that
fan out into 8 grouped samples, RLHF prompts into 2, and multi-turn agentic sessions whose turns are
separated by tool intervals.  Each step the controller (misa_t.controller) snapshots the instance, updates
its caps from the demand ledger and admits held requests (Admit, Sec. 4.1); admitted work then runs on
the paged KV pool through the library's calls:

  * kv_append of every new token (prompts, turn chunks, decode tokens);
  * prefix_chunk_prefill_attn for prompts and agentic turns over their cached history (Eq. 1: only the
    L - H uncached tokens are prefilled; an evicted history is prefilled again from scratch);
  * paged_decode_attn for every decoding session, with the rollout groups' shared prompt pages as the
    group-prefix hint.

Pages come from a free list over the pool.  A group's whole prompt pages are allocated once and shared by
its samples (Sec. 4.4 block-granular reuse); an agentic session keeps its pages through tool intervals
(its residency, Sec. 4.3) unless the pool runs short, when idle histories are evicted oldest first.

Lengths follow the class profiles of the synthetic workloads (Tables 1-2 stand-ins), scaled by
`length_scale` so a replay of a few hundred steps completes many units.  `engine=None` replays the
control logic alone and checks every batch's block tables with the library's host validator; with an
`Engine` the calls run on the GPU.
"""
from __future__ import annotations

import math
from collections import OrderedDict, deque
from dataclasses import dataclass, field

import numpy as np

from .controller import CLASSES, ClassEstimator, Controller

PAGE = 16
GROUP = {"rlvr": 8, "rlhf": 2, "agentic": 1}


@dataclass
class ReplayConfig:
    steps: int = 400
    pool_pages: int = 6144
    protected_frac: float = 0.9
    mixture: dict = field(default_factory=lambda: {"rlvr": 0.4, "rlhf": 0.3, "agentic": 0.3})
    max_outstanding: int = 64        # trainer's concurrency limit, in rollout units
    tokens_per_step: int = 16        # decode tokens a session produces per engine step
    length_scale: float = 1.0 / 16
    agentic_turns: tuple = (2, 4)
    tool_steps: tuple = (3, 12)
    Hq: int = 32
    Hkv: int = 4
    d: int = 128
    seed: int = 0


@dataclass
class Session:
    sid: int
    cls: str
    unit: int
    group: int                 # prompt group (rlvr / rlhf), -1 for agentic
    prompt: int                # tokens of the prompt (shared within the group)
    decode: int                # decode tokens of this sample (per turn for agentic)
    turns: int = 1
    turn: int = 0
    chunk: int = 0             # agentic: new tokens of each later turn
    state: str = "held"        # held -> prefill -> decode -> (tool -> prefill ...) -> done
    pages: list = field(default_factory=list)
    logical: int = 0           # tokens of the trajectory so far
    length: int = 0            # of them, tokens whose KV is in the pool (0 after an eviction)
    todo: int = 0              # decode tokens left in this turn
    tool_left: int = 0
    admitted_at: int = -1
    peak_pages: int = 0


def _lognormal(rng, median, lo, hi):
    sigma = math.log(4.0) / 1.6448536269514722
    return int(np.clip(round(math.exp(math.log(median) + sigma * rng.standard_normal())), lo, hi))


class Replay:
    def __init__(self, cfg: ReplayConfig, policy: str = "time", engine=None):
        self.cfg = cfg
        self.rng = np.random.default_rng(cfg.seed)
        self.engine = engine
        s = cfg.length_scale
        kbar_prior = {"rlvr": max(1, int(9000 * s / PAGE)), "rlhf": max(1, int(2500 * s / PAGE)),
                      "agentic": max(1, int(90000 * s / PAGE))}
        self.est = ClassEstimator(kbar_prior, T_prior=50.0)
        self.C = int(cfg.protected_frac * cfg.pool_pages)
        self.ctl = Controller(self.C, self.est, policy)
        self.free = deque(int(p) for p in self.rng.permutation(cfg.pool_pages))
        self.page_refs = np.zeros(cfg.pool_pages, np.int32)
        self.sessions: dict[int, Session] = {}
        self.held: "OrderedDict[int, Session]" = OrderedDict()
        self.group_pages: dict[int, list] = {}      # group -> its shared whole prompt pages
        self.group_written: set = set()             # groups whose shared pages hold the prompt
        self.group_members: dict[int, set] = {}
        self.idle_lru: "OrderedDict[int, None]" = OrderedDict()  # agentic sessions in a tool interval
        self.released = {b: 0 for b in CLASSES}
        self.completed = {b: 0 for b in CLASSES}
        self.unit_left: dict[int, int] = {}
        self.unit_cls: dict[int, str] = {}
        self.next_sid = self.next_unit = self.next_group = 0
        self.finished_since_snapshot = []
        self.hit_tokens = self.prefill_tokens = 0
        self.step_idx = 0
        self.history = []

    # ------------------------------------------------------------------ trainer
    def _release(self):
        cfg, rng, s = self.cfg, self.rng, self.cfg.length_scale
        outstanding = sum(self.unit_left.values())
        while outstanding < cfg.max_outstanding:
            tot = sum(self.released.values()) + 1
            b = max(CLASSES, key=lambda c: cfg.mixture[c] * tot - self.released[c])
            unit_group = self.next_group
            self.next_group += 1
            if b == "rlvr":
                prompt = max(1, int(rng.integers(128, 1025) * s))
            elif b == "rlhf":
                prompt = max(1, int(_lognormal(rng, 1024, 256, 4096) * s))
            else:
                prompt = max(1, int(rng.integers(32768, 131073) * s))
            for _ in range(GROUP[b]):
                u = self.next_unit
                self.next_unit += 1
                self.unit_left[u], self.unit_cls[u] = 1, b
                if b == "rlvr":
                    dec = max(1, int(rng.integers(1024, 16385) * s))
                    sess = Session(self.next_sid, b, u, unit_group, prompt, dec)
                elif b == "rlhf":
                    dec = max(1, int(_lognormal(rng, 1024, 128, 4096) * s))
                    sess = Session(self.next_sid, b, u, unit_group, prompt, dec)
                else:
                    sess = Session(self.next_sid, b, u, -1, prompt, max(1, int(256 * s)),
                                   turns=int(rng.integers(cfg.agentic_turns[0], cfg.agentic_turns[1] + 1)),
                                   chunk=max(1, int(2048 * s)))
                self.next_sid += 1
                self.sessions[sess.sid] = sess
                self.held[sess.sid] = sess
                if sess.group >= 0:
                    self.group_members.setdefault(sess.group, set()).add(sess.sid)
                self.released[b] += 1
            outstanding += GROUP[b]

    # ------------------------------------------------------------------ pages
    def _alloc(self, n: int):
        if len(self.free) < n:
            self._evict(n - len(self.free))
        if len(self.free) < n:
            return None
        out = [self.free.popleft() for _ in range(n)]
        for p in out:
            self.page_refs[p] += 1
        return out

    def _release_pages(self, pages):
        for p in pages:
            self.page_refs[p] -= 1
            assert self.page_refs[p] >= 0
            if self.page_refs[p] == 0:
                self.free.append(p)

    def _evict(self, need: int):
        """Drop idle agentic histories (oldest tool interval first) until `need` pages are free."""
        while need > 0 and self.idle_lru:
            sid, _ = self.idle_lru.popitem(last=False)
            s = self.sessions[sid]
            freed = len(s.pages)
            self._release_pages(s.pages)
            s.pages, s.length = [], 0
            self.ctl.O.pop(sid, None)  # its cache is gone: the next turn must be admitted again
            need -= freed

    def _grow(self, s: Session, new_len: int) -> bool:
        need = (new_len + PAGE - 1) // PAGE - len(s.pages)
        if need > 0:
            got = self._alloc(need)
            if got is None:
                return False
            s.pages += got
        s.peak_pages = max(s.peak_pages, len(s.pages))
        return True

    # ------------------------------------------------------------------ admission
    def _demand(self):
        n = {b: 0 for b in CLASSES}
        for s in self.sessions.values():
            if s.state != "done":
                n[s.cls] += 1
        return n

    def _admit(self):
        for sid in list(self.held):
            s = self.held[sid]
            if not self.ctl.admit(sid, s.cls):
                continue
            ok = self._place(s)
            if not ok:  # the pool cannot hold it now: undo the admission, keep holding
                self.ctl.P.pop(sid, None)
                continue
            del self.held[sid]
            s.admitted_at = self.step_idx if s.admitted_at < 0 else s.admitted_at
            s.state = "prefill"

    def _prefill_span(self, s: Session):
        """(H, L) of the session's next prefill: L tokens after it, H of them already in the pool."""
        if s.cls == "agentic":
            L = s.prompt if s.turn == 0 else s.logical + s.chunk
            return s.length, L
        whole = (s.prompt // PAGE) * PAGE
        return (whole if s.group in self.group_written else 0), s.prompt

    def _place(self, s: Session) -> bool:
        """Reserve the pages of the request's prefill: a group's shared prompt pages once per group."""
        if s.cls == "agentic":
            return self._grow(s, self._prefill_span(s)[1])
        whole = s.prompt // PAGE
        shared = self.group_pages.get(s.group)
        if shared is None and whole:
            shared = self._alloc(whole)
            if shared is None:
                return False
            self.group_pages[s.group] = shared
        if whole:
            s.pages = list(shared)
            for p in shared:
                self.page_refs[p] += 1
        if not self._grow(s, s.prompt):
            self._release_pages(s.pages)
            s.pages = []
            return False
        return True

    # ------------------------------------------------------------------ one engine step
    def step(self):
        cfg = self.cfg
        self._release()
        self.ctl.snapshot(self.finished_since_snapshot)
        self.finished_since_snapshot = []
        hit = self.hit_tokens / max(1, self.hit_tokens + self.prefill_tokens) if self.step_idx else None
        self.ctl.update_caps(self._demand(), hit)
        self._admit()

        # prefill: prompts (a group's shared whole pages are written by the first member to prefill) and
        # agentic turns over their cached history (all of it again after an eviction)
        prefill_batch = []
        for s in [x for x in self.sessions.values() if x.state == "prefill"]:
            H, L = self._prefill_span(s)
            if s.group >= 0:
                self.group_written.add(s.group)
            self.hit_tokens += H
            self.prefill_tokens += L - H
            prefill_batch.append((s, H, L))
        if prefill_batch:
            self._check_tables([s for s, _, _ in prefill_batch], [L for _, _, L in prefill_batch])
            if self.engine is not None:
                self.engine.prefill(self, prefill_batch)
        for s, H, L in prefill_batch:
            s.length = s.logical = L
            s.todo = s.decode
            s.state = "decode"

        # decode: every decoding session adds up to tokens_per_step tokens, then one attention call
        dec = []
        for s in self.sessions.values():
            if s.state != "decode":
                continue
            n = min(cfg.tokens_per_step, s.todo)
            if not self._grow(s, s.length + n):
                continue  # no page for its growth this step: it waits
            dec.append((s, s.length, n))
        if dec:
            lens = [a + n for _, a, n in dec]
            self._check_tables([s for s, _, _ in dec], lens)
            if self.engine is not None:
                self.engine.decode(self, dec)
            for s, a, n in dec:
                s.length = s.logical = a + n
                s.todo -= n
                if s.todo == 0:
                    self._turn_done(s)

        for sid in list(self.idle_lru):
            s = self.sessions[sid]
            s.tool_left -= 1
            if s.tool_left <= 0:
                del self.idle_lru[sid]
                s.turn += 1
                # a continuation whose session is still protected is admitted at once; after an eviction it
                # must acquire admission again (and will prefill its whole history)
                if s.length > 0 and (sid in self.ctl.O or sid in self.ctl.P) and self._grow(s, s.logical + s.chunk):
                    s.state = "prefill"
                else:
                    s.state = "held"
                    self.held[sid] = s
        self.history.append(self.metrics())
        self.step_idx += 1

    def _turn_done(self, s: Session):
        if s.cls == "agentic" and s.turn + 1 < s.turns:
            s.state = "tool"
            s.tool_left = int(self.rng.integers(self.cfg.tool_steps[0], self.cfg.tool_steps[1] + 1))
            self.idle_lru[s.sid] = None
            return
        s.state = "done"
        self.est.observe(s.cls, s.peak_pages, self.step_idx - s.admitted_at + 1)
        self._release_pages(s.pages)
        s.pages = []
        if s.group >= 0:
            self.group_members[s.group].discard(s.sid)
            if not self.group_members[s.group]:
                self.group_written.discard(s.group)
                if s.group in self.group_pages:
                    self._release_pages(self.group_pages.pop(s.group))
        self.finished_since_snapshot.append(s.sid)
        self.unit_left[s.unit] -= 1
        if self.unit_left[s.unit] == 0:
            del self.unit_left[s.unit]
            self.completed[s.cls] += 1

    # ------------------------------------------------------------------ checks and metrics
    def table_rows(self, sessions, lens):
        maxp = max(1, max((n + PAGE - 1) // PAGE for n in lens))
        bt = np.full((len(sessions), maxp), -1, np.int32)
        for i, s in enumerate(sessions):
            bt[i, :len(s.pages)] = s.pages[:maxp]
        return bt

    def group_hint(self, sessions):
        """Groups of the batch whose members all share the group's whole prompt pages."""
        gid = np.full(len(sessions), -1, np.int32)
        shared, index = [], {}
        for i, s in enumerate(sessions):
            if s.group >= 0 and s.group in self.group_pages and self.group_pages[s.group]:
                if s.group not in index:
                    index[s.group] = len(shared)
                    shared.append(len(self.group_pages[s.group]))
                gid[i] = index[s.group]
        return gid, np.asarray(shared, np.int32)

    def _check_tables(self, sessions, lens):
        if not sessions:
            return
        from paper_2608_11152_amd import kvpattn as kp  # host-only validator of the library
        bt = self.table_rows(sessions, lens)
        gid, shared = self.group_hint(sessions)
        gp = kp.group_prefix(gid, shared) if len(shared) else None
        rc = kp.kvp_check_tables(bt, np.asarray(lens, np.int32), self.cfg.pool_pages, gp)
        assert rc == kp.KVP_OK, f"step {self.step_idx}: block tables rejected ({kp.kvp_strerror(rc)})"

    def metrics(self):
        done = sum(self.completed.values())
        p = np.array([self.completed[b] / done if done else 0.0 for b in CLASSES])
        q = np.array([self.cfg.mixture[b] for b in CLASSES])
        protected = sum(len(self.sessions[s].pages) for s in list(self.ctl.O) + list(self.ctl.P))
        return {"step": self.step_idx, "completed": dict(self.completed), "throughput": done / (self.step_idx + 1),
                "tv_distance": 0.5 * float(np.abs(p - q).sum()) if done else None,
                "hit_rate": self.hit_tokens / max(1, self.hit_tokens + self.prefill_tokens),
                "protected_pages": protected, "free_pages": len(self.free), "cap": self.ctl.K,
                "class_caps": dict(self.ctl.class_caps), "held": len(self.held)}

    def run(self, steps: int | None = None):
        for _ in range(steps or self.cfg.steps):
            self.step()
        return self.history[-1]
