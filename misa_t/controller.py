"""MISA-T's admission controller for one inference instance w, restated from Sec. 3-4 of the paper.

Quantities (the paper's notation; blocks are 16-token KV pages):
  C_w          protected KV budget of the instance, in blocks                       (Sec. 3.2, Eq. 3)
  O_w, P_w     active protected sessions, and pending ones admitted since the last snapshot  (Sec. 4.1)
  K_w(t)       operational global session cap, at most K^base = floor(C_w / kbar_w)         (Sec. 4.1)
  N_{w,b}      distinct unfinished session demands of class b visible at evaluation: active, pending,
               held and candidate sessions count one each                                   (Sec. 4.2)
  kbar_b       conservative reference footprint (blocks) of a class-b session
  That_b       recent estimate of how long a class-b session's KV stays resident             (Sec. 4.3)

Equations:
  prefill cost        c = d + (L - H) / mu                                         (Eq. prefill-cost)
  hold rule           hold for the cached instance iff Delta + q_hit - q_cold < H / F     (Eq. hold-condition)
  spatial demand      S_b = N_b kbar_b                                             (Eq. spatial-demand)
  MISA caps           M_b = C S_b / sum S,   K_b = max{1, floor(M_b / kbar_b)}     (Eq. workloadcap)
  block-time demand   R_b = N_b kbar_b That_b                                      (Eq. block-time-demand)
  drain time          tau_b = N_b kbar_b That_b / M_b                              (Eq. backlog-drain-time)
  MISA-T caps         M_b = C R_b / sum R,   K_b = max{1, floor(M_b / kbar_b)}     (Eq. residency-quota)
  hit degradation     G_w = max{0, h* - h}                                          (Sec. 4.1)
  Admit(r, w) = 1 if s_r in O_w or P_w;  1 if |O_w| + |P_w| < K_w(t) (and, with class caps, the class's
  sessions in O_w and P_w are fewer than K_b);  0 otherwise                          (Sec. 4.1, 4.2)

Readings where the paper gives no formula (each listed in the design notes):
  * kbar_b: the larger of a class prior and the 90th percentile of the last `window` completed sessions'
    peak blocks; kbar_w (the global reference): the demand-weighted mean of the kbar_b, sum_b N_b kbar_b /
    sum_b N_b, i.e. the expected footprint of a session of the current mix (the mean of the class priors
    when nothing is pending);
  * That_b: the mean of the last `window` completed durations of the class, shrunk toward one neutral
    prior shared by all classes with `prior_weight` pseudo-observations;
  * when no class has demand (sum S = 0 or sum R = 0) every quota M_b is 0, so every class cap is 1;
  * overload pressure: G_w above `g_threshold` for `confirm` consecutive evaluations contracts K_w by
    `contract` (at least 1); otherwise K_w recovers by one session per evaluation up to K^base; h* is the
    best hit rate of the last `window` evaluations in which no pressure was applied.
"""
from __future__ import annotations

import math
from collections import deque

CLASSES = ("rlvr", "rlhf", "agentic")


def prefill_cost(d: float, L: float, H: float, mu: float) -> float:
    """Estimated prefill cost on an instance: backlog delay plus uncached tokens over prefill throughput."""
    return d + (L - H) / mu


def hold_preferable(delta: float, q_hit: float, q_cold: float, H: float, F: float) -> bool:
    """Holding for the cached instance beats routing cold when the extra wait is less than the prefill
    time of the reusable prefix."""
    return delta + q_hit - q_cold < H / F


def base_cap(C: float, kbar: float) -> int:
    """K^base = floor(C / kbar): how many reference-size sessions the protected budget holds."""
    return int(math.floor(C / kbar))


def hit_degradation(h_ref: float, h_obs: float) -> float:
    """G_w = max{0, h* - h}."""
    return max(0.0, h_ref - h_obs)


def spatial_demand(N: dict, kbar: dict) -> dict:
    return {b: N[b] * kbar[b] for b in N}


def _caps(C: float, demand: dict, kbar: dict):
    tot = sum(demand.values())
    M = {b: (C * demand[b] / tot if tot > 0 else 0.0) for b in demand}
    K = {b: max(1, int(math.floor(M[b] / kbar[b]))) for b in demand}
    return M, K


def space_caps(C: float, N: dict, kbar: dict):
    """MISA: block quota proportional to spatial demand, converted back to a session cap."""
    return _caps(C, spatial_demand(N, kbar), kbar)


def block_time_demand(N: dict, kbar: dict, That: dict) -> dict:
    return {b: N[b] * kbar[b] * That[b] for b in N}


def time_caps(C: float, N: dict, kbar: dict, That: dict):
    """MISA-T: block quota proportional to block-time demand, converted back to a session cap."""
    return _caps(C, block_time_demand(N, kbar, That), kbar)


def drain_times(N: dict, kbar: dict, That: dict, M: dict) -> dict:
    """Estimated backlog drain time of each class under block quotas M (inf for a class without quota)."""
    return {b: (N[b] * kbar[b] * That[b] / M[b] if M[b] > 0 else math.inf) for b in N}


class ClassEstimator:
    """Bounded histories of completed sessions: peak blocks and residency duration per class."""

    def __init__(self, kbar_prior: dict, T_prior: float, window: int = 64, prior_weight: float = 4.0):
        self.kbar_prior = dict(kbar_prior)
        self.T_prior = float(T_prior)
        self.window = window
        self.prior_weight = prior_weight
        self.blocks = {b: deque(maxlen=window) for b in kbar_prior}
        self.durations = {b: deque(maxlen=window) for b in kbar_prior}
        self.all_blocks = deque(maxlen=window)

    def observe(self, b: str, peak_blocks: int, duration: float):
        self.blocks[b].append(peak_blocks)
        self.durations[b].append(duration)
        self.all_blocks.append(peak_blocks)

    @staticmethod
    def _p90(xs) -> float:
        s = sorted(xs)
        return float(s[min(len(s) - 1, int(math.ceil(0.9 * len(s))) - 1)])

    def kbar(self, b: str) -> float:
        h = self.blocks[b]
        return max(self.kbar_prior[b], self._p90(h)) if h else float(self.kbar_prior[b])

    def kbar_global(self, N: dict | None = None) -> float:
        """Reference footprint of a session of the mix N (demand per class)."""
        tot = sum(N.values()) if N else 0
        if tot == 0:
            return sum(self.kbar(b) for b in self.kbar_prior) / len(self.kbar_prior)
        return sum(N[b] * self.kbar(b) for b in N) / tot

    def That(self, b: str) -> float:
        h = self.durations[b]
        return (self.prior_weight * self.T_prior + sum(h)) / (self.prior_weight + len(h))


class Controller:
    """Admission for one instance.  policy: 'global' (the session cap of Sec. 4.1 only), 'space' (MISA: plus
    the class caps of Eq. workloadcap) or 'time' (MISA-T: plus the class caps of Eq. residency-quota)."""

    def __init__(self, C: int, estimator: ClassEstimator, policy: str = "time", g_threshold: float = 0.1,
                 confirm: int = 3, contract: float = 0.8, window: int = 32):
        assert policy in ("global", "space", "time")
        self.C, self.est, self.policy = C, estimator, policy
        self.O, self.P = {}, {}          # session -> class (active / pending)
        self.K = base_cap(C, estimator.kbar_global())
        self.g_threshold, self.confirm, self.contract = g_threshold, confirm, contract
        self.healthy = deque(maxlen=window)
        self.bad_streak = 0
        self.class_caps = {b: self.K for b in CLASSES}
        self.quota = {b: 0.0 for b in CLASSES}

    def snapshot(self, finished):
        """A new cache snapshot: pending sessions become visible as active, finished ones leave."""
        self.O.update(self.P)
        self.P.clear()
        for s in finished:
            self.O.pop(s, None)

    def update_caps(self, demand: dict, hit_rate: float | None = None):
        """Recompute the global cap (with overload pressure) and the class caps from the demand ledger
        N_b (active, pending, held and candidate sessions of each class)."""
        N = {b: demand.get(b, 0) for b in CLASSES}
        kb = max(1, base_cap(self.C, self.est.kbar_global(N)))
        if hit_rate is not None:
            h_ref = max(self.healthy) if self.healthy else hit_rate
            if hit_degradation(h_ref, hit_rate) > self.g_threshold:
                self.bad_streak += 1
            else:
                self.bad_streak = 0
                self.healthy.append(hit_rate)
        if self.bad_streak >= self.confirm:
            self.K = max(1, int(self.K * self.contract))
            self.bad_streak = 0
        else:
            self.K = min(kb, self.K + 1) if self.K < kb else kb
        kbar = {b: self.est.kbar(b) for b in CLASSES}
        if self.policy == "space":
            self.quota, self.class_caps = space_caps(self.C, N, kbar)
        elif self.policy == "time":
            self.quota, self.class_caps = time_caps(self.C, N, kbar, {b: self.est.That(b) for b in CLASSES})
        else:
            self.quota, self.class_caps = {b: float(self.C) for b in CLASSES}, {b: self.K for b in CLASSES}

    def admit(self, s, b: str) -> bool:
        """Admit(r, w) for a request of session s, class b; a newly admitted session becomes pending."""
        if s in self.O or s in self.P:
            return True
        if len(self.O) + len(self.P) >= self.K:
            return False
        if self.policy != "global":
            held = sum(1 for c in self.O.values() if c == b) + sum(1 for c in self.P.values() if c == b)
            if held >= self.class_caps[b]:
                return False
        self.P[s] = b
        return True
