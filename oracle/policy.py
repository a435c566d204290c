"""Layout-switch policy (Sec. 4.5) and the TP->EP request partition
(Sec. 3.2), written out from the paper's description: a plain, slow CPU
reference.

TEST INFRASTRUCTURE ONLY: imported by tests/ and never by the product path.

Readings where the paper leaves a choice (each also listed with the design
notes):
  P1  "Balancing request and token counts together": a rank's load is the sum
      of its share of all tokens and its share of all requests,
      tokens_r / T + requests_r / N (exact rationals here).  Ties between
      ranks go to the lower rank; requests of equal length keep their input
      order.
  P2  The policy's window holds the counts of the last W iterations whatever
      the mode was; with fewer than W samples so far the mean is over those.
  P3  The cooldown C runs from the last switch and from the last cancelled
      attempt; no attempt is made while it runs.  At start there is none.
  P4  "Exceeds" and "falls below" are strict: count > T_h, mean < T_l.
  P5  KV capacity is counted in (page, head) units per rank: a request of n
      tokens takes ceil(n / page_size) pages of every head its rank holds.
      Under EP a rank holds all n_kv heads of its own requests; under TP each
      rank holds max(1, n_kv / P) heads of every request (a head is
      replicated over P / n_kv ranks when n_kv < P).
  P6  Calibration picks, among the probed batch sizes, the smallest from
      which EP is no slower than TP at that size and every larger one; when
      EP never wins the threshold is infinite (stay in TP).
"""
from __future__ import annotations

from collections import deque
from fractions import Fraction
import math

TP, EP = 0, 1
STAY, SWITCH, CANCELLED = 0, 1, 2


def partition(tokens: list, P: int) -> list:
    """Owner rank of every request: sorted by decreasing length, each placed
    on the rank whose load (P1) is smallest at that moment."""
    N = len(tokens)
    T = sum(tokens)
    order = sorted(range(N), key=lambda i: (-tokens[i], i))
    tok = [0] * P
    req = [0] * P
    owner = [0] * N

    def load(r):
        a = Fraction(tok[r], T) if T else Fraction(0)
        return a + Fraction(req[r], N)

    for i in order:
        best = min(range(P), key=lambda r: (load(r), r))
        owner[i] = best
        tok[best] += tokens[i]
        req[best] += 1
    return owner


def kv_fits(mode: int, tokens: list, P: int, n_kv: int, page_size: int, capacity: int,
            owner: list | None = None) -> bool:
    """Whether every rank's pool (`capacity` (page, head) units) holds the
    live requests in `mode` (P5); EP needs the owner of every request."""
    pages = [-(-n // page_size) for n in tokens]
    if mode == TP:
        heads = max(1, n_kv // P)
        return sum(pages) * heads <= capacity
    use = [0] * P
    for i, p in enumerate(pages):
        use[owner[i]] += p * n_kv
    return max(use) <= capacity


class Policy:
    """The coordinator's state machine, sampled once per decode iteration."""

    def __init__(self, t_high: float, t_low: float, window: int, cooldown_s: float, mode: int = TP):
        self.t_high, self.t_low, self.window, self.cooldown = t_high, t_low, window, cooldown_s
        self.mode = mode
        self.hist = deque(maxlen=window)
        self.last_event = None

    def step(self, count: int, now_s: float, target_fits: bool) -> int:
        self.hist.append(count)
        if self.last_event is not None and now_s - self.last_event < self.cooldown:
            return STAY
        if self.mode == TP:
            want = count > self.t_high
        else:
            want = sum(self.hist) / len(self.hist) < self.t_low
        if not want:
            return STAY
        self.last_event = now_s
        if not target_fits:
            return CANCELLED
        self.mode = EP if self.mode == TP else TP
        return SWITCH


def crossover(batch: list, tp_cost: list, ep_cost: list) -> float:
    """Initial threshold from probed decode costs (P6)."""
    pts = sorted(zip(batch, tp_cost, ep_cost))
    best = math.inf
    for b, t, e in reversed(pts):
        if e <= t:
            best = b
        else:
            break
    return best
