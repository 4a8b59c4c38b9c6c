"""Shared-stage path rotation (the temporal scheduler).  TEST INFRASTRUCTURE ONLY.

Follows §4.2 ("Remaining-slack ratio"), §4.3 (path rotation, slack guard,
adaptive rotation ratio, long-path admission cap) and steps 1 and 2 of
Algorithm 1, in their order and notation:

* Slack: u_i(t) = (d_i - t) / r_hat_i(t); request i is protected when
  u_i(t) < u_guard.
* Adaptive ratio: M is fixed; N is the fraction of waiting short-path
  requests that are protected, mapped linearly onto [N_min, N_max] and
  rounded.
* Rotation: step k is a short-path phase when k mod (N + M) < N, else a
  long-path phase.  Ordinary prefills of the other path are hidden for the
  step; protected requests and decode continuations stay visible.
* Long-path cap: at most `long_cap` ordinary long-path prefills stay visible;
  when more are candidates, earlier deadlines go first.  Protected requests
  are exempt (always visible, not counted).

Readings of what the paper leaves open (each also listed in the design notes):

* "Waiting short-path requests" are short-path prefills in the queue; with
  none waiting the fraction is 0 (N = N_min).
* Rounding is to the nearest integer, halves upward.
* N is re-evaluated every step and the phase test uses the current N with the
  global step counter k.
* During a long-path phase ordinary short-path prefills are hidden (the paper
  says they "can be"; hiding is the symmetric reading).
* Ties in the cap's deadline order go to the earlier queue position.
* The cap value is not printed: it is a configuration parameter; a negative
  cap means no cap.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Sequence

SHORT, LONG = 0, 1
PREFILL, DECODE = 0, 1


class TemporalError(ValueError):
    pass


@dataclass
class Request:
    path: int          # SHORT or LONG
    work: int          # PREFILL (waiting) or DECODE (continuation)
    deadline: float    # d_i
    remaining: float   # r_hat_i(t) > 0


@dataclass
class StepInfo:
    step: int
    n: int
    phase: int
    n_protected: int
    n_hidden: int
    n_capped: int


def round_half_up(x: float) -> int:
    return int(math.floor(x + 0.5))


class TemporalScheduler:
    def __init__(self, n_min: int = 2, n_max: int = 8, m: int = 2, u_guard: float = 1.0, long_cap: int = -1):
        if not (1 <= n_min <= n_max) or m < 1 or not (u_guard > 0.0):
            raise TemporalError("need 1 <= N_min <= N_max, M >= 1, u_guard > 0")
        self.n_min, self.n_max, self.m = int(n_min), int(n_max), int(m)
        self.u_guard, self.long_cap = float(u_guard), int(long_cap)
        self.k = 0

    def step(self, now: float, reqs: Sequence[Request]):
        """Returns (visible flags, StepInfo); the queue itself is never changed."""
        for r in reqs:
            if not (r.remaining > 0.0) or not math.isfinite(r.deadline):
                raise TemporalError("remaining estimates must be > 0 and deadlines finite")
        # Step 1: slack and the protected bit.
        prot = [(r.deadline - now) / r.remaining < self.u_guard for r in reqs]
        # Adaptive ratio: protected share of the waiting short-path prefills.
        short_wait = [i for i, r in enumerate(reqs) if r.work == PREFILL and r.path == SHORT]
        frac = (sum(prot[i] for i in short_wait) / len(short_wait)) if short_wait else 0.0
        n = round_half_up(self.n_min + frac * (self.n_max - self.n_min))
        # Rotation phase of step k.
        phase = SHORT if self.k % (n + self.m) < n else LONG
        visible = []
        for i, r in enumerate(reqs):
            visible.append(r.work == DECODE or prot[i] or r.path == phase)
        n_hidden = sum(1 for v in visible if not v)
        # Long-path cap over the ordinary long-path prefills still visible.
        cand = [i for i, r in enumerate(reqs)
                if visible[i] and r.work == PREFILL and r.path == LONG and not prot[i]]
        n_capped = 0
        if self.long_cap >= 0 and len(cand) > self.long_cap:
            order = sorted(cand, key=lambda i: (reqs[i].deadline, i))
            for i in order[self.long_cap:]:
                visible[i] = False
                n_capped += 1
        info = StepInfo(self.k, n, phase, sum(prot), n_hidden, n_capped)
        self.k += 1
        return visible, info


def run(sched: TemporalScheduler, steps) -> List:
    """steps: sequence of (now, requests); returns [(visible, info)]."""
    return [sched.step(t, reqs) for t, reqs in steps]
