"""Bandwidth-guided shared-stage cap (the spatial controller).  TEST INFRASTRUCTURE ONLY.

Follows the paper's spatial controller, §4.4 ("Bandwidth-guided SM
throttling"), and step 3 of Algorithm 1, in their order and notation:

* Bandwidth-pressure signal: the sampled memory activity B(t) is smoothed by
  an EWMA  B_hat(t) = gamma * B(t) + (1 - gamma) * B_hat(t - 1).
* Ladder, Eq. (1): rho(t) = clamp(B_hat(t) / B_sat, 0, 1) and
      s*(t) = S_aggr                                         if A(t) = 0
      s*(t) = snap_S(S_min + rho(t) * (S_cap - S_min))       if A(t) > 0
  where S = (S_min, ..., S_cap) is the co-running ladder and
  S_cap < S_aggr <= S_tot.
* Step 3: apply s* if downstream stages are inactive or the ladder level
  moves by at least Delta_step from the previous cap; otherwise keep s_prev.
  The downstream stage gets s_down = max(0, S_tot - s_shared).

Readings of what the paper leaves open (each also listed in the design notes):

* gamma weighs the newest sample; the first sample initialises B_hat.
* snap_S is the nearest ladder level; a tie goes to the larger level.
* "the ladder level changes by Delta_step" compares ladder indices.  When the
  previous cap is not a ladder level (the first step, or the aggressive cap
  while downstream was idle) the new level is applied.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence


class ControllerError(ValueError):
    pass


@dataclass
class Decision:
    shared: int
    down: int
    level: int        # index into the ladder, -1 for the aggressive cap
    changed: bool
    pressure: float   # B_hat
    rho: float


def snap(ladder: Sequence[int], x: float) -> int:
    """Index of the ladder level nearest to x (ties to the larger level)."""
    best = 0
    for i, s in enumerate(ladder):
        if abs(s - x) <= abs(ladder[best] - x):
            best = i
    return best


class SpatialController:
    def __init__(self, total: int, aggressive: int, ladder: Sequence[int], gamma: float, saturation: float,
                 hysteresis_steps: int = 1):
        ladder = [int(s) for s in ladder]
        if not ladder or any(b <= a for a, b in zip(ladder, ladder[1:])) or ladder[0] < 1:
            raise ControllerError("ladder must be strictly increasing and start at >= 1")
        if not (ladder[-1] < aggressive <= total):
            raise ControllerError("need S_cap < S_aggr <= S_tot")
        if not (0.0 < gamma <= 1.0) or not (saturation > 0.0) or hysteresis_steps < 1:
            raise ControllerError("need 0 < gamma <= 1, B_sat > 0, Delta_step >= 1")
        self.total, self.aggressive, self.ladder = int(total), int(aggressive), ladder
        self.gamma, self.saturation, self.step_min = float(gamma), float(saturation), int(hysteresis_steps)
        self.b_hat: Optional[float] = None
        self.prev_shared: Optional[int] = None
        self.prev_level = -1

    def step(self, downstream_active: bool, sample: float) -> Decision:
        # Step 1: refresh the pressure signal.
        if self.b_hat is None:
            self.b_hat = float(sample)
        else:
            self.b_hat = self.gamma * float(sample) + (1.0 - self.gamma) * self.b_hat
        rho = min(max(self.b_hat / self.saturation, 0.0), 1.0)
        # Eq. (1).
        if not downstream_active:
            target, level = self.aggressive, -1
        else:
            s_min, s_cap = self.ladder[0], self.ladder[-1]
            level = snap(self.ladder, s_min + rho * (s_cap - s_min))
            target = self.ladder[level]
        # Step 3: hysteresis on the ladder level.
        apply = (not downstream_active or self.prev_shared is None or self.prev_level < 0
                 or abs(level - self.prev_level) >= self.step_min)
        if apply:
            changed = self.prev_shared != target
            self.prev_shared, self.prev_level = target, level
        else:
            changed = False
        shared = self.prev_shared
        return Decision(shared, max(0, self.total - shared), self.prev_level, changed, self.b_hat, rho)


def run(ctrl: SpatialController, active: Sequence[bool], samples: Sequence[float]) -> List[Decision]:
    return [ctrl.step(bool(a), float(b)) for a, b in zip(active, samples)]
