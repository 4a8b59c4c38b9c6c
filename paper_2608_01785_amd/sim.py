"""Discrete-event model of one GPU serving a shared stage and a downstream stage.

It runs the scheduling loop of Algorithm 1 (§4.5) step by step.  The temporal
scheduler and the spatial controller are the library's own, called through
the C ABI.  Kernel times come from a Timing table filled with measured
values.  The model reproduces the shape of the policy comparison (baseline,
temporal only, spatial only, joint) without the paper's models or datasets.
Its numbers are model outputs, not measurements.

Model:
* Requests arrive as a seeded Poisson process.  A fraction `p_long` are
  long-path requests (they continue to the downstream stage); the rest are
  short-path requests, which end with the shared stage.  Prompt lengths follow
  the thinker workload's recipe (uniform 256..2048 tokens).
* First response: a short request's is the end of the shared-stage step that
  prefills it.  A long request's comes after `first_chunk_steps` downstream
  decode steps; it then decodes `tail_steps` more steps before leaving.
* Deadlines follow §4.2: Delta_c = m_c x p95 of the class's solo
  first-response time (each request alone on the whole GPU).  The remaining
  time estimate r_hat is that solo time, less the downstream steps done.
* One scheduling step: the temporal view (all requests visible without
  temporal control), then an FCFS base scheduler over the visible waiting
  prefills up to `token_budget` prompt tokens (always at least one), then the
  CU split.  Without spatial control both stages run unmasked on the whole
  chip and slow each other by the measured unmasked co-run factors.  With it
  the controller's split applies, times come from the per-CU tables, and the
  measured masked co-run factors apply while both stages run.
* The downstream stage decodes all active long requests as one batch.  Its
  step time scales with the batch the way the talker step's bytes do
  (weights once, plus the key/value rows of each sequence).
* The memory-pressure sample is the downstream stage's share of peak HBM
  bandwidth while it runs (0 otherwise).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np


@dataclasses.dataclass
class Timing:
    prefill_ms_per_token: Dict[int, float]   # shared-stage CU cap -> ms per prompt token, solo
    decode_ms_per_step: Dict[int, float]     # downstream CU count -> ms per step at decode_batch, solo
    decode_batch: int                        # batch those step times were measured at
    weight_share: float                      # fraction of a measured step's bytes that are weights
    masked_prefill_factor: float             # prefill time while the downstream co-runs on the complement
    masked_decode_factor: float
    unmasked_prefill_factor: float           # both stages unmasked on the whole chip
    unmasked_decode_factor: float
    decode_full_ms: float                    # downstream step on the whole chip, solo, at decode_batch
    hbm_share: float                         # downstream share of peak HBM bandwidth at decode_batch, masked co-run

    def down_hbm_share(self, batch: int) -> float:
        """Memory-pressure sample while the downstream runs: its bytes scale with the batch."""
        return min(1.0, self.hbm_share * (self.weight_share + (1.0 - self.weight_share) * batch / self.decode_batch))

    def prefill_ms(self, tokens: int, cus: int) -> float:
        caps = sorted(self.prefill_ms_per_token)
        per = float(np.interp(cus, caps, [self.prefill_ms_per_token[c] for c in caps]))
        return tokens * per

    def decode_ms(self, batch: int, cus: Optional[int]) -> float:
        """cus None: the whole chip."""
        if cus is None:
            base = self.decode_full_ms
        else:
            caps = sorted(self.decode_ms_per_step)
            base = float(np.interp(cus, caps, [self.decode_ms_per_step[c] for c in caps]))
        return base * (self.weight_share + (1.0 - self.weight_share) * batch / self.decode_batch)


@dataclasses.dataclass
class Workload:
    n_requests: int = 400
    rate_per_s: float = 20.0
    p_long: float = 0.5
    first_chunk_steps: int = 20
    tail_steps: int = 100
    token_budget: int = 8192
    slo_multiplier: float = 5.0
    idle_tick_ms: float = 1.0       # a scheduling step with an empty view lasts at most this long
    seed: int = 7


@dataclasses.dataclass
class Request:
    arrival: float
    tokens: int
    long: bool
    deadline: float = 0.0
    solo: float = 0.0
    prefilled_at: Optional[float] = None
    steps_done: int = 0
    first_response: Optional[float] = None
    done: bool = False


def make_requests(w: Workload) -> List[Request]:
    rng = np.random.default_rng(w.seed)
    gaps = rng.exponential(1000.0 / w.rate_per_s, size=w.n_requests)
    arrivals = np.cumsum(gaps)
    tokens = rng.integers(256, 2048, size=w.n_requests, endpoint=True)
    long = rng.uniform(size=w.n_requests) < w.p_long
    return [Request(float(a), int(t), bool(l)) for a, t, l in zip(arrivals, tokens, long)]


def assign_deadlines(reqs: List[Request], t: Timing, w: Workload, total_cus: int) -> Dict[str, float]:
    """Delta_c = m_c x p95 of the class's solo first-response times (§4.2)."""
    for r in reqs:
        r.solo = t.prefill_ms(r.tokens, total_cus) + (w.first_chunk_steps * t.decode_ms(1, None) if r.long else 0.0)
    delta = {}
    for name, flag in (("short", False), ("long", True)):
        solos = [r.solo for r in reqs if r.long == flag]
        delta[name] = w.slo_multiplier * float(np.percentile(solos, 95)) if solos else 0.0
    for r in reqs:
        r.deadline = r.arrival + delta["long" if r.long else "short"]
    return delta


def simulate(policy: str, t: Timing, w: Workload, temporal_cfg=None, controller_cfg=None,
             total_cus: int = 256) -> dict:
    """policy: "baseline", "temporal", "spatial" or "joint"."""
    from paper_2608_01785_amd import binding as B
    use_temporal = policy in ("temporal", "joint")
    use_spatial = policy in ("spatial", "joint")
    reqs = make_requests(w)
    delta = assign_deadlines(reqs, t, w, total_cus)
    tc = temporal_cfg or dict(n_min=2, n_max=8, m=2, u_guard=1.0, long_cap=4)
    cc = controller_cfg or dict(total_cus=total_cus, aggressive_cus=total_cus, ladder=[64, 96, 128, 160, 192],
                                ewma_weight=0.4, saturation=0.5, hysteresis_steps=1)
    sched = B.Temporal(**tc) if use_temporal else None
    ctrl = B.Controller(**cc) if use_spatial else None
    now, nxt = 0.0, 0
    waiting: List[Request] = []
    active: List[Request] = []      # long requests in the downstream stage
    shares = []
    down_progress = 0.0             # fractional downstream steps carried between events
    try:
        while nxt < len(reqs) or waiting or active:
            while nxt < len(reqs) and reqs[nxt].arrival <= now:
                waiting.append(reqs[nxt])
                nxt += 1
            if not waiting and not active:
                now = reqs[nxt].arrival
                continue
            # Step 1-2: the temporal view and the base scheduler's batch.
            visible = [True] * len(waiting)
            if sched is not None and waiting:
                views = [(B.HS_PATH_LONG if r.long else B.HS_PATH_SHORT, B.HS_WORK_PREFILL, r.deadline,
                          max(r.solo, 1e-6)) for r in waiting]
                visible, _ = B.hs_temporal_step(sched, now, views)
            batch, tokens = [], 0
            for r, v in zip(waiting, visible):
                if v and (not batch or tokens + r.tokens <= w.token_budget):
                    batch.append(r)
                    tokens += r.tokens
            # Step 3: the CU split.
            down_on = bool(active)
            s_shared = total_cus
            if ctrl is not None:
                sample = t.down_hbm_share(len(active)) if down_on else 0.0
                sp = B.hs_controller_step(ctrl, down_on, sample)
                s_shared = sp.shared_cus
            shares.append(s_shared)
            # Step 4: execute.  Duration of this step and the downstream's progress during it.
            if batch:
                if ctrl is None:
                    dur = t.prefill_ms(tokens, total_cus) * (t.unmasked_prefill_factor if down_on else 1.0)
                else:
                    dur = t.prefill_ms(tokens, s_shared) * (t.masked_prefill_factor if down_on else 1.0)
            else:
                # Nothing visible to prefill (an empty queue view): the step passes
                # after one downstream step, the next arrival or an idle tick.
                next_arrival = reqs[nxt].arrival - now if nxt < len(reqs) else float("inf")
                one = t.decode_ms(len(active), None if ctrl is None else total_cus - s_shared) if active else w.idle_tick_ms
                dur = max(min(next_arrival, one, w.idle_tick_ms if waiting else float("inf")), 1e-3)
            if active:
                cus = None if ctrl is None else (total_cus - s_shared if s_shared < total_cus else None)
                step = t.decode_ms(len(active), cus)
                if batch:
                    step *= t.unmasked_decode_factor if cus is None else t.masked_decode_factor
                down_progress += dur / step
                k = int(down_progress)
                down_progress -= k
                for _ in range(k):
                    for r in active:
                        r.steps_done += 1
                        if r.first_response is None and r.steps_done >= w.first_chunk_steps:
                            r.first_response = now + dur
                        if r.steps_done >= w.first_chunk_steps + w.tail_steps:
                            r.done = True
                    active = [r for r in active if not r.done]
                    if not active:
                        break
            now += dur
            for r in batch:
                r.prefilled_at = now
                waiting.remove(r)
                if r.long:
                    active.append(r)
                else:
                    r.first_response = now
                    r.done = True
            if not active:
                down_progress = 0.0
    finally:
        if sched is not None:
            sched.close()
        if ctrl is not None:
            ctrl.close()
    out = {"policy": policy, "delta_ms": {k: round(v, 2) for k, v in delta.items()},
           "mean_shared_cus": round(float(np.mean(shares)), 1) if shares else None}
    for name, flag in (("short", False), ("long", True)):
        rs = [r for r in reqs if r.long == flag]
        lat = np.array([r.first_response - r.arrival for r in rs])
        met = np.array([r.first_response <= r.deadline for r in rs])
        out[name] = {"n": len(rs), "slo_attainment": round(float(met.mean()), 4) if len(rs) else None,
                     "p50_ms": round(float(np.percentile(lat, 50)), 2) if len(rs) else None,
                     "p95_ms": round(float(np.percentile(lat, 95)), 2) if len(rs) else None}
    return out


def compare(t: Timing, w: Optional[Workload] = None) -> List[dict]:
    w = w or Workload()
    return [simulate(p, t, w) for p in ("baseline", "temporal", "spatial", "joint")]
