"""Algorithm 1 (§4.5) on the GPU: the scheduling loop over the library's kernels.

Each scheduling step k:

1. the pressure sample B(k) and each request's remaining-time estimate are read
   (step 1 of the algorithm);
2. the temporal scheduler forms the visible view of the queue: path rotation,
   slack guard, long-path cap (step 2; ``hs_temporal_step``);
3. the spatial controller picks the shared stage's CU cap from the smoothed
   pressure and whether the downstream stage is active; the downstream stage
   gets the complement (step 3; ``hs_controller_step``);
4. the base scheduler (first come, first served over the visible prefills, up
   to a prompt-token budget) forms the batch, which is prefilled through the
   shared stage on the CU-masked stream of the cap, while decode steps of the
   active downstream requests loop on the complementary stream (step 4;
   ``hs_shared_stage_forward``, ``hs_downstream_decode_step``).

The baseline policy shows every request and runs both stages unmasked on the
whole chip.  First responses come from GPU events: a short-path request's is
the end of its prefill step, a long-path request's the end of its
``first_chunk``-th downstream step, each measured from its arrival.

Pressure signal.  The paper samples the GPU's memory activity.  MI355X's
memory-controller activity (``hs_pressure_sample``) is a firmware average
refreshed about once per second, far longer than a scheduling step, so the
default signal here is the downstream stage's own traffic: the algorithmic
bytes of the decode steps completed in the previous scheduling step (weights
once, cached keys and values read, new rows written) over the GPU time they
took, as a share of the 8 TB/s peak.  ``pressure="amdsmi"`` uses the AMD SMI
reading instead, polled while the previous step's work was in flight.
"""
from __future__ import annotations

import dataclasses
import time
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import binding

PEAK_HBM_BYTES_PER_MS = 8.0e9   # 8 TB/s


def decode_step_bytes(shape, n_layers: int, kv_lens) -> int:
    """Algorithmic HBM bytes of one decode step: every weight once, the cached
    keys and values of each row read once, the new rows written (fp16 cache)."""
    per_row = 2 * shape.n_kv_heads * shape.head_dim * 2
    kv = np.asarray(kv_lens, np.int64)
    return int(n_layers * (shape.params_per_layer * 2 + per_row * (int(kv.sum()) + len(kv))))


@dataclasses.dataclass
class LoopConfig:
    policy: str = "joint"               # "baseline" or "joint"
    token_budget: int = 4096            # base scheduler: prompt tokens per step
    short_budget: int = 0               # joint: prompt tokens per short-path phase step (0: token_budget)
    first_chunk: int = 20               # downstream steps before a long-path request's first response
    n_min: int = 2
    n_max: int = 8
    m: int = 2
    u_guard: float = 1.0
    long_cap: int = 4
    ladder: Sequence[int] = (128, 160, 192, 224)
    ewma: float = 0.4
    saturation: float = 0.25            # B_sat, in the pressure signal's units
    hysteresis: int = 1
    pressure: str = "traffic"           # "traffic" or "amdsmi"


@dataclasses.dataclass
class Request:
    rid: int
    arrival: float       # ms from the loop's start
    tokens: int          # prompt rows
    long: bool           # continues to the downstream stage
    kv0: int             # downstream cache rows before its first downstream step
    deadline: float      # ms from the loop's start
    solo: float          # solo first-response estimate (ms)


@dataclasses.dataclass
class StepRecord:
    k: int
    now: float
    waiting: List[int]
    views: List[tuple]              # (path, work, deadline, remaining) passed to the temporal scheduler
    visible: List[bool]
    info: Dict[str, int]
    active: bool
    sample: float
    split: Dict[str, float]
    batch: List[int]
    batch_tokens: int
    offsets: List[int]
    down_ids: List[int]
    down_steps: int
    down_cus: int


class Algorithm1:
    """The loop of Algorithm 1 over one context.

    thinker / talker: (shape, device weights, n_layers).  x_pool: bf16 device
    rows [>= token_budget, hidden]; a batch's prompt rows are its first rows.
    requests must be sorted by arrival.  max_ctx: downstream positions per
    request (one cache page each)."""

    def __init__(self, ctx, thinker, talker, requests: List[Request], x_pool, cfg: LoopConfig, max_ctx: int,
                 x_talker=None, device="cuda"):
        import torch
        from .device_data import DeviceCache
        self.torch, self.ctx, self.cfg = torch, ctx, cfg
        self.th_shape, self.th_w, self.th_layers = thinker
        self.tk_shape, self.tk_w, self.tk_layers = talker
        self.reqs = requests
        n = len(requests)
        self.n_cus = 256
        self.joint = cfg.policy == "joint"
        if cfg.policy not in ("joint", "baseline"):
            raise ValueError(f"policy {cfg.policy!r}")
        if cfg.pressure not in ("traffic", "amdsmi"):
            raise ValueError(f"pressure signal {cfg.pressure!r}")
        self.x_pool = x_pool
        self.y = torch.empty((cfg.token_budget, self.th_shape.hidden), dtype=torch.float32, device=device)
        max_pos = int(max(r.tokens for r in requests))
        self.ws = torch.empty(binding.hs_workspace_size(self.th_shape, cfg.token_budget, n, max_pos),
                              dtype=torch.uint8, device=device)
        self.max_ctx = max_ctx
        self.cache = DeviceCache(self.tk_layers, n, max_ctx, self.tk_shape.n_kv_heads, self.tk_shape.head_dim, device)
        gen = torch.Generator(device=device)
        gen.manual_seed(12345)
        for l in range(self.tk_layers):
            for r in requests:
                if r.long:
                    self.cache.fill_random(l, r.rid, int(r.kv0), gen)
        if x_talker is None:
            x_talker = torch.zeros((n, self.tk_shape.hidden), dtype=torch.bfloat16, device=device)
        self.xt = x_talker
        self.yt = torch.empty((n, self.tk_shape.hidden), dtype=torch.float32, device=device)
        self.wst = torch.empty(binding.hs_workspace_size_paged(self.tk_shape, n, n, max_ctx, max_ctx),
                               dtype=torch.uint8, device=device)
        self.sched = binding.Temporal(cfg.n_min, cfg.n_max, cfg.m, cfg.u_guard, cfg.long_cap) if self.joint else None
        self.ctrl = binding.Controller(self.n_cus, self.n_cus, list(cfg.ladder), cfg.ewma, cfg.saturation,
                                       cfg.hysteresis) if self.joint else None
        self.full = torch.cuda.Stream(device=device)
        self.s_full = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, self.n_cus, binding.HS_ROLE_SHARED))
        self.waiting: List[int] = []
        self.active: List[int] = []
        self.nxt = 0
        self.kv = np.array([r.kv0 for r in requests], np.int32)
        self.issued = np.zeros(n, int)
        self.done_steps = np.zeros(n, int)
        self.first = np.full(n, np.nan)
        self.k = 0
        self.records: List[StepRecord] = []
        self._sample = 0.0          # B(k) for the next step
        self._polls: List[float] = []
        self.start = None
        self.t0 = None

    # ------------------------------------------------------------------ helpers
    def now(self) -> float:
        return (time.perf_counter() - self.t0) * 1e3

    def _down_stream(self, s_shared: int):
        if self.joint and s_shared < self.n_cus:
            return self.torch.cuda.ExternalStream(binding.hs_context_stream(self.ctx, s_shared, binding.HS_ROLE_DOWN))
        return self.full

    def _talker_step(self, s_shared: int, ids: np.ndarray):
        table = ids[:, None].astype(np.int32)
        kv = (self.cache.k, self.cache.v, len(self.reqs), self.max_ctx, table)
        if self.joint and s_shared < self.n_cus:
            binding.hs_downstream_decode_step(self.ctx, self.tk_shape, self.tk_w, self.xt, self.yt, kv, self.kv[ids],
                                              self.n_cus - s_shared, None, self.wst)
        else:
            binding.hs_downstream_decode_step(self.ctx, self.tk_shape, self.tk_w, self.xt, self.yt, kv, self.kv[ids],
                                              self.n_cus, self.full.cuda_stream, self.wst)
        e = self.torch.cuda.Event(enable_timing=True)
        e.record(self._down_stream(s_shared))
        return e

    def _poll(self):
        if self.cfg.pressure == "amdsmi":
            self._polls.append(binding.hs_pressure_sample(0))   # raises when AMD SMI cannot be read

    # ------------------------------------------------------------------ one step
    def begin(self):
        torch = self.torch
        torch.cuda.synchronize()
        self.start = torch.cuda.Event(enable_timing=True)
        self.start.record(self.s_full)
        self.full.wait_event(self.start)
        self.t0 = time.perf_counter()

    def step(self) -> Optional[StepRecord]:
        """One scheduling step; None when every request has its first response."""
        torch, cfg = self.torch, self.cfg
        n = len(self.reqs)
        now = self.now()
        while self.nxt < n and self.reqs[self.nxt].arrival <= now:
            self.waiting.append(self.nxt)
            self.nxt += 1
        if not self.waiting and not self.active:
            if self.nxt >= n:
                return None
            time.sleep(max(0.0, (self.reqs[self.nxt].arrival - now) / 1e3))
            return self.step()
        # Step 1: remaining-time estimates (each waiting prefill's solo time).
        waiting = list(self.waiting)
        views = []
        for i in self.waiting:
            r = self.reqs[i]
            views.append((binding.HS_PATH_LONG if r.long else binding.HS_PATH_SHORT, binding.HS_WORK_PREFILL,
                          r.deadline, r.solo))
        # Step 2: the visible view.
        visible, info = [True] * len(self.waiting), None
        if self.sched is not None and self.waiting:
            vis, inf = binding.hs_temporal_step(self.sched, now, views)
            visible = [bool(v) for v in vis]
            info = {"step": int(inf.step), "n": int(inf.n), "phase": int(inf.phase),
                    "n_protected": int(inf.n_protected), "n_hidden": int(inf.n_hidden),
                    "n_capped": int(inf.n_capped)}
        # Step 3: the CU split.
        act = bool(self.active)
        sample = self._sample
        split = {"shared_cus": self.n_cus, "down_cus": 0, "level": -1, "changed": 0, "pressure": 0.0, "rho": 0.0}
        if self.ctrl is not None:
            sp = binding.hs_controller_step(self.ctrl, act, sample)
            split = {"shared_cus": int(sp.shared_cus), "down_cus": int(sp.down_cus), "level": int(sp.level),
                     "changed": int(sp.changed), "pressure": float(sp.pressure), "rho": float(sp.rho)}
        s_sh = split["shared_cus"]
        # Step 4: the base scheduler's batch over the visible view.
        budget = cfg.token_budget
        if self.joint and cfg.short_budget and info is not None and info["phase"] == binding.HS_PATH_SHORT:
            budget = cfg.short_budget
        batch, tok = [], 0
        for i, v in zip(self.waiting, visible):
            if v and (not batch or tok + self.reqs[i].tokens <= budget):
                batch.append(i)
                tok += self.reqs[i].tokens
        offsets = [0]
        for i in batch:
            offsets.append(offsets[-1] + self.reqs[i].tokens)
        cur_ids = [i for i in self.active if self.issued[i] < cfg.first_chunk]
        down_cus = self.n_cus - s_sh if (self.joint and s_sh < self.n_cus) else self.n_cus
        pend, p_end = [], None
        t_down0 = None
        if batch:
            stream = self.s_full if s_sh == self.n_cus else torch.cuda.ExternalStream(
                binding.hs_context_stream(self.ctx, s_sh, binding.HS_ROLE_SHARED))
            if cur_ids:
                t_down0 = torch.cuda.Event(enable_timing=True)
                t_down0.record(self._down_stream(s_sh))
            binding.hs_shared_stage_forward(self.ctx, self.th_shape, self.th_w, self.x_pool[:tok], self.y[:tok],
                                            offsets, None, None, s_sh, None, self.ws)
            p_end = torch.cuda.Event(enable_timing=True)
            p_end.record(stream)
            while not p_end.query():
                cur = np.array([i for i in self.active if self.issued[i] < cfg.first_chunk], np.int32)
                if len(cur) == 0:
                    break
                pend.append((self._talker_step(s_sh, cur), cur,
                             decode_step_bytes(self.tk_shape, self.tk_layers, self.kv[cur])))
                self.kv[cur] += 1
                self.issued[cur] += 1
                self._poll()
                if len(pend) > 3:
                    pend[-4][0].synchronize()
        elif self.active:
            cur = np.array(cur_ids, np.int32)
            if len(cur):
                t_down0 = torch.cuda.Event(enable_timing=True)
                t_down0.record(self._down_stream(s_sh))
                pend.append((self._talker_step(s_sh, cur), cur,
                             decode_step_bytes(self.tk_shape, self.tk_layers, self.kv[cur])))
                self.kv[cur] += 1
                self.issued[cur] += 1
                self._poll()
        torch.cuda.synchronize()
        for i in batch:
            self.waiting.remove(i)
            if self.reqs[i].long:
                self.active.append(i)
            else:
                self.first[i] = self.start.elapsed_time(p_end)
        down_ids = sorted({int(i) for _, ids, _ in pend for i in ids})
        for e, ids, _ in pend:
            for i in ids:
                self.done_steps[i] += 1
                if self.done_steps[i] >= cfg.first_chunk and np.isnan(self.first[i]):
                    self.first[i] = self.start.elapsed_time(e)
        self.active = [i for i in self.active if np.isnan(self.first[i])]
        # B(k + 1): the downstream traffic of this step's decode steps over their GPU time.
        if cfg.pressure == "traffic":
            if pend:
                nbytes = sum(b for _, _, b in pend)
                dt = t_down0.elapsed_time(pend[-1][0])
                self._sample = nbytes / max(dt, 1e-3) / PEAK_HBM_BYTES_PER_MS
            else:
                self._sample = 0.0
        else:
            self._sample = float(np.mean(self._polls)) if self._polls else binding.hs_pressure_sample(0)
            self._polls = []
        rec = StepRecord(self.k, now, waiting, views, visible, info or {}, act, sample,
                         split, batch, tok, offsets, down_ids, len(pend), down_cus)
        self.records.append(rec)
        self.k += 1
        return rec

    def run(self, max_steps: int = 1000) -> Dict[str, object]:
        self.begin()
        for _ in range(max_steps):
            if self.step() is None:
                break
        return self.summary()

    def summary(self) -> Dict[str, object]:
        reqs = self.reqs
        arrival = np.array([r.arrival for r in reqs])
        deadline = np.array([r.deadline for r in reqs])
        long = np.array([r.long for r in reqs])
        shares = [r.split["shared_cus"] for r in self.records]
        out = {"policy": self.cfg.policy, "n_requests": len(reqs), "steps": len(self.records),
               "mean_shared_cus": round(float(np.mean(shares)), 1) if shares else None,
               "makespan_ms": round(float(np.nanmax(self.first)), 2) if np.any(~np.isnan(self.first)) else None,
               "unfinished": int(np.isnan(self.first).sum())}
        resp = self.first - arrival
        for name, flag in (("short", False), ("long", True)):
            lat = resp[long == flag]
            lat = lat[~np.isnan(lat)]
            met = self.first[long == flag] <= deadline[long == flag]
            out[name] = {"n": int((long == flag).sum()), "slo_attainment": round(float(met.mean()), 4),
                         "p50_ms": round(float(np.percentile(lat, 50)), 2) if len(lat) else None,
                         "p95_ms": round(float(np.percentile(lat, 95)), 2) if len(lat) else None}
        out["trace"] = [{"k": r.k, "now_ms": round(r.now, 2), "waiting": len(r.waiting),
                         "phase": r.info.get("phase"), "n": r.info.get("n"), "protected": r.info.get("n_protected"),
                         "batch_tokens": r.batch_tokens, "active": r.active, "sample": round(r.sample, 4),
                         "b_hat": round(r.split["pressure"], 4), "shared_cus": r.split["shared_cus"],
                         "down_steps": r.down_steps} for r in self.records]
        return out

    def close(self):
        if self.sched is not None:
            self.sched.close()
        if self.ctrl is not None:
            self.ctrl.close()


def make_requests(n: int, seed: int, load: float, per_token_ms: float, talker_step_ms: float, first_chunk: int,
                  tokens_lo: int = 256, tokens_hi: int = 1024, kv_lo: int = 128, kv_hi: int = 512,
                  p_long: float = 0.5, m_c: float = 5.0, burst: bool = False) -> List[Request]:
    """Seeded requests: prompts U{tokens_lo..tokens_hi}, a p_long share of long-path
    requests with kv0 U{kv_lo..kv_hi} cached downstream rows, Poisson arrivals at
    `load` times the shared stage's capacity (per_token_ms at the full chip), or all
    at t = 0 with burst.  Deadlines follow §4.2: arrival + m_c x the class's p95 solo
    first-response time."""
    rng = np.random.default_rng(seed)
    tokens = rng.integers(tokens_lo, tokens_hi, size=n, endpoint=True).astype(int)
    long = rng.uniform(size=n) < p_long
    kv0 = rng.integers(kv_lo, kv_hi, size=n, endpoint=True).astype(int)
    if burst:
        arrival = np.zeros(n)
    else:
        arrival = np.cumsum(rng.exponential(float(np.mean(tokens)) * per_token_ms / load, size=n))
    solo = tokens * per_token_ms + np.where(long, first_chunk * talker_step_ms, 0.0)
    delta = {c: m_c * float(np.percentile(solo[long == c], 95)) if np.any(long == c) else 0.0 for c in (False, True)}
    return [Request(i, float(arrival[i]), int(tokens[i]), bool(long[i]), int(kv0[i]),
                    float(arrival[i] + delta[bool(long[i])]), float(solo[i])) for i in range(n)]
