"""Algorithm 1 on the GPU: every scheduling step checked against the reference policies.

Each step of the serving loop runs the library's temporal view, its controller
split and a real shared-stage forward on the chosen CU-masked stream, with
downstream decode steps on the complement.  The test replays each step's
inputs through the reference temporal scheduler and spatial controller and
checks the view, the split and the base scheduler's batch against them, and
checks the prefill output of every step against the float64 reference layer.
"""
import numpy as np
import pytest

from oracle import layer as ref
from oracle.controller import SpatialController
from oracle.temporal import Request as RefRequest, TemporalScheduler
from paper_2608_01785_amd import workloads as W
from tests.gpu_common import TOL, err_ratio, log, require_gpu
from tests.util import f64, weights_f64

pytestmark = pytest.mark.gpu

LADDER = (128, 160, 192, 224)


@pytest.fixture(scope="module")
def env():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    ctx = binding.Context(0, budgets=LADDER + (256,))
    yield torch, ctx
    torch.cuda.synchronize()
    ctx.close()


def _loop(env, policy, n_req=12, seed=3, **kw):
    torch, ctx = env
    from paper_2608_01785_amd import serving
    from paper_2608_01785_amd.device_data import to_device, upload_weights
    th, tk = W.TINY, W.TINY
    th_layers = W.make_weights(th, 2, 81)
    tk_layers = W.make_weights(tk, 2, 82)
    cfg = serving.LoopConfig(policy=policy, token_budget=512, short_budget=256, first_chunk=3, ladder=LADDER,
                             saturation=0.25, **kw)
    reqs = serving.make_requests(n_req, seed, load=1.0, per_token_ms=0.002, talker_step_ms=0.3,
                                 first_chunk=cfg.first_chunk, tokens_lo=64, tokens_hi=256, kv_lo=64, kv_hi=200,
                                 burst=True)
    x_bits = W.token_rows(83, cfg.token_budget, th.hidden)
    loop = serving.Algorithm1(ctx, (th, upload_weights(th_layers), 2), (tk, upload_weights(tk_layers), 2), reqs,
                              to_device(x_bits), cfg, max_ctx=256)
    return loop, reqs, x_bits, th_layers


def test_algorithm1_steps_match_the_reference_policies(env):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    loop, reqs, x_bits, th_layers = _loop(env, "joint")
    cfg = loop.cfg
    sched = TemporalScheduler(cfg.n_min, cfg.n_max, cfg.m, cfg.u_guard, cfg.long_cap)
    ctrl = SpatialController(256, 256, LADDER, cfg.ewma, cfg.saturation, cfg.hysteresis)
    w64 = weights_f64(th_layers)
    x64 = f64(x_bits)
    loop.begin()
    seen_shared, n_steps = set(), 0
    try:
        while True:
            rec = loop.step()
            if rec is None:
                break
            n_steps += 1
            assert n_steps < 200, "the loop did not finish"
            log(f"[algorithm 1] step {rec.k}: waiting {len(rec.waiting)} phase {rec.info.get('phase')} "
                f"batch {rec.batch_tokens} tokens, active {rec.active}, sample {rec.sample:.3f}, "
                f"shared {rec.split['shared_cus']} CUs, {rec.down_steps} downstream steps")
            # Step 2: the view, against the reference scheduler fed the same queue.
            if rec.waiting:
                vis, info = sched.step(rec.now, [RefRequest(p, w_, d, r) for p, w_, d, r in rec.views])
                assert list(rec.visible) == list(vis)
                assert (rec.info["n"], rec.info["phase"], rec.info["n_protected"], rec.info["n_hidden"],
                        rec.info["n_capped"]) == (info.n, info.phase, info.n_protected, info.n_hidden,
                                                  info.n_capped)
            # Step 3: the split, against the reference controller fed the same sample.
            d = ctrl.step(rec.active, rec.sample)
            assert (rec.split["shared_cus"], rec.split["down_cus"], rec.split["level"]) == (d.shared, d.down, d.level)
            assert abs(rec.split["pressure"] - d.pressure) <= 1e-12
            if rec.active:
                assert rec.split["shared_cus"] in LADDER
            seen_shared.add(rec.split["shared_cus"])
            if rec.down_steps:
                assert rec.down_cus == 256 - rec.split["shared_cus"]
                assert 0.0 <= loop._sample <= 1.0
            # Step 4: first come, first served over the visible prefills within the step's budget.
            budget = cfg.token_budget
            if rec.info and rec.info["phase"] == binding.HS_PATH_SHORT:
                budget = cfg.short_budget
            expect, tok = [], 0
            for i, v in zip(rec.waiting, rec.visible):
                if v and (not expect or tok + reqs[i].tokens <= budget):
                    expect.append(i)
                    tok += reqs[i].tokens
            assert rec.batch == expect and rec.batch_tokens == tok
            # The forward that ran on the chosen stream, against the reference layer stack.
            if rec.batch:
                got = loop.y[:tok].cpu().numpy().astype(np.float64)
                want, _ = ref.stack_forward(x64[:tok], w64, W.TINY, rec.offsets)
                e = err_ratio(got, want)
                assert e <= TOL, (rec.k, e)
        s = loop.summary()
    finally:
        loop.close()
    log(f"[algorithm 1] {n_steps} steps, caps used {sorted(seen_shared)}, short p95 {s['short']['p95_ms']} ms, "
        f"long p95 {s['long']['p95_ms']} ms")
    assert s["unfinished"] == 0
    assert 256 in seen_shared and len(seen_shared & set(LADDER)) >= 1


def test_baseline_policy_shows_everything_unmasked(env):
    torch, ctx = env
    loop, reqs, x_bits, th_layers = _loop(env, "baseline", n_req=6, seed=4)
    loop.begin()
    try:
        for _ in range(100):
            rec = loop.step()
            if rec is None:
                break
            assert all(rec.visible) and rec.split["shared_cus"] == 256
            if rec.down_steps:
                assert rec.down_cus == 256
        s = loop.summary()
    finally:
        loop.close()
    assert s["unfinished"] == 0


def test_memory_activity_signal_drives_the_loop(env):
    """The AMD SMI reading as the pressure signal: polled while downstream steps
    are in flight; the controller receives it unchanged."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    try:
        binding.hs_pressure_sample(0)
    except binding.HorizonError as e:
        pytest.skip(f"AMD SMI reading unavailable: {e}")
    loop, reqs, x_bits, th_layers = _loop(env, "joint", n_req=6, seed=5, pressure="amdsmi")
    ctrl = SpatialController(256, 256, LADDER, loop.cfg.ewma, loop.cfg.saturation, loop.cfg.hysteresis)
    loop.begin()
    try:
        for _ in range(100):
            rec = loop.step()
            if rec is None:
                break
            assert 0.0 <= rec.sample <= 1.0
            d = ctrl.step(rec.active, rec.sample)
            assert rec.split["shared_cus"] == d.shared
    finally:
        loop.close()
