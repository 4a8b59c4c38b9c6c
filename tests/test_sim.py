"""The serving-loop model: structure checks on a synthetic timing table (CPU only).

The model's outputs are not measurements; these tests check that it runs the
library's policies and keeps its own invariants: every request gets a first
response after it arrives, a lone request meets its deadline, the baseline
never throttles, and more load never improves attainment.
"""
import pytest

from paper_2608_01785_amd import sim


def timing():
    return sim.Timing(prefill_ms_per_token={64: 0.0050, 128: 0.0027, 192: 0.0021, 256: 0.0019},
                      decode_ms_per_step={64: 1.6, 128: 0.90, 160: 0.80, 192: 0.75, 224: 0.72, 240: 0.71},
                      decode_batch=32, weight_share=0.32, masked_prefill_factor=1.14, masked_decode_factor=1.14,
                      unmasked_prefill_factor=1.3, unmasked_decode_factor=1.8, decode_full_ms=0.70, hbm_share=0.41)


@pytest.fixture(scope="module")
def lib():
    from paper_2608_01785_amd import binding
    binding.lib()


@pytest.mark.parametrize("policy", ["baseline", "temporal", "spatial", "joint"])
def test_every_request_gets_a_first_response(lib, policy):
    w = sim.Workload(n_requests=120, rate_per_s=30.0)
    out = sim.simulate(policy, timing(), w)
    assert out["short"]["n"] + out["long"]["n"] == 120
    for cls in ("short", "long"):
        assert out[cls]["p50_ms"] > 0 and out[cls]["p95_ms"] >= out[cls]["p50_ms"]
        assert 0.0 <= out[cls]["slo_attainment"] <= 1.0
    if policy in ("baseline", "temporal"):
        assert out["mean_shared_cus"] == 256.0
    else:
        assert 64 <= out["mean_shared_cus"] <= 256


def test_light_load_meets_every_deadline(lib):
    w = sim.Workload(n_requests=40, rate_per_s=0.5)
    for out in sim.compare(timing(), w):
        assert out["short"]["slo_attainment"] == 1.0 and out["long"]["slo_attainment"] == 1.0


def test_more_load_never_helps(lib):
    t = timing()
    lo = sim.simulate("joint", t, sim.Workload(n_requests=200, rate_per_s=5.0))
    hi = sim.simulate("joint", t, sim.Workload(n_requests=200, rate_per_s=80.0))
    assert hi["short"]["p95_ms"] >= lo["short"]["p95_ms"]
    assert hi["short"]["slo_attainment"] <= lo["short"]["slo_attainment"]


def test_deadlines_follow_the_solo_p95_rule():
    t, w = timing(), sim.Workload(n_requests=50)
    reqs = sim.make_requests(w)
    delta = sim.assign_deadlines(reqs, t, w, 256)
    import numpy as np
    short = [t.prefill_ms(r.tokens, 256) for r in reqs if not r.long]
    assert delta["short"] == pytest.approx(5.0 * float(np.percentile(short, 95)))
    assert all(r.deadline - r.arrival == pytest.approx(delta["long" if r.long else "short"]) for r in reqs)
