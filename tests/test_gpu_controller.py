"""Spatial controller in the loop on the GPU (§4.4, Algorithm 1 steps 1 and 3).

Each step samples AMD SMI memory activity, asks the controller for the split
and runs a talker decode step on the downstream stream of the chosen ladder
level while the downstream stage is active.  Checks: every decision selects a
pre-built stream pair whose masks are complementary and hold the decided CU
counts; the decode output does not depend on the split (bit-identical to a
fixed-split run); the sampled activity is a fraction.
"""
import numpy as np
import pytest

from oracle.controller import SpatialController
from paper_2608_01785_amd import workloads as W
from tests.gpu_common import log, require_gpu, workspace

pytestmark = pytest.mark.gpu

LADDER = [64, 96, 128, 160, 192]
N_CUS = 256


def popcount(words):
    return sum(bin(int(w)).count("1") for w in words)


def test_pressure_sample_is_a_fraction():
    require_gpu()
    from paper_2608_01785_amd import binding
    try:
        v = binding.hs_pressure_sample(0)
    except binding.HorizonError as e:
        pytest.skip(f"AMD SMI memory activity unavailable on this box: {e}")
    log(f"[pressure] AMD SMI memory activity = {v}")
    assert 0.0 <= v <= 1.0


def test_pressure_tracks_the_hbm_rate_of_a_bandwidth_bound_load():
    """The sample follows this device's memory traffic.  AMD SMI's UMC activity
    is the firmware's average over its last interval, which it refreshes about
    once per second on MI355X, so the load (device-to-device copies, HBM-bound)
    runs for ~2.6 s and the host polls through it.  The reading under load must
    be well above the idle reading and close to the copies' measured HBM rate
    as a share of the 8 TB/s peak."""
    import time
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    try:
        binding.hs_pressure_sample(0)
    except binding.HorizonError as e:
        pytest.skip(f"AMD SMI memory activity unavailable on this box: {e}")
    torch.cuda.synchronize()
    idle = []
    for _ in range(12):                      # 1.2 s: at least one refresh of an idle device
        idle.append(binding.hs_pressure_sample(0))
        time.sleep(0.1)
    a = torch.empty(256 << 20, dtype=torch.float32, device="cuda")    # 1 GiB
    b = torch.empty_like(a)
    a.fill_(1.0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    n_copies = 6000
    e0.record()
    for _ in range(n_copies):
        b.copy_(a)
    e1.record()
    busy = []
    while not e1.query():
        busy.append(binding.hs_pressure_sample(0))
        time.sleep(0.05)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    share = n_copies * 2 * a.numel() * 4 / (ms / 1e3) / 8e12
    del a, b
    log(f"[pressure] idle max {max(idle):.3f}; {ms:.0f} ms of copies at {share * 8:.2f} TB/s ({share:.3f} of "
        f"8 TB/s): readings {sorted(set(round(v, 3) for v in busy))} over {len(busy)} polls")
    assert ms > 2000 and len(busy) >= 20
    top = max(busy)
    assert top > max(idle) + 0.25
    assert abs(top - share) <= 0.15


def test_controller_drives_the_ladder_with_decode_running():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, prepare_f16, to_device, upload_weights
    ctx = binding.Context(0, budgets=tuple(LADDER) + (N_CUS,))
    ctrl = binding.Controller(N_CUS, N_CUS, LADDER, 0.4, 0.5, 1)
    ref = SpatialController(N_CUS, N_CUS, LADDER, 0.4, 0.5, 1)
    try:
        shape, n_layers, batch = W.TALKER, 2, 16
        rng = np.random.default_rng(5)
        kv_lens = rng.integers(64, 500, size=batch).astype(np.int32)
        layers = W.make_weights(shape, n_layers, 77)
        wdev = prepare_f16(ctx, upload_weights(layers))
        cache = DeviceCache(n_layers, batch, 512, shape.n_kv_heads, shape.head_dim, fill=0.0)
        prefix = W.make_cache(shape, n_layers, kv_lens, seed=78)
        for l in range(n_layers):
            for b in range(batch):
                cache.load_prefix(l, b, prefix.k[l][b], prefix.v[l][b])
        x = to_device(W.token_rows(79, batch, shape.hidden))
        ws = workspace(torch, shape, batch, batch, int(kv_lens.max()) + 1)
        y_fixed = torch.empty(x.shape, dtype=torch.float32, device="cuda")
        binding.hs_downstream_decode_step(ctx, shape, wdev, x, y_fixed, cache.as_arg(), kv_lens, 128, None, ws)
        torch.cuda.synchronize()

        try:
            binding.hs_pressure_sample(0)
            sampled = True
        except binding.HorizonError:
            sampled = False
        # Downstream idle, active, idle; the seeded fallback samples sweep the ladder.
        active = [0] * 3 + [1] * 18 + [0] * 3
        fallback = np.linspace(0.0, 1.0, len(active))
        y = torch.empty_like(y_fixed)
        seen = set()
        for k, a in enumerate(active):
            sample = binding.hs_pressure_sample(0) if sampled else float(fallback[k])
            sp = binding.hs_controller_step(ctrl, bool(a), sample)
            r = ref.step(bool(a), sample)
            assert (sp.shared_cus, sp.down_cus, sp.level) == (r.shared, r.down, r.level)
            sh, dn = binding.hs_context_masks(ctx, sp.shared_cus)
            assert popcount(sh) == sp.shared_cus and popcount(dn) == sp.down_cus
            assert all((int(a_) & int(b_)) == 0 for a_, b_ in zip(sh, dn))
            binding.hs_context_stream(ctx, sp.shared_cus, binding.HS_ROLE_SHARED)
            if a:
                assert sp.shared_cus in LADDER
                binding.hs_downstream_decode_step(ctx, shape, wdev, x, y, cache.as_arg(), kv_lens, sp.down_cus,
                                                  None, ws)
                torch.cuda.synchronize()
                assert torch.equal(y, y_fixed)
            else:
                assert sp.shared_cus == N_CUS and sp.down_cus == 0
            seen.add(sp.shared_cus)
        log(f"[controller] sampled={sampled} caps used: {sorted(seen)}")
        if not sampled:
            assert len(seen) >= 3
    finally:
        torch.cuda.synchronize()
        ctrl.close()
        ctx.close()
