"""The decode step replayed from a captured graph, against the eager step and the reference.

Both paths run the same kernels on the same inputs, so every replay's output and
every cache byte it writes must equal the eager step's bit for bit; the first
step is also checked against the float64 reference.
"""
import numpy as np
import pytest

from oracle import layer as ref
from paper_2608_01785_amd import workloads as W
from tests.gpu_common import TOL, err_ratio, log, require_gpu
from tests.util import f64, h64, weights_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    ctx = binding.Context(0, budgets=(64, 128, 160))
    yield torch, ctx
    torch.cuda.synchronize()
    ctx.close()


def _caches(shape, n_layers, batch, kv_lens, max_ctx, seed, paged_table=None, page=None):
    """Two device caches (eager, graph) holding the same seeded prefix rows."""
    from paper_2608_01785_amd.device_data import DeviceCache, PagedCache
    prefix = W.make_cache(shape, n_layers, kv_lens, seed=seed)
    out = []
    for _ in range(2):
        if paged_table is None:
            c = DeviceCache(n_layers, batch, max_ctx, shape.n_kv_heads, shape.head_dim, fill=0.0)
        else:
            c = PagedCache(n_layers, int(paged_table.max()) + 1, page, shape.n_kv_heads, shape.head_dim,
                           paged_table, fill=0.0)
        for l in range(n_layers):
            for b in range(batch):
                c.load_prefix(l, b, prefix.k[l][b], prefix.v[l][b])
        out.append(c)
    return prefix, out


def _run_steps(env, shape, n_layers, batch, kv0, caches, budget, n_steps, table=None, prefix=None, layers=None,
               wdev=None):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import to_device
    eager, graphed = caches
    max_pos = int(kv0.max()) + n_steps
    if table is None:
        ws_e = torch.empty(binding.hs_workspace_size(shape, batch, batch, max_pos), dtype=torch.uint8, device="cuda")
        ws_g = torch.empty(binding.hs_workspace_size(shape, batch, batch, graphed.max_ctx), dtype=torch.uint8,
                           device="cuda")
    else:
        cap = table.shape[1] * graphed.max_ctx
        ws_e = torch.empty(binding.hs_workspace_size_paged(shape, batch, batch, cap, graphed.max_ctx),
                           dtype=torch.uint8, device="cuda")
        ws_g = torch.empty_like(ws_e)
    xe = torch.empty((batch, shape.hidden), dtype=torch.bfloat16, device="cuda")
    xg = torch.empty_like(xe)
    ye = torch.empty((batch, shape.hidden), dtype=torch.float32, device="cuda")
    yg = torch.empty_like(ye)
    torch.cuda.synchronize()
    graph = binding.DecodeGraph(ctx, shape, wdev, xg, yg, graphed.as_arg(), batch, budget, None, ws_g)
    kv = kv0.copy()
    try:
        for step in range(n_steps):
            x = W.token_rows(700 + step, batch, shape.hidden)
            xd = to_device(x)
            xe.copy_(xd)
            xg.copy_(xd)
            log(f"  step {step}: kv_lens {kv.min()}..{kv.max()}")
            binding.hs_downstream_decode_step(ctx, shape, wdev, xe, ye, eager.as_arg(), kv, budget, None, ws_e)
            graph.launch(kv, table)
            torch.cuda.synchronize()
            assert torch.equal(ye, yg), f"step {step}: graph output differs from the eager step"
            if step == 0 and prefix is not None:
                expect, _ = ref.decode_step(f64(x), weights_f64(layers), shape, kv,
                                            [[h64(k) for k in prefix.k[l]] for l in range(n_layers)],
                                            [[h64(v) for v in prefix.v[l]] for l in range(n_layers)])
                e = err_ratio(ye.cpu().numpy(), expect)
                log(f"  step 0 max err / rms = {e:.3e}")
                assert e <= TOL
            kv += 1
    finally:
        graph.close()
    for l in range(n_layers):
        assert torch.equal(eager.k[l], graphed.k[l]) and torch.equal(eager.v[l], graphed.v[l]), f"layer {l} cache"


@pytest.mark.parametrize("batch,budget", [(40, 128), (128, 160)])
def test_graph_replays_equal_eager_steps(env, batch, budget):
    """Three replays of one graph with growing caches, including a row whose key
    range crosses the single-row attention split (1024 keys at head_dim 64), so
    the number of attention work items changes between replays."""
    torch, ctx = env
    from paper_2608_01785_amd.device_data import prepare_f16, upload_weights
    shape, n_layers = W.TALKER, 4
    rng = np.random.default_rng(50 + batch)
    kv0 = rng.integers(1, 1000, size=batch).astype(np.int32)
    kv0[0] = 1022   # 1023, 1024, 1025 keys over the three steps: one work item, then two
    kv0[1] = 0      # an empty prefix
    layers = W.make_weights(shape, n_layers, 51)
    wdev = prepare_f16(ctx, upload_weights(layers))
    prefix, caches = _caches(shape, n_layers, batch, kv0, 1088, seed=52)
    log(f"[graph] talker {n_layers} layers, batch {batch}, {256 - budget} shared CUs / {budget} down")
    _run_steps(env, shape, n_layers, batch, kv0, caches, 256 - budget, 3, prefix=prefix, layers=layers, wdev=wdev)


def test_graph_on_a_paged_cache(env):
    """Pages of 256 positions in a shuffled pool; every launch takes the step's table."""
    torch, ctx = env
    from paper_2608_01785_amd.device_data import upload_weights
    shape, n_layers, batch, page, pps = W.TALKER, 3, 24, 256, 5
    rng = np.random.default_rng(60)
    kv0 = rng.integers(1, 1200, size=batch).astype(np.int32)
    kv0[0] = 1277   # the new rows reach the last position of the last page
    table = rng.permutation(batch * pps).astype(np.int32).reshape(batch, pps)
    layers = W.make_weights(shape, n_layers, 61)
    wdev = upload_weights(layers)
    prefix, caches = _caches(shape, n_layers, batch, kv0, None, seed=62, paged_table=table, page=page)
    log(f"[graph] paged talker, {n_layers} layers, batch {batch}, pages of {page}")
    _run_steps(env, shape, n_layers, batch, kv0, caches, 128, 3, table=table, prefix=prefix, layers=layers,
               wdev=wdev)


def test_graph_launch_refuses_rows_beyond_its_capacity(env):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, upload_weights
    shape, batch = W.TALKER, 8
    wdev = upload_weights(W.make_weights(shape, 1, 71))
    cache = DeviceCache(1, batch, 128, shape.n_kv_heads, shape.head_dim, fill=0.0)
    ws = torch.empty(binding.hs_workspace_size(shape, batch, batch, 128), dtype=torch.uint8, device="cuda")
    x = torch.zeros((batch, shape.hidden), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((batch, shape.hidden), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    g = binding.DecodeGraph(ctx, shape, wdev, x, y, cache.as_arg(), batch, 128, None, ws)
    try:
        with pytest.raises(binding.HorizonError):
            g.launch(np.full(batch, 127, np.int32))       # row 127 would sit at position 127 < 128: fine ...
            torch.cuda.synchronize()
            g.launch(np.full(batch, 128, np.int32))       # ... position 128 is outside the slots
        with pytest.raises(binding.HorizonError):
            g.launch(np.zeros(batch, np.int32), np.zeros((batch, 1), np.int32))  # no table for slot caches
        torch.cuda.synchronize()
    finally:
        g.close()
