"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times, through the C ABI.

Every output row is compared element by element with the float64 reference:
* the 4-layer thinker stack over all 10,515 rows (sequences never see each
  other, so the reference runs request by request);
* the 4096-wide mixed step (four 2048-row chunks behind up to 6,144 cached
  rows, 64 decode rows) and its cache rows;
* the talker step at batch 32 (128 CUs) and batch 128 (the 160-CU downstream
  stream);
* the thinker's decode rows behind 1-2k cached rows (seven query heads per
  key/value head).
Properties that hold at any size are checked as well: bit-identical results
across CU budgets, and a co-running decode stage that changes nothing.
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
    ctx = binding.Context(0, budgets=(64, 96, 128, 192, 256))
    yield torch, ctx
    torch.cuda.synchronize()
    ctx.close()


@pytest.fixture(scope="module")
def thinker(env):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import prepare_f16, to_device, upload_weights
    log("[thinker] generating 4-layer weights and the 8-request batch")
    layers = W.make_weights(W.THINKER, 4, W.SEEDS["thinker"]["weights"])
    batch = W.thinker_batch()
    wdev = prepare_f16(ctx, upload_weights(layers))
    x = to_device(batch.x)
    ws = torch.empty(binding.hs_workspace_size(W.THINKER, batch.n_tokens, batch.n_seqs, int(batch.lengths.max())),
                     dtype=torch.uint8, device="cuda")
    return layers, batch, wdev, x, ws


def run_thinker(env, thinker, budget, stream=None):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    layers, batch, wdev, x, ws = thinker
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    binding.hs_shared_stage_forward(ctx, W.THINKER, wdev, x, y, batch.seq_offsets, None, None, budget, stream, ws)
    return y


def test_thinker_stack_every_row(env, thinker):
    """All 10,515 rows of the 4-layer launch at 256 CUs against the reference,
    element by element.  Sequences never see each other, so the reference runs
    request by request; the longest request (1,901 rows, keys up to position
    1,900) is one of them."""
    torch, _ = env
    layers, batch, _, _, _ = thinker
    log("[thinker] full stack at 256 CUs")
    y = run_thinker(env, thinker, 256)
    torch.cuda.synchronize()
    got = y.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    w64 = weights_f64(layers)
    off = batch.seq_offsets
    assert int(np.max(np.diff(off))) == 1901
    worst = 0.0
    for b in range(batch.n_seqs):
        lo, hi = int(off[b]), int(off[b + 1])
        exp, _ = ref.stack_forward(f64(batch.x[lo:hi]), w64, W.THINKER, [0, hi - lo])
        e = err_ratio(got[lo:hi], exp)
        log(f"  request {b} ({hi - lo} rows): max err / rms = {e:.3e}")
        assert e <= TOL, (b, e)
        worst = max(worst, e)
    log(f"  every row: worst max err / rms = {worst:.3e}")


def test_thinker_budgets_bit_identical(env, thinker):
    torch, _ = env
    outs = {}
    for b in (256, 192, 128, 64):
        log(f"[thinker] budget {b}")
        outs[b] = run_thinker(env, thinker, b)
        torch.cuda.synchronize()
    for b in (192, 128, 64):
        assert torch.equal(outs[b], outs[256]), f"budget {b} differs from 256"


def test_thinker_bf16_weights_match_prepared(env, thinker):
    """Weights converted inside each GEMM give the same bits as prepared fp16 copies."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import upload_weights
    layers, batch, wdev, x, ws = thinker
    y_f16 = run_thinker(env, thinker, 256)
    wb = upload_weights(layers)
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    log("[thinker] bf16 weights, converted in the GEMM")
    binding.hs_shared_stage_forward(ctx, W.THINKER, wb, x, y, batch.seq_offsets, None, None, 256, None, ws)
    torch.cuda.synchronize()
    assert torch.equal(y, y_f16)


def talker_setup(env, batch, seeds, n_layers=16):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, prepare_f16, to_device, upload_weights
    shape = W.TALKER
    layers = W.make_weights(shape, n_layers, seeds["weights"])
    d = W.talker_batch(shape, n_layers, batch, seeds)
    max_ctx = int(np.ceil((d.kv_lens.max() + 1) / 64) * 64)
    cache = DeviceCache(n_layers, batch, max_ctx, shape.n_kv_heads, shape.head_dim, fill=0.0)
    for l in range(n_layers):
        for b in range(batch):
            cache.load_prefix(l, b, d.cache.k[l][b], d.cache.v[l][b])
    wdev = prepare_f16(ctx, upload_weights(layers))
    ws = torch.empty(binding.hs_workspace_size(shape, batch, batch, int(d.kv_lens.max()) + 1), dtype=torch.uint8,
                     device="cuda")
    return layers, d, cache, wdev, to_device(d.x), ws


def test_talker_decode_step_full(env):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    shape, n_layers, batch = W.TALKER, 16, 32
    log("[talker] 16 layers, batch 32, seeded cache")
    layers, d, cache, wdev, x, ws = talker_setup(env, batch, W.SEEDS["talker"])
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    binding.hs_downstream_decode_step(ctx, shape, wdev, x, y, cache.as_arg(), d.kv_lens, 128, None, ws)
    torch.cuda.synchronize()
    expect, kv_new = ref.decode_step(f64(d.x), weights_f64(layers), shape, d.kv_lens,
                                     [[h64(k) for k in d.cache.k[l]] for l in range(n_layers)],
                                     [[h64(v) for v in d.cache.v[l]] for l in range(n_layers)])
    e = err_ratio(y.cpu().numpy(), expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    for l in (0, 7, 15):
        kn = np.stack([h64(cache.rows(l, b, int(d.kv_lens[b]), int(d.kv_lens[b]) + 1)[0][0]) for b in range(batch)])
        vn = np.stack([h64(cache.rows(l, b, int(d.kv_lens[b]), int(d.kv_lens[b]) + 1)[1][0]) for b in range(batch)])
        assert err_ratio(kn, kv_new[l][0]) <= TOL
        assert err_ratio(vn, kv_new[l][1]) <= TOL


def test_thinker_mixed_step_every_row(env):
    """One layer at hidden 4096: four 2048-row chunks behind 0/2048/4096/6144 cached
    rows and 64 single-row sequences behind 4096 cached rows, at 96 CUs.  Every
    row against the reference (the last chunk's rows sit at positions
    6,144-8,191), and the new cache rows of every sequence."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, prepare_f16, to_device, upload_weights
    shape = W.THINKER_MIXED
    seeds = W.SEEDS["thinker_mixed"]
    lengths, ctx_lens = W.thinker_mixed_layout()
    layers = W.make_weights(shape, 1, seeds["weights"])
    batch = W.random_batch(shape.hidden, lengths, seeds["tokens"], ctx_lens)
    log("[mixed] generating prefix caches")
    prefix = W.make_cache(shape, 1, ctx_lens, seeds["cache"])
    B = len(lengths)
    cache = DeviceCache(1, B, 8192, shape.n_kv_heads, shape.head_dim, fill=0.0)
    for b in range(B):
        cache.load_prefix(0, b, prefix.k[0][b], prefix.v[0][b])
    wdev = prepare_f16(ctx, upload_weights(layers))
    x = to_device(batch.x)
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    ws = torch.empty(binding.hs_workspace_size(shape, batch.n_tokens, B, 8192), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    log("[mixed] layer at 96 CUs")
    binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, batch.seq_offsets, ctx_lens, cache.as_arg(), 96, None, ws)
    torch.cuda.synchronize()
    got = y.cpu().numpy().astype(np.float64)
    off = batch.seq_offsets
    w64 = weights_f64(layers)[0]
    log("[mixed] reference, every row")
    exp, k_new, v_new = ref.layer_forward(f64(batch.x), w64, shape, off, [int(c) for c in ctx_lens],
                                          [h64(k) for k in prefix.k[0]], [h64(v) for v in prefix.v[0]])
    for b in range(4):
        e = err_ratio(got[off[b]:off[b + 1]], exp[off[b]:off[b + 1]])
        log(f"  chunk {b} (positions {ctx_lens[b]}..{ctx_lens[b] + lengths[b] - 1}): max err / rms = {e:.3e}")
        assert e <= TOL, (b, e)
    e = err_ratio(got[off[4]:], exp[off[4]:])
    log(f"  64 decode rows: max err / rms = {e:.3e}")
    assert e <= TOL
    # The new rows in the cache, at positions ctx .. ctx + len - 1 of each sequence.
    kc = np.concatenate([h64(cache.rows(0, b, int(ctx_lens[b]), int(ctx_lens[b] + lengths[b]))[0]) for b in range(B)])
    vc = np.concatenate([h64(cache.rows(0, b, int(ctx_lens[b]), int(ctx_lens[b] + lengths[b]))[1]) for b in range(B)])
    assert err_ratio(kc, k_new) <= TOL
    assert err_ratio(vc, v_new) <= TOL


class _LazyLayers:
    """Per-layer lists of float64 cache prefixes, converted when the reference reaches the layer
    (a whole 16-layer cache in float64 would take tens of GB)."""

    def __init__(self, per_layer):
        self.per_layer = per_layer

    def __getitem__(self, layer):
        return [h64(a) for a in self.per_layer[layer]]


def test_talker_batch128_on_the_160_cu_down_stream(env):
    """The downstream-heavy talker: 16 layers, batch 128, cached lengths in
    [128, 1024], on the DOWN stream of the 96-CU level (160 CUs)."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    shape, n_layers, batch = W.TALKER, 16, 128
    log("[talker-128] 16 layers, batch 128, seeded cache")
    layers, d, cache, wdev, x, ws = talker_setup(env, batch, W.SEEDS["talker_mixed"], n_layers)
    assert int(d.kv_lens.sum()) == 75820 and int(d.kv_lens.max()) <= 1024
    s_dn = binding.hs_context_stream(ctx, 96, binding.HS_ROLE_DOWN)
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    binding.hs_downstream_decode_step(ctx, shape, wdev, x, y, cache.as_arg(), d.kv_lens, 160, s_dn, ws)
    torch.cuda.synchronize()
    log("[talker-128] reference")
    expect, kv_new = ref.decode_step(f64(d.x), weights_f64(layers), shape, d.kv_lens,
                                     _LazyLayers(d.cache.k), _LazyLayers(d.cache.v))
    e = err_ratio(y.cpu().numpy(), expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    for l in (0, 8, 15):
        kn = np.stack([h64(cache.rows(l, b, int(d.kv_lens[b]), int(d.kv_lens[b]) + 1)[0][0]) for b in range(batch)])
        vn = np.stack([h64(cache.rows(l, b, int(d.kv_lens[b]), int(d.kv_lens[b]) + 1)[1][0]) for b in range(batch)])
        assert err_ratio(kn, kv_new[l][0]) <= TOL
        assert err_ratio(vn, kv_new[l][1]) <= TOL


def test_thinker_decode_rows_behind_long_prefixes(env, thinker):
    """The thinker stack's decode step (seven query heads per key/value head):
    one row for each of 16 sequences behind 1,024-2,048 cached rows, the
    workload of the decode-TPOT sweep, at caps 64/96/192/256.  Parity against
    the reference, and the same bits at every cap."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, to_device
    layers, _, wdev, _, _ = thinker
    shape, n_layers, nb = W.THINKER, 4, 16
    assert shape.n_q_heads // shape.n_kv_heads == 7
    ctx_lens = np.random.default_rng(5001).integers(1024, 2048, size=nb, endpoint=True).astype(np.int32)
    max_ctx = int(np.ceil((ctx_lens.max() + 1) / 64) * 64)
    log(f"[thinker-decode] caches behind {ctx_lens.min()}-{ctx_lens.max()} rows")
    pre = W.make_cache(shape, n_layers, ctx_lens, 5002)
    xb = W.token_rows(5003, nb, shape.hidden)
    outs = {}
    for cap in (256, 192, 96, 64):
        cache = DeviceCache(n_layers, nb, max_ctx, shape.n_kv_heads, shape.head_dim, fill=0.0)
        for l in range(n_layers):
            for b in range(nb):
                cache.load_prefix(l, b, pre.k[l][b], pre.v[l][b])
        x = to_device(xb)
        y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
        ws = torch.empty(binding.hs_workspace_size(shape, nb, nb, max_ctx), dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        log(f"[thinker-decode] cap {cap}")
        binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, list(range(nb + 1)), ctx_lens, cache.as_arg(), cap,
                                        None, ws)
        torch.cuda.synchronize()
        outs[cap] = (y.cpu().numpy(), cache.rows(3, nb - 1, int(ctx_lens[-1]), int(ctx_lens[-1]) + 1))
        del cache
    expect, kv_new = ref.decode_step(f64(xb), weights_f64(layers), shape, ctx_lens,
                                     _LazyLayers(pre.k), _LazyLayers(pre.v))
    e = err_ratio(outs[256][0], expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    assert err_ratio(h64(outs[256][1][0][0]), kv_new[3][0][nb - 1]) <= TOL
    for cap in (192, 96, 64):
        assert np.array_equal(outs[cap][0], outs[256][0]), f"cap {cap} differs from 256"


def test_corun_changes_nothing(env, thinker):
    """Prefill on a 128-CU mask with talker steps on the other 128 CUs: both
    outputs equal their solo runs bit for bit, and the two stages overlap."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    layers_t, d, cache, wdev_t, xt, ws_t = talker_setup(env, 32, W.SEEDS["talker"])
    kv0 = [c.clone() for c in cache.k] + [c.clone() for c in cache.v]
    yt_solo = torch.empty(xt.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    binding.hs_downstream_decode_step(ctx, W.TALKER, wdev_t, xt, yt_solo, cache.as_arg(), d.kv_lens, 128, None, ws_t)
    y_solo = run_thinker(env, thinker, 128)
    torch.cuda.synchronize()
    # The decode step rewrote the new rows with identical values; restore anyway.
    for i, c in enumerate(cache.k + cache.v):
        c.copy_(kv0[i])
    torch.cuda.synchronize()
    s_sh = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 128, binding.HS_ROLE_SHARED))
    s_dn = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 128, binding.HS_ROLE_DOWN))
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    yt = torch.empty_like(yt_solo)
    log("[co-run] prefill @128 + decode @128")
    _, batch, wdev, x, ws = thinker
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    ev[0].record(s_sh)
    binding.hs_shared_stage_forward(ctx, W.THINKER, wdev, x, y, batch.seq_offsets, None, None, 128, None, ws)
    ev[1].record(s_sh)
    s_dn.wait_event(ev[0])
    ev[2].record(s_dn)
    for _ in range(3):
        binding.hs_downstream_decode_step(ctx, W.TALKER, wdev_t, xt, yt, cache.as_arg(), d.kv_lens, 128, None, ws_t)
    ev[3].record(s_dn)
    torch.cuda.synchronize()
    assert torch.equal(y, y_solo)
    assert torch.equal(yt, yt_solo)
    t_pre = (ev[0].elapsed_time(ev[0]), ev[0].elapsed_time(ev[1]))
    t_dec = (ev[0].elapsed_time(ev[2]), ev[0].elapsed_time(ev[3]))
    log(f"  prefill window {t_pre}, decode window {t_dec} (ms from the common start)")
    assert t_dec[0] < t_pre[1], "decode did not start before the prefill ended"


def test_queued_prefill_never_blocks_decode_calls(env, thinker):
    """Several thinker forwards queued on the shared stream must not make a
    decode call on the downstream stream wait on the host (the calls' metadata
    staging must not serialise the two stages)."""
    import time
    torch, ctx = env
    from paper_2608_01785_amd import binding
    layers_t, d, cache, wdev_t, xt, ws_t = talker_setup(env, 32, W.SEEDS["talker"])
    _, batch, wdev, x, ws = thinker
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    yt = torch.empty(xt.shape, dtype=torch.float32, device="cuda")
    s_sh = torch.cuda.ExternalStream(binding.hs_context_stream(ctx, 128, binding.HS_ROLE_SHARED))
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s_sh)
    for _ in range(6):
        binding.hs_shared_stage_forward(ctx, W.THINKER, wdev, x, y, batch.seq_offsets, None, None, 128, None, ws)
    e1.record(s_sh)
    t0 = time.perf_counter()
    for _ in range(6):
        binding.hs_downstream_decode_step(ctx, W.TALKER, wdev_t, xt, yt, cache.as_arg(), d.kv_lens, 128, None, ws_t)
    host_ms = (time.perf_counter() - t0) * 1e3
    torch.cuda.synchronize()
    queued_ms = e0.elapsed_time(e1)
    log(f"  6 decode calls issued in {host_ms:.1f} ms on the host behind {queued_ms:.1f} ms of queued prefill")
    assert host_ms < queued_ms / 4
