"""The no-allocation decode step against the workspace decode step, through the
C ABI: two calls in a row (the second with a smaller batch and shorter caches),
each checked bit for bit against hs_downstream_decode_step on the same inputs,
output and cache rows; oversized requests are refused before any GPU work."""
import ctypes

import numpy as np
import pytest

from paper_2608_01785_amd import workloads as W
from tests.gpu_common import log, require_gpu, workspace

pytestmark = pytest.mark.gpu


def _case(torch, binding, ctx, shape, layers, wdev, batch, seed, lo, hi):
    from paper_2608_01785_amd.device_data import DeviceCache, to_device
    n_layers = len(layers)
    kv_lens = np.random.default_rng(seed).integers(lo, hi, size=batch, endpoint=True).astype(np.int32)
    max_ctx = int(np.ceil((kv_lens.max() + 1) / 64) * 64)
    prefix = W.make_cache(shape, n_layers, kv_lens, seed + 1)
    caches = []
    for _ in range(2):
        c = DeviceCache(n_layers, batch, max_ctx, shape.n_kv_heads, shape.head_dim, fill=0.0)
        for l in range(n_layers):
            for b in range(batch):
                c.load_prefix(l, b, prefix.k[l][b], prefix.v[l][b])
        caches.append(c)
    x = to_device(W.token_rows(seed + 2, batch, shape.hidden))
    y_ref = torch.empty((batch, shape.hidden), dtype=torch.float32, device="cuda")
    y = torch.full_like(y_ref, float("nan"))
    ws = workspace(torch, shape, batch, batch, int(kv_lens.max()) + 1)
    torch.cuda.synchronize()
    log(f"[no-alloc] batch {batch}, cached rows {kv_lens.min()}-{kv_lens.max()}")
    binding.hs_downstream_decode_step(ctx, shape, wdev, x, y_ref, caches[0].as_arg(), kv_lens, 128, None, ws)
    binding.hs_downstream_decode_step_noalloc(ctx, shape, wdev, x, y, caches[1].as_arg(), kv_lens, 128)
    torch.cuda.synchronize()
    assert torch.equal(y, y_ref)
    for l in range(n_layers):
        assert torch.equal(caches[0].k[l], caches[1].k[l]), l
        assert torch.equal(caches[0].v[l], caches[1].v[l]), l


def test_noalloc_decode_step_matches_the_workspace_call():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import prepare_f16, upload_weights
    ctx = binding.Context(0, budgets=(128, 256))
    try:
        shape = W.TALKER
        layers = W.make_weights(shape, 4, 901)
        wdev = prepare_f16(ctx, upload_weights(layers))
        _case(torch, binding, ctx, shape, layers, wdev, 96, 910, 300, 1000)   # first call
        _case(torch, binding, ctx, shape, layers, wdev, 9, 920, 10, 200)      # smaller, right after
        _case(torch, binding, ctx, shape, layers, wdev, 96, 910, 300, 1000)   # the first again
    finally:
        torch.cuda.synchronize()
        ctx.close()


def test_noalloc_refuses_oversized_calls_before_any_gpu_work():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    ctx = binding.Context(0, budgets=(128, 256))
    try:
        shape = W.THINKER
        w = [{n: 0x1000 for n in ("ln1", "w_qkv", "w_o", "ln2", "w_gate_up", "w_down")}] * 4
        kv = ([0x5000] * 4, [0x6000] * 4, 1024, 8192)
        # 1024 rows of the thinker need far more than the 64 MiB scratch.
        with pytest.raises(binding.HorizonError) as e:
            binding.hs_downstream_decode_step_noalloc(ctx, shape, w, 1 << 20, 2 << 20, kv, [100] * 1024, 128)
        assert e.value.status == binding.HS_ERR_WORKSPACE and "static scratch" in str(e.value), str(e.value)
        with pytest.raises(binding.HorizonError) as e:
            binding.hs_downstream_decode_step_noalloc(ctx, shape, w, 1 << 20, 2 << 20, kv, [100] * 1025, 128)
        assert e.value.status == binding.HS_ERR_UNSUPPORTED
        with pytest.raises(binding.HorizonError) as e:
            binding.hs_downstream_decode_step_noalloc(ctx, shape, w, 1 << 20, 2 << 20, None, [100], 128)
        assert e.value.status == binding.HS_ERR_INVALID_ARG
    finally:
        ctx.close()
