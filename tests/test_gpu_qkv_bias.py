"""GPU parity with a bias on the QKV projection (the optional b_qkv weight).

The bias is added to the projection before RoPE rotates the query and key
heads; value heads take it unrotated.  Biases here are N(0, 0.5), as large as
the projection itself, so a bias dropped, added after RoPE or to the wrong
column fails the float64 reference by far more than the tolerance.  Cases
cover the tiled GEMM (more than 128 rows) and the skinny GEMM (128 rows or
fewer), both head sizes, both weight formats, and the decode step.
"""
import numpy as np
import pytest

from oracle import layer as ref
from paper_2608_01785_amd import workloads as W
from tests.gpu_common import TOL, err_ratio, log, require_gpu, workspace
from tests.util import f64, h64, weights_f64

pytestmark = pytest.mark.gpu

BIAS_STD = 0.5


@pytest.fixture(scope="module")
def env():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    ctx = binding.Context(0, budgets=(96, 256))
    yield torch, ctx
    torch.cuda.synchronize()
    ctx.close()


@pytest.mark.parametrize("shape_name,lengths,fmt", [
    ("tiny", [1, 5, 255, 257, 33], "bf16"),      # tiled GEMM, head_dim 64
    ("thinker", [300, 129, 1, 64, 2], "f16"),    # tiled GEMM, head_dim 128
    ("talker", [33, 31], "bf16"),                # skinny GEMM, head_dim 64
    ("thinker", [60, 1, 3], "f16"),              # skinny GEMM, head_dim 128
])
def test_prefill_with_qkv_bias(env, shape_name, lengths, fmt):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import prepare_f16, to_device, upload_weights
    shape = {"thinker": W.THINKER, "tiny": W.TINY, "talker": W.TALKER}[shape_name]
    layers = W.make_weights(shape, 1, 91, qkv_bias_std=BIAS_STD)
    batch = W.random_batch(shape.hidden, lengths, seed=92)
    log(f"[qkv bias prefill] {shape_name} lengths={lengths} weights={fmt}")
    expect, _ = ref.stack_forward(f64(batch.x), weights_f64(layers), shape, batch.seq_offsets)
    no_bias = [{k: v for k, v in lw.items() if k != "b_qkv"} for lw in layers]
    expect_nb, _ = ref.stack_forward(f64(batch.x), weights_f64(no_bias), shape, batch.seq_offsets)
    assert err_ratio(expect_nb, expect) > 10 * TOL  # the bias matters at this size
    wdev = upload_weights(layers)
    if fmt == "f16":
        wdev = prepare_f16(ctx, wdev)
    offsets = [int(o) for o in batch.seq_offsets]
    ws = workspace(torch, shape, offsets[-1], len(lengths), max(lengths))
    x = to_device(batch.x)
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    outs = []
    for budget in (96, 256):
        binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, offsets, None, None, budget, None, ws)
        torch.cuda.synchronize()
        outs.append(y.cpu().numpy().astype(np.float64))
        e = err_ratio(outs[-1], expect)
        log(f"  budget {budget}: max err / rms = {e:.3e}")
        assert e <= TOL
    np.testing.assert_array_equal(outs[0], outs[1])


def test_decode_step_with_qkv_bias(env):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, prepare_f16, to_device, upload_weights
    shape, n_layers, batch = W.TALKER, 2, 40
    rng = np.random.default_rng(93)
    kv_lens = rng.integers(1, 300, size=batch).astype(np.int32)
    layers = W.make_weights(shape, n_layers, 94, qkv_bias_std=BIAS_STD)
    x = W.token_rows(95, batch, shape.hidden)
    prefix = W.make_cache(shape, n_layers, kv_lens, seed=96)
    cache = DeviceCache(n_layers, batch, 320, shape.n_kv_heads, shape.head_dim, fill=0.0)
    for l in range(n_layers):
        for b in range(batch):
            cache.load_prefix(l, b, prefix.k[l][b], prefix.v[l][b])
    log(f"[qkv bias decode] talker layers={n_layers} batch={batch}")
    expect, kv_new = ref.decode_step(f64(x), weights_f64(layers), shape, kv_lens,
                                     [[h64(k) for k in prefix.k[l]] for l in range(n_layers)],
                                     [[h64(v) for v in prefix.v[l]] for l in range(n_layers)])
    ws = workspace(torch, shape, batch, batch, int(kv_lens.max()) + 1)
    xd = to_device(x)
    y = torch.empty(xd.shape, dtype=torch.float32, device="cuda")
    wdev = prepare_f16(ctx, upload_weights(layers))
    binding.hs_downstream_decode_step(ctx, shape, wdev, xd, y, cache.as_arg(), kv_lens, 160, None, ws)
    torch.cuda.synchronize()
    e = err_ratio(y.cpu().numpy(), expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    for l in range(n_layers):
        for b in range(batch):
            kb, vb = cache.rows(l, b, int(kv_lens[b]), int(kv_lens[b]) + 1)
            assert err_ratio(h64(kb[0]), kv_new[l][0][b]) <= TOL
            assert err_ratio(h64(vb[0]), kv_new[l][1][b]) <= TOL
