"""GPU parity with multimodal RoPE positions (rows of image patches, then text).

Each row carries a temporal, height and width position and the rotary pairs
are split into sections (8/12/12 pairs for head_dim 64, 16/24/24 for 128), so
keys and queries of patch rows turn by their grid coordinates.  The key rows
the QKV epilogue writes to the cache are checked as well as the output: RoPE
turns them directly, so they expose a wrong angle even where the residual
stream dominates the output.  Cases cover the tiled and the skinny QKV
epilogues; with three equal components the result must be bit-identical to
the plain forward.
"""
import dataclasses

import numpy as np
import pytest

from oracle import layer as ref
from paper_2608_01785_amd import workloads as W
from tests.gpu_common import TOL, err_ratio, log, require_gpu, workspace
from tests.util import f64, h64, weights_f64

pytestmark = pytest.mark.gpu

SECTIONS = {64: (8, 12, 12), 128: (16, 24, 24)}


@pytest.fixture(scope="module")
def env():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    ctx = binding.Context(0, budgets=(128, 256))
    yield torch, ctx
    torch.cuda.synchronize()
    ctx.close()


@pytest.mark.parametrize("shape_name,lengths,n_img", [
    ("tiny", [1, 5, 255, 257, 33], [0, 3, 180, 100, 33]),
    ("thinker", [300, 129, 1, 64, 2], [200, 64, 1, 0, 2]),
    ("tiny", [50, 1, 40], [30, 0, 40]),
    ("thinker", [60, 1, 3], [45, 1, 0]),
])
def test_prefill_with_mrope_positions(env, shape_name, lengths, n_img):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, to_device, upload_weights
    base = {"tiny": W.TINY, "thinker": W.THINKER}[shape_name]
    shape = dataclasses.replace(base, mrope_sections=SECTIONS[base.head_dim])
    layers = W.make_weights(shape, 1, 101)
    batch = W.random_batch(shape.hidden, lengths, seed=102)
    pos3 = W.mrope_positions(lengths, n_img, grid_w=16)
    log(f"[mrope] {shape_name} lengths={lengths} n_img={n_img}")
    ctx_lens = [0] * len(lengths)
    expect, kv = ref.stack_forward(f64(batch.x), weights_f64(layers), shape, batch.seq_offsets, ctx_lens,
                                   positions3=pos3)
    _, kv_plain = ref.stack_forward(f64(batch.x), weights_f64(layers), shape, batch.seq_offsets, ctx_lens)
    assert err_ratio(kv_plain[0][0], kv[0][0]) > 10 * TOL  # the positions turn the keys
    cache = DeviceCache(1, len(lengths), -(-max(lengths) // 64) * 64, shape.n_kv_heads, shape.head_dim, fill=0.0)
    offsets = [int(o) for o in batch.seq_offsets]
    ws = workspace(torch, shape, offsets[-1], len(lengths), max(lengths))
    wdev = upload_weights(layers)
    x = to_device(batch.x)
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    binding.hs_shared_stage_forward_mrope(ctx, shape, wdev, x, y, offsets, pos3, ctx_lens, cache.as_arg(), 128,
                                          None, ws)
    torch.cuda.synchronize()
    got = y.cpu().numpy().astype(np.float64)
    e = err_ratio(got, expect)
    k_rows = np.concatenate([h64(cache.rows(0, b, 0, n)[0]) for b, n in enumerate(lengths)])
    ek = err_ratio(k_rows, kv[0][0])
    log(f"  max err / rms = {e:.3e} (output), {ek:.3e} (keys)")
    assert e <= TOL and ek <= TOL
    # Three equal components: bit-identical to the plain forward.
    lin = np.concatenate([np.arange(n) for n in lengths]).astype(np.int32)
    binding.hs_shared_stage_forward_mrope(ctx, shape, wdev, x, y, offsets, np.stack([lin, lin, lin]), ctx_lens,
                                          cache.as_arg(), 128, None, ws)
    torch.cuda.synchronize()
    y_eq = y.cpu().numpy()
    binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, offsets, ctx_lens, cache.as_arg(), 128, None, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(y_eq, y.cpu().numpy())
