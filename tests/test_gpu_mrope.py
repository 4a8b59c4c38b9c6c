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


def test_talker_decode_step_with_mrope_positions(env):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, prepare_f16, to_device, upload_weights
    shape = dataclasses.replace(W.TALKER, mrope_sections=SECTIONS[64])
    n_layers, batch = 2, 24
    rng = np.random.default_rng(111)
    kv_lens = rng.integers(1, 400, size=batch).astype(np.int32)
    # New rows of an audio-output stream: temporal position kv_len, height and width
    # positions of a 2-D layout below it.
    pos3 = np.stack([kv_lens, kv_lens // 2, kv_lens // 3]).astype(np.int32)
    layers = W.make_weights(shape, n_layers, 112)
    x = W.token_rows(113, batch, shape.hidden)
    prefix = W.make_cache(shape, n_layers, kv_lens, seed=114)
    cache = DeviceCache(n_layers, batch, 448, shape.n_kv_heads, shape.head_dim, fill=0.0)
    for l in range(n_layers):
        for b in range(batch):
            cache.load_prefix(l, b, prefix.k[l][b], prefix.v[l][b])
    log(f"[mrope decode] talker layers={n_layers} batch={batch}")
    pk = [[h64(k) for k in prefix.k[l]] for l in range(n_layers)]
    pv = [[h64(v) for v in prefix.v[l]] for l in range(n_layers)]
    expect, kv_new = ref.decode_step(f64(x), weights_f64(layers), shape, kv_lens, pk, pv, positions3=pos3)
    _, kv_plain = ref.decode_step(f64(x), weights_f64(layers), shape, kv_lens, pk, pv)
    assert err_ratio(kv_plain[0][0], kv_new[0][0]) > 10 * TOL
    ws = workspace(torch, shape, batch, batch, int(kv_lens.max()) + 1)
    wdev = prepare_f16(ctx, upload_weights(layers))
    xd = to_device(x)
    y = torch.empty(xd.shape, dtype=torch.float32, device="cuda")
    binding.hs_downstream_decode_step_mrope(ctx, shape, wdev, xd, y, cache.as_arg(), kv_lens, pos3, 128, None, ws)
    torch.cuda.synchronize()
    e = err_ratio(y.cpu().numpy(), expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    for l in range(n_layers):
        for b in range(batch):
            kb, vb = cache.rows(l, b, int(kv_lens[b]), int(kv_lens[b]) + 1)
            assert err_ratio(h64(kb[0]), kv_new[l][0][b]) <= TOL
            assert err_ratio(h64(vb[0]), kv_new[l][1][b]) <= TOL
