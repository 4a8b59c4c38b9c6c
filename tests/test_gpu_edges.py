"""GPU parity on the degenerate and limit cases of a prefill batch.

* Empty sequences at the start, middle and end of a batch (no rows, no
  attention work, no cache writes), on the tiled and the skinny paths, with
  and without a cached prefix behind the empty sequence.
* A batch of one row.
* The largest supported hidden size (8192; RMSNorm keeps a row in registers
  up to that width).
"""
import dataclasses

import numpy as np
import pytest

from oracle import layer as ref
from paper_2608_01785_amd import workloads as W
from tests.gpu_common import TOL, err_ratio, log, require_gpu, workspace
from tests.util import f64, h64, weights_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    ctx = binding.Context(0, budgets=(128, 256))
    yield torch, ctx
    torch.cuda.synchronize()
    ctx.close()


def run(env, shape, layers, batch, ctx_lens=None, prefix=None, max_ctx=0):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, to_device, upload_weights
    offsets = [int(o) for o in batch.seq_offsets]
    B = len(offsets) - 1
    cache = None
    if ctx_lens is not None:
        cache = DeviceCache(1, B, max_ctx, shape.n_kv_heads, shape.head_dim, fill=3.0)
        for b in range(B):
            cache.load_prefix(0, b, prefix.k[0][b], prefix.v[0][b])
    ends = [(0 if ctx_lens is None else int(ctx_lens[b])) + offsets[b + 1] - offsets[b] for b in range(B)]
    ws = workspace(torch, shape, offsets[-1], B, max(max(ends), 1))
    x = to_device(batch.x)
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    binding.hs_shared_stage_forward(ctx, shape, upload_weights(layers), x, y, offsets, ctx_lens,
                                    cache.as_arg() if cache is not None else None, 128, None, ws)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64), cache


@pytest.mark.parametrize("lengths", [[0, 5, 0, 130, 0], [0, 3, 0, 1], [1]])
def test_empty_sequences_and_single_row(env, lengths):
    shape = W.TINY
    layers = W.make_weights(shape, 2, 121)
    batch = W.random_batch(shape.hidden, lengths, seed=122)
    log(f"[edges] tiny lengths={lengths}")
    expect, _ = ref.stack_forward(f64(batch.x), weights_f64(layers), shape, batch.seq_offsets)
    got, _ = run(env, shape, layers, batch)
    e = err_ratio(got, expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL


def test_empty_sequence_behind_a_cached_prefix_writes_nothing(env):
    shape = W.TINY
    lengths, ctx_lens = [0, 40, 0, 1], [70, 10, 0, 129]
    layers = W.make_weights(shape, 1, 123)
    batch = W.random_batch(shape.hidden, lengths, seed=124, ctx_lens=ctx_lens)
    prefix = W.make_cache(shape, 1, ctx_lens, seed=125)
    log(f"[edges] cached prefixes ctx={ctx_lens} lengths={lengths}")
    expect, k_new, _ = ref.layer_forward(f64(batch.x), weights_f64(layers)[0], shape, batch.seq_offsets, ctx_lens,
                                         [h64(k) for k in prefix.k[0]], [h64(v) for v in prefix.v[0]])
    got, cache = run(env, shape, layers, batch, ctx_lens, prefix, max_ctx=192)
    assert err_ratio(got, expect) <= TOL
    off = batch.seq_offsets
    for b, (c, n) in enumerate(zip(ctx_lens, lengths)):
        kb, vb = cache.rows(0, b, 0, 192)
        np.testing.assert_array_equal(kb[:c], prefix.k[0][b])
        assert err_ratio(h64(kb[c:c + n]), k_new[off[b]:off[b + 1]]) <= TOL if n else True
        assert np.all(h64(kb[c + n:]) == 3.0) and np.all(h64(vb[c + n:]) == 3.0)  # nothing past the rows


@pytest.mark.parametrize("lengths", [[200, 40], [17, 1]])
def test_largest_hidden_size(env, lengths):
    shape = W.LayerShape(8192, 64, 8, 128, 1024)
    layers = W.make_weights(shape, 1, 126)
    batch = W.random_batch(shape.hidden, lengths, seed=127)
    log(f"[edges] hidden 8192 lengths={lengths}")
    expect, _ = ref.stack_forward(f64(batch.x), weights_f64(layers), shape, batch.seq_offsets)
    got, _ = run(env, shape, layers, batch)
    e = err_ratio(got, expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL


def _score_jumps(x, w, shape, lengths):
    """Largest rise, over the rows of every sequence and query head, of the
    running score maximum (log2 units, scale included) after the row's first
    64 keys: the prefill attention moves its reference maximum only when a
    tile's maximum exceeds it by more than 8."""
    n = ref.rms_norm(x, w["ln1"], shape.rms_eps)
    qkv = n @ w["w_qkv"].T
    hq, hkv, dh = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    T = x.shape[0]
    q = qkv[:, : hq * dh].reshape(T, hq, dh)
    k = qkv[:, hq * dh: (hq + hkv) * dh].reshape(T, hkv, dh)
    best, off = 0.0, 0
    for L in lengths:
        pos = np.arange(L)
        qs = ref.rope(q[off:off + L], pos, shape.rope_base)
        ks = ref.rope(k[off:off + L], pos, shape.rope_base)
        for h in range(hq):
            s = qs[:, h] @ ks[:, h // (hq // hkv)].T / np.sqrt(dh) * np.log2(np.e)
            for i in range(64, L):
                best = max(best, s[i, 64:i + 1].max() - s[i, :64].max())
        off += L
    return best


@pytest.mark.parametrize("shape", [W.TINY, W.LayerShape(512, 4, 2, 128, 1024)], ids=["dh64", "dh128"])
def test_sharp_scores_move_the_running_maximum(env, shape):
    """Query and key projections 6x the usual scale make the scores span tens of
    log2 units, so rows meet keys far above their first tile's maximum: the
    reference maximum moves on later tiles (output rescale) and weights up to
    2^8 pass through fp16.  Checked against the oracle; the premise itself is
    checked on the oracle's scores."""
    layers = W.make_weights(shape, 1, 131)
    w = layers[0]["w_qkv"]
    layers[0]["w_qkv"] = W.bf16_bits(W.bf16_to_f32(w) * np.float32(6.0))
    lengths = [300, 130, 1]
    batch = W.random_batch(shape.hidden, lengths, seed=132)
    wf = weights_f64(layers)
    jump = _score_jumps(f64(batch.x), wf[0], shape, lengths)
    log(f"[edges] sharp scores dh={shape.head_dim}: largest rise of a row's maximum after its first tile "
        f"{jump:.1f} (log2 units)")
    assert jump > 8.0
    expect, _ = ref.stack_forward(f64(batch.x), wf, shape, batch.seq_offsets)
    got, _ = run(env, shape, layers, batch)
    e = err_ratio(got, expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
