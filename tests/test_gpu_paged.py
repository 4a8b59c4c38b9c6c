"""GPU parity on a paged key/value cache.

A block table maps each sequence's logical pages onto slots of a pool; the
layer's arithmetic is the same as on contiguous slots, so every case is
checked against the float64 reference on the sequences' logical contents.
Cases: chunked prefill behind cached prefixes with pages smaller than a
prefill query block, two sequences sharing a read-only prefix page, single-row
attention whose key range crosses many pages, and the decode step.  Cache
contents are read back through the table with plain tensor indexing; pool
positions that no sequence owns must keep their fill value.  With pages that
hold whole single-row work units the paged run is bit-identical to the slot
layout.
"""
import numpy as np
import pytest

from oracle import layer as ref
from paper_2608_01785_amd import workloads as W
from tests.gpu_common import TOL, err_ratio, log, require_gpu
from tests.util import f64, h64, weights_f64

pytestmark = pytest.mark.gpu

FILL = 7.0


@pytest.fixture(scope="module")
def env():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    ctx = binding.Context(0, budgets=(128, 192, 256))
    yield torch, ctx
    torch.cuda.synchronize()
    ctx.close()


def make_table(rng, ends, page, spare=3, share=None):
    """Distinct random slots for every page each sequence reaches; share = (src, dst, n): the
    first n pages of sequence dst are those of src.  Unreached entries are -1."""
    need = [-(-int(e) // page) for e in ends]
    pps = max(need) + 1
    n_pages = sum(need) + spare
    perm = rng.permutation(n_pages)
    table = np.full((len(ends), pps), -1, np.int32)
    k = 0
    for b, n in enumerate(need):
        table[b, :n] = perm[k:k + n]
        k += n
    if share is not None:
        src, dst, n = share
        table[dst, :n] = table[src, :n]
    return table, n_pages


def gather(cache, layer, table, page, b, start, stop):
    """Logical rows [start, stop) of sequence b as fp16 bits [n, Hkv, dh] (keys, values)."""
    import torch
    pos = torch.arange(start, stop)
    slots = torch.as_tensor(table[b], dtype=torch.long)[pos // page]
    i = pos % page
    k = cache.k[layer][slots.cuda(), :, i.cuda()]                      # [n, Hkv, dh]
    v = cache.v[layer][slots.cuda(), :, (i // 32).cuda(), :, (i % 32).cuda()]
    return (k.cpu().contiguous().view(torch.int16).numpy().view(np.uint16),
            v.cpu().contiguous().view(torch.int16).numpy().view(np.uint16))


def untouched_positions_hold_fill(cache, layer, table, page, ends):
    """Every pool position outside all sequences' reach still holds the fill value."""
    import torch
    used = torch.zeros((cache.n_slots, page), dtype=torch.bool)
    for b, e in enumerate(ends):
        for p0 in range(0, int(e), page):
            used[int(table[b, p0 // page]), :min(page, int(e) - p0)] = True
    k = cache.k[layer].float().cpu()      # [slots, Hkv, page, dh]
    v = cache.v[layer].float().cpu()      # [slots, Hkv, page / 32, dh, 32]
    v = v.permute(0, 1, 2, 4, 3).reshape(cache.n_slots, v.shape[1], page, v.shape[3])
    free = ~used
    return bool(torch.all(k.permute(0, 2, 1, 3)[free] == FILL)) and bool(torch.all(v.permute(0, 2, 1, 3)[free] == FILL))


@pytest.mark.parametrize("shape_name,page", [("tiny", 64), ("thinker_mixed", 128)])
def test_chunked_prefill_on_paged_cache(env, shape_name, page):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import PagedCache, to_device, upload_weights
    shape = {"tiny": W.TINY, "thinker_mixed": W.THINKER_MIXED}[shape_name]
    lengths, ctx_lens = [200, 1, 1, 130, 70], [300, 70, 500, 0, 128]
    ends = [c + n for c, n in zip(ctx_lens, lengths)]
    rng = np.random.default_rng(61)
    # Sequence 4 reads its first 128 positions from sequence 0's pages (a shared prefix).
    table, n_pages = make_table(rng, ends, page, share=(0, 4, 128 // page))
    layers = W.make_weights(shape, 1, 62)
    batch = W.random_batch(shape.hidden, lengths, seed=63, ctx_lens=ctx_lens)
    prefix = W.make_cache(shape, 1, ctx_lens, seed=64)
    prefix.k[0][4][:] = prefix.k[0][0][:128]
    prefix.v[0][4][:] = prefix.v[0][0][:128]
    cache = PagedCache(1, n_pages, page, shape.n_kv_heads, shape.head_dim, table, fill=FILL)
    for b in range(len(lengths)):
        cache.load_prefix(0, b, prefix.k[0][b], prefix.v[0][b])
    log(f"[paged prefill] {shape_name} page={page} lengths={lengths} ctx={ctx_lens} pool={n_pages}")
    expect, k_new, v_new = ref.layer_forward(
        f64(batch.x), weights_f64(layers)[0], shape, batch.seq_offsets, ctx_lens,
        [h64(k) for k in prefix.k[0]], [h64(v) for v in prefix.v[0]])
    offsets = [int(o) for o in batch.seq_offsets]
    ws = torch.empty(binding.hs_workspace_size_paged(shape, offsets[-1], len(lengths), max(ends), page),
                     dtype=torch.uint8, device="cuda")
    x = to_device(batch.x)
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    binding.hs_shared_stage_forward(ctx, shape, upload_weights(layers), x, y, offsets, ctx_lens, cache.as_arg(),
                                    192, None, ws)
    torch.cuda.synchronize()
    e = err_ratio(y.cpu().numpy(), expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    for b, (c, n) in enumerate(zip(ctx_lens, lengths)):
        kb, vb = gather(cache, 0, table, page, b, 0, c + n)
        np.testing.assert_array_equal(kb[:c], prefix.k[0][b])
        np.testing.assert_array_equal(vb[:c], prefix.v[0][b])
        assert err_ratio(h64(kb[c:]), k_new[offsets[b]:offsets[b + 1]]) <= TOL
        assert err_ratio(h64(vb[c:]), v_new[offsets[b]:offsets[b + 1]]) <= TOL
    assert untouched_positions_hold_fill(cache, 0, table, page, ends)


@pytest.mark.parametrize("page", [64, 256])
def test_decode_rows_cross_many_pages(env, page):
    """Single-row sequences of the 128-wide-head shape behind up to 2000 cached rows."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import PagedCache, to_device, upload_weights
    shape = W.THINKER_MIXED
    n = 12
    rng = np.random.default_rng(71)
    ctx_lens = rng.integers(0, 2000, size=n).astype(np.int32)
    ctx_lens[:5] = [0, page - 1, page, 2 * page - 1, 1999]
    ends = [int(c) + 1 for c in ctx_lens]
    table, n_pages = make_table(rng, ends, page)
    layers = W.make_weights(shape, 1, 72)
    batch = W.random_batch(shape.hidden, [1] * n, seed=73, ctx_lens=ctx_lens)
    prefix = W.make_cache(shape, 1, ctx_lens, seed=74)
    cache = PagedCache(1, n_pages, page, shape.n_kv_heads, shape.head_dim, table, fill=FILL)
    for b in range(n):
        cache.load_prefix(0, b, prefix.k[0][b], prefix.v[0][b])
    log(f"[paged decode rows] page={page} ctx={ctx_lens.tolist()}")
    expect, k_new, v_new = ref.layer_forward(
        f64(batch.x), weights_f64(layers)[0], shape, batch.seq_offsets, ctx_lens,
        [h64(k) for k in prefix.k[0]], [h64(v) for v in prefix.v[0]])
    ws = torch.empty(binding.hs_workspace_size_paged(shape, n, n, max(ends), page), dtype=torch.uint8,
                     device="cuda")
    x = to_device(batch.x)
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    binding.hs_shared_stage_forward(ctx, shape, upload_weights(layers), x, y, list(range(n + 1)), ctx_lens,
                                    cache.as_arg(), 128, None, ws)
    torch.cuda.synchronize()
    e = err_ratio(y.cpu().numpy(), expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    for b in range(n):
        kb, vb = gather(cache, 0, table, page, b, int(ctx_lens[b]), int(ctx_lens[b]) + 1)
        assert err_ratio(h64(kb), k_new[b:b + 1]) <= TOL
        assert err_ratio(h64(vb), v_new[b:b + 1]) <= TOL
    assert untouched_positions_hold_fill(cache, 0, table, page, ends)


@pytest.mark.parametrize("page", [64, 1024])
def test_talker_decode_step_on_paged_cache(env, page):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, PagedCache, prepare_f16, to_device, upload_weights
    shape, n_layers, batch = W.TALKER, 3, 24
    rng = np.random.default_rng(81)
    kv_lens = rng.integers(1, 1400, size=batch).astype(np.int32)
    kv_lens[:4] = [63, 64, 1023, 1024]
    ends = [int(k) + 1 for k in kv_lens]
    table, n_pages = make_table(rng, ends, page)
    layers = W.make_weights(shape, n_layers, 82)
    x = W.token_rows(83, batch, shape.hidden)
    prefix = W.make_cache(shape, n_layers, kv_lens, seed=84)
    cache = PagedCache(n_layers, n_pages, page, shape.n_kv_heads, shape.head_dim, table, fill=FILL)
    for l in range(n_layers):
        for b in range(batch):
            cache.load_prefix(l, b, prefix.k[l][b], prefix.v[l][b])
    log(f"[paged talker decode] page={page} layers={n_layers} batch={batch} kv_lens={kv_lens.tolist()}")
    expect, kv_new = ref.decode_step(f64(x), weights_f64(layers), shape, kv_lens,
                                     [[h64(k) for k in prefix.k[l]] for l in range(n_layers)],
                                     [[h64(v) for v in prefix.v[l]] for l in range(n_layers)])
    ws = torch.empty(binding.hs_workspace_size_paged(shape, batch, batch, max(ends), page), dtype=torch.uint8,
                     device="cuda")
    wdev = prepare_f16(ctx, upload_weights(layers))
    xd = to_device(x)
    y = torch.empty(xd.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    binding.hs_downstream_decode_step(ctx, shape, wdev, xd, y, cache.as_arg(), kv_lens, 128, None, ws)
    torch.cuda.synchronize()
    e = err_ratio(y.cpu().numpy(), expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    for l in range(n_layers):
        for b in range(batch):
            kb, vb = gather(cache, l, table, page, b, int(kv_lens[b]), int(kv_lens[b]) + 1)
            assert err_ratio(h64(kb[0]), kv_new[l][0][b]) <= TOL
            assert err_ratio(h64(vb[0]), kv_new[l][1][b]) <= TOL
        assert untouched_positions_hold_fill(cache, l, table, page, ends)
    if page % 1024 == 0:
        # Pages holding whole work units: the same arithmetic as contiguous slots, bit for bit.
        slots = DeviceCache(n_layers, batch, 1472, shape.n_kv_heads, shape.head_dim, fill=FILL)
        for l in range(n_layers):
            for b in range(batch):
                slots.load_prefix(l, b, prefix.k[l][b], prefix.v[l][b])
        ws2 = torch.empty(binding.hs_workspace_size(shape, batch, batch, max(ends)), dtype=torch.uint8,
                          device="cuda")
        y2 = torch.empty_like(y)
        binding.hs_downstream_decode_step(ctx, shape, wdev, xd, y2, slots.as_arg(), kv_lens, 128, None, ws2)
        torch.cuda.synchronize()
        assert torch.equal(y, y2)
