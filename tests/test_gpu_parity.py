"""GPU parity of the HIP path against the float64 reference, through the C ABI.

Sizes here are small enough for the reference to run in seconds yet span
several GEMM tiles, ragged tails, both head sizes, grouped-query heads,
single-row (decode-path) sequences and cached prefixes.
"""
import numpy as np
import pytest

from oracle import layer as ref
from paper_2608_01785_amd import workloads as W
from tests.gpu_common import TOL, err_ratio, log, require_gpu, workspace
from tests.util import f64, h64, weights_f64

pytestmark = pytest.mark.gpu

BUDGETS = (64, 96, 128, 160, 192, 256)


@pytest.fixture(scope="module")
def env():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    ctx = binding.Context(0, budgets=BUDGETS)
    yield torch, ctx
    torch.cuda.synchronize()
    ctx.close()


def run_prefill(env, shape, wdev, x_bits, offsets, ctx_lens=None, cache=None, budget=256):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import to_device, to_bits
    offsets = [int(o) for o in offsets]
    B = len(offsets) - 1
    cl = [0] * B if ctx_lens is None else [int(c) for c in ctx_lens]
    max_pos = max(cl[b] + offsets[b + 1] - offsets[b] for b in range(B))
    ws = workspace(torch, shape, offsets[-1], B, max_pos)
    x = to_device(x_bits)
    y = torch.empty(x.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    binding.hs_shared_stage_forward(ctx, shape, wdev, x, y, offsets, ctx_lens,
                                    cache.as_arg() if cache is not None else None, budget, None, ws)
    torch.cuda.synchronize()
    return y.cpu().numpy().astype(np.float64)


def seeded_layers(shape, n_layers, seed):
    return W.make_weights(shape, n_layers, seed)


def test_tiny_layer_all_budgets(env):
    torch, _ = env
    from paper_2608_01785_amd.device_data import upload_weights
    shape = W.TINY
    layers = seeded_layers(shape, 1, W.SEEDS["tiny"]["weights"])
    batch = W.tiny_batch()
    expect, _ = ref.stack_forward(f64(batch.x), weights_f64(layers), shape, batch.seq_offsets)
    wdev = upload_weights(layers)
    outs = {}
    for b in BUDGETS:
        log(f"[tiny layer] budget {b}, T={batch.n_tokens}")
        outs[b] = run_prefill(env, shape, wdev, batch.x, batch.seq_offsets, budget=b)
        e = err_ratio(outs[b], expect)
        log(f"  max err / rms = {e:.3e}")
        assert e <= TOL
    for b in BUDGETS:
        np.testing.assert_array_equal(outs[b], outs[256])


@pytest.mark.parametrize("shape_name,lengths,n_layers,fmt", [
    ("thinker", [300, 129, 1, 64, 2], 1, "bf16"),
    ("thinker", [300, 129, 1, 64, 2], 1, "f16"),
    ("tiny", [1, 5, 255, 257, 33], 2, "bf16"),
    ("tiny", [1, 5, 255, 257, 33], 2, "f16"),
    ("talker", [70, 1, 190], 1, "f16"),
    # 128 rows or fewer: the skinny GEMM (one, two and four 32-row subtiles).
    ("tiny", [50, 1, 40], 1, "bf16"),
    ("tiny", [17, 3, 1, 9], 1, "f16"),
    ("talker", [33, 31], 2, "bf16"),
    ("thinker", [60, 1, 3], 1, "bf16"),
    ("thinker", [128], 1, "f16"),
])
def test_ragged_prefill_parity(env, shape_name, lengths, n_layers, fmt):
    from paper_2608_01785_amd.device_data import prepare_f16, upload_weights
    shape = {"thinker": W.THINKER, "tiny": W.TINY, "talker": W.TALKER}[shape_name]
    layers = seeded_layers(shape, n_layers, 77)
    batch = W.random_batch(shape.hidden, lengths, seed=78)
    log(f"[ragged prefill] {shape_name} lengths={lengths} layers={n_layers} weights={fmt}")
    expect, _ = ref.stack_forward(f64(batch.x), weights_f64(layers), shape, batch.seq_offsets)
    wdev = upload_weights(layers)
    if fmt == "f16":
        wdev = prepare_f16(env[1], wdev)
    got = run_prefill(env, shape, wdev, batch.x, batch.seq_offsets, budget=128)
    e = err_ratio(got, expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL


def test_weight_preparation_layout(env):
    """hs_convert_weights_f16: fp16 of every value, in panel-major order [K / 32][N][32]."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import f16_bits_of, to_device
    rng = np.random.default_rng(51)
    n, k = 96, 160
    w = W.bf16_bits(rng.standard_normal((n, k), dtype=np.float32) * np.float32(0.02))
    w[0, :4] = W.bf16_bits(np.array([1e-6, -3e-5, 7.0, -59904.0], np.float32))  # subnormals, large normals
    src = to_device(w)
    dst = torch.empty((k // 32, n, 32), dtype=torch.float16, device="cuda")
    binding.hs_convert_weights_f16(ctx, src, dst)
    torch.cuda.synchronize()
    got = f16_bits_of(dst).view(np.float16).astype(np.float64)
    vals = W.bf16_to_f32(w).astype(np.float64)
    expect = vals.reshape(n, k // 32, 32).transpose(1, 0, 2)
    normal = np.abs(expect) >= 2.0 ** -14
    np.testing.assert_array_equal(got[normal], expect[normal])              # exact in the normal range
    assert np.all(np.abs(got[~normal] - expect[~normal]) < 2.0 ** -24)     # subnormals: toward zero
    with pytest.raises(binding.HorizonError):
        binding.hs_convert_weights_f16(ctx, src, dst, n, 100)              # cols not a multiple of 32


def test_residual_identity_bit_exact(env):
    from paper_2608_01785_amd.device_data import upload_weights
    shape = W.TINY
    layers = seeded_layers(shape, 2, 5)
    for lw in layers:
        lw["w_o"][:] = 0
        lw["w_down"][:] = 0
    batch = W.random_batch(shape.hidden, [40, 300, 1], seed=6)
    log("[residual identity] tiny, 2 layers, W_o = W_down = 0")
    got = run_prefill(env, shape, upload_weights(layers), batch.x, batch.seq_offsets)
    np.testing.assert_array_equal(got, f64(batch.x))


def test_causal_invariance_and_isolation(env):
    from paper_2608_01785_amd.device_data import upload_weights
    shape = W.TINY
    wdev = upload_weights(seeded_layers(shape, 1, 9))
    batch = W.random_batch(shape.hidden, [200, 150], seed=10)
    log("[causal] tiny, perturb rows >= 120 of sequence 0")
    y1 = run_prefill(env, shape, wdev, batch.x, batch.seq_offsets)
    x2 = batch.x.copy()
    x2[120:200] = W.token_rows(11, 80, shape.hidden)
    y2 = run_prefill(env, shape, wdev, x2, batch.seq_offsets)
    np.testing.assert_array_equal(y2[:120], y1[:120])
    np.testing.assert_array_equal(y2[200:], y1[200:])   # the other sequence is untouched
    assert np.any(y2[120:200] != y1[120:200])
    # Swapping the two sequences swaps the outputs.
    xs = np.concatenate([batch.x[200:], batch.x[:200]])
    ys = run_prefill(env, shape, wdev, xs, [0, 150, 350])
    np.testing.assert_array_equal(ys[:150], y1[200:])
    np.testing.assert_array_equal(ys[150:], y1[:200])


def test_cached_prefix_chunks_and_cache_writes(env):
    torch, _ = env
    from paper_2608_01785_amd.device_data import DeviceCache, upload_weights
    shape = W.THINKER_MIXED
    lengths, ctx_lens = [200, 1, 1, 130], [300, 70, 500, 0]
    layers = seeded_layers(shape, 1, 21)
    batch = W.random_batch(shape.hidden, lengths, seed=22, ctx_lens=ctx_lens)
    prefix = W.make_cache(shape, 1, ctx_lens, seed=23)
    cache = DeviceCache(1, 4, 640, shape.n_kv_heads, shape.head_dim, fill=7.0)
    for b, c in enumerate(ctx_lens):
        cache.load_prefix(0, b, prefix.k[0][b], prefix.v[0][b])
    torch.cuda.synchronize()
    log(f"[cached prefix] thinker-mixed shape lengths={lengths} ctx={ctx_lens}")
    expect, k_new, v_new = ref.layer_forward(
        f64(batch.x), weights_f64(layers)[0], shape, batch.seq_offsets, ctx_lens,
        [h64(k) for k in prefix.k[0]], [h64(v) for v in prefix.v[0]])
    got = run_prefill(env, shape, upload_weights(layers), batch.x, batch.seq_offsets, ctx_lens, cache, budget=96)
    e = err_ratio(got, expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    off = batch.seq_offsets
    for b in range(4):
        c, n = ctx_lens[b], lengths[b]
        kb, vb = cache.rows(0, b, 0, 640)
        # Prefix untouched, new rows match the reference, the rest still holds the fill value.
        np.testing.assert_array_equal(kb[:c], prefix.k[0][b])
        np.testing.assert_array_equal(vb[:c], prefix.v[0][b])
        assert err_ratio(h64(kb[c:c + n]), k_new[off[b]:off[b + 1]]) <= TOL
        assert err_ratio(h64(vb[c:c + n]), v_new[off[b]:off[b + 1]]) <= TOL
        assert np.all(h64(kb[c + n:]) == 7.0) and np.all(h64(vb[c + n:]) == 7.0)


@pytest.mark.parametrize("batch,fmt", [(8, "bf16"), (40, "f16"), (97, "bf16"), (128, "f16")])
def test_talker_decode_step_parity(env, batch, fmt):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import DeviceCache, prepare_f16, to_device, upload_weights
    shape = W.TALKER
    n_layers = 4
    rng = np.random.default_rng(31 + batch)
    kv_lens = rng.integers(1, 300, size=batch).astype(np.int32)
    kv_lens[0] = 255  # new key lands at the end of a 256-key chunk
    kv_lens[1] = 256  # new key starts a chunk
    layers = seeded_layers(shape, n_layers, 32)
    x = W.token_rows(33, batch, shape.hidden)
    prefix = W.make_cache(shape, n_layers, kv_lens, seed=34)
    cache = DeviceCache(n_layers, batch, 320, shape.n_kv_heads, shape.head_dim, fill=0.0)
    for l in range(n_layers):
        for b in range(batch):
            cache.load_prefix(l, b, prefix.k[l][b], prefix.v[l][b])
    log(f"[talker decode] layers={n_layers} batch={batch} weights={fmt} kv_lens={kv_lens.tolist()}")
    expect, kv_new = ref.decode_step(f64(x), weights_f64(layers), shape, kv_lens,
                                     [[h64(k) for k in prefix.k[l]] for l in range(n_layers)],
                                     [[h64(v) for v in prefix.v[l]] for l in range(n_layers)])
    ws = workspace(torch, shape, batch, batch, int(kv_lens.max()) + 1)
    xd = to_device(x)
    y = torch.empty(xd.shape, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    wdev = upload_weights(layers)
    if fmt == "f16":
        wdev = prepare_f16(ctx, wdev)
    binding.hs_downstream_decode_step(ctx, shape, wdev, xd, y, cache.as_arg(), kv_lens, 128, None, ws)
    torch.cuda.synchronize()
    e = err_ratio(y.cpu().numpy(), expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    # Split-K partial sums are added in a fixed order: a repeat (same cache
    # positions rewritten with the same rows) at another budget is bit-identical.
    y2 = torch.empty_like(y)
    binding.hs_downstream_decode_step(ctx, shape, wdev, xd, y2, cache.as_arg(), kv_lens, 64, None, ws)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    for l in range(n_layers):
        for b in range(batch):
            kb, vb = cache.rows(l, b, int(kv_lens[b]), int(kv_lens[b]) + 1)
            assert err_ratio(h64(kb[0]), kv_new[l][0][b]) <= TOL
            assert err_ratio(h64(vb[0]), kv_new[l][1][b]) <= TOL


def test_decode_rows_behind_long_prefixes(env):
    """Single-row sequences of the 128-wide-head shape behind cached prefixes up to 2000 rows."""
    torch, _ = env
    from paper_2608_01785_amd.device_data import DeviceCache, upload_weights
    shape = W.THINKER_MIXED
    n = 24
    rng = np.random.default_rng(41)
    ctx_lens = rng.integers(0, 2000, size=n).astype(np.int32)
    ctx_lens[:4] = [0, 31, 32, 1999]
    lengths = [1] * n
    layers = seeded_layers(shape, 1, 42)
    batch = W.random_batch(shape.hidden, lengths, seed=43, ctx_lens=ctx_lens)
    prefix = W.make_cache(shape, 1, ctx_lens, seed=44)
    cache = DeviceCache(1, n, 2048, shape.n_kv_heads, shape.head_dim, fill=0.0)
    for b in range(n):
        cache.load_prefix(0, b, prefix.k[0][b], prefix.v[0][b])
    torch.cuda.synchronize()
    log(f"[decode rows] thinker-mixed shape, {n} rows, ctx={ctx_lens.tolist()}")
    expect, k_new, v_new = ref.layer_forward(
        f64(batch.x), weights_f64(layers)[0], shape, batch.seq_offsets, ctx_lens,
        [h64(k) for k in prefix.k[0]], [h64(v) for v in prefix.v[0]])
    got = run_prefill(env, shape, upload_weights(layers), batch.x, batch.seq_offsets, ctx_lens, cache, budget=192)
    e = err_ratio(got, expect)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
    for b in range(n):
        kb, vb = cache.rows(0, b, int(ctx_lens[b]), int(ctx_lens[b]) + 1)
        assert err_ratio(h64(kb), k_new[b:b + 1]) <= TOL
        assert err_ratio(h64(vb), v_new[b:b + 1]) <= TOL


@pytest.fixture(scope="module")
def hw_table(env):
    """Measured topology: for every mask bit, the (XCD, shader engine, CU) it names.

    The runtime refuses a CU mask that leaves an XCD without CUs, so each bit is
    found by difference: a stream masked to a base set of eight bits (one per
    XCD by the default mapping) plus the bit runs on the base set's CUs and one
    more, which is the bit's (probe kernel, 1024 work-groups per stream)."""
    import ctypes
    torch, ctx = env
    from paper_2608_01785_amd import binding
    hip = ctypes.CDLL("libamdhip64.so.7")           # the runtime already loaded in this process
    hip.hipExtStreamCreateWithCUMask.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint32,
                                                 ctypes.POINTER(ctypes.c_uint32)]
    hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    n = 1024
    out = torch.zeros(n * 4, dtype=torch.int32, device="cuda")

    def probe(bits):
        mask = (ctypes.c_uint32 * 8)()
        for i in bits:
            mask[i // 32] |= 1 << (i % 32)
        s = ctypes.c_void_p()
        rc = hip.hipExtStreamCreateWithCUMask(ctypes.byref(s), 8, mask)
        if rc != 0:
            hip.hipGetLastError()                       # leave no sticky error for later calls
            raise AssertionError(f"stream with mask bits {sorted(bits)[:10]} refused: error {rc}")
        try:
            out.zero_()
            torch.cuda.synchronize()
            binding.hs_probe_hw_ids(ctx, s.value, n, out)
            torch.cuda.synchronize()
        finally:
            hip.hipStreamDestroy(s)
        return {(int(a), int(b_), int(c)) for a, b_, c, _ in out.view(n, 4).cpu().numpy()}

    log("[topology] probing every mask bit against a one-CU-per-XCD base set")
    bases = [list(range(8 * j, 8 * j + 8)) for j in (0, 1)]
    base_ids = [probe(b) for b in bases]
    for b, ids in zip(bases, base_ids):
        assert len(ids) == 8, (b, ids)
    table = []
    for i in range(256):
        k = 1 if i < 8 else 0                           # a base that does not hold bit i
        extra = probe(bases[k] + [i]) - base_ids[k]
        assert len(extra) == 1, (i, extra)
        table.append(extra.pop())
    return table


def test_measured_topology_matches_the_default_xcd_mapping(hw_table):
    """Every mask bit is a distinct CU; bit i sits on XCD i % 8 as the default
    topology (and so the partition) assumes, and each XCD holds 32 bits."""
    from paper_2608_01785_amd import binding
    assert len(set(hw_table)) == 256
    d = binding.hs_default_topology()
    bad = [i for i in range(256) if hw_table[i][0] != d.xcc[i]]
    assert not bad, f"bits on another XCD than the default topology says: {bad[:16]}"
    per_xcd = np.bincount([t[0] for t in hw_table], minlength=8)
    assert per_xcd.tolist() == [32] * 8
    same = sum((hw_table[i][1], hw_table[i][2]) == (d.se[i], d.cu[i]) for i in range(256))
    log(f"[topology] XCD of every bit as assumed; shader engine and CU as assumed for {same} of 256 bits")
    # The partition from the measured table is balanced per XCD at every ladder budget.
    t = binding.topology_from_lists([x for x, _, _ in hw_table], [s for _, s, _ in hw_table],
                                    [c for _, _, c in hw_table], 8)
    for c in (16, 64, 96, 128, 160, 192, 224):
        sh, _ = binding.hs_cu_partition(t, c)
        bits = [i for i in range(256) if (sh[i // 32] >> (i % 32)) & 1]
        cnt = np.bincount([hw_table[i][0] for i in bits], minlength=8)
        assert cnt.max() - cnt.min() <= 1 and cnt.sum() == c, (c, cnt)


def test_masks_hold_on_hardware(env, hw_table):
    """Waves of each ladder stream run only on the CUs its mask names (by the
    measured table), the two sides are disjoint, and each side is balanced over
    the eight XCDs."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    popc = lambda ws: sum(bin(w).count("1") for w in ws)
    for budget in (64, 128, 192):
        sh, dn = binding.hs_context_masks(ctx, budget)
        assert popc(sh) == budget and popc(dn) == 256 - budget
        seen = {}
        for role, words in ((binding.HS_ROLE_SHARED, sh), (binding.HS_ROLE_DOWN, dn)):
            allowed = {hw_table[i] for i in range(256) if (words[i // 32] >> (i % 32)) & 1}
            cnt = np.bincount([x for x, _, _ in allowed], minlength=8)
            assert cnt.max() - cnt.min() <= 1, (budget, role, cnt)
            s = binding.hs_context_stream(ctx, budget, role)
            n = 4096
            out = torch.zeros(n * 4, dtype=torch.int32, device="cuda")
            torch.cuda.synchronize()
            log(f"[probe] budget {budget} role {role}")
            binding.hs_probe_hw_ids(ctx, s, n, out)
            torch.cuda.synchronize()
            ids = out.view(n, 4).cpu().numpy()
            seen[role] = {(int(a), int(b_), int(c)) for a, b_, c, _ in ids}
            log(f"  distinct CUs used: {len(seen[role])}")
            assert seen[role] <= allowed, sorted(seen[role] - allowed)[:8]
        assert not (seen[0] & seen[1])
        assert len(seen[0]) >= 0.9 * budget  # 4096 blocks spread over (nearly) every CU of the mask



def test_graph_replay_keeps_the_stream_mask(env, hw_table):
    """Kernels replayed from a captured graph run on the CUs of the stream the
    graph is launched on: a probe captured once and replayed on each side of a
    ladder level stays inside that side's mask."""
    torch, ctx = env
    from paper_2608_01785_amd import binding
    n = 4096
    out = torch.zeros(n * 4, dtype=torch.int32, device="cuda")
    sh, dn = binding.hs_context_masks(ctx, 128)
    for role, words in ((binding.HS_ROLE_SHARED, sh), (binding.HS_ROLE_DOWN, dn)):
        allowed = {hw_table[i] for i in range(256) if (words[i // 32] >> (i % 32)) & 1}
        s = binding.hs_context_stream(ctx, 128, role)
        ext = torch.cuda.ExternalStream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=ext):
            binding.hs_probe_hw_ids(ctx, s, n, out)
        out.zero_()
        torch.cuda.synchronize()
        log(f"[graph probe] role {role}")
        with torch.cuda.stream(ext):
            g.replay()
        torch.cuda.synchronize()
        seen = {(int(a), int(b_), int(c)) for a, b_, c, _ in out.view(n, 4).cpu().numpy()}
        log(f"  distinct CUs used by the replay: {len(seen)}")
        assert seen <= allowed, sorted(seen - allowed)[:8]
        assert len(seen) >= 0.9 * 128
        del g
