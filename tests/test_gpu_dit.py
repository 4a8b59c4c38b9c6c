"""GPU parity of the DiT denoising step (hs_dit_forward) against the float64 reference."""
import numpy as np
import pytest

from oracle import dit as D
from paper_2608_01785_amd import workloads as W
from tests.gpu_common import TOL, err_ratio, log, require_gpu
from tests.util import f64

pytestmark = pytest.mark.gpu

BUDGETS = (96, 128, 192)   # ladder levels; the DiT runs on the complement (160, 128, 64 CUs)


@pytest.fixture(scope="module")
def env():
    torch = require_gpu()
    from paper_2608_01785_amd import binding
    ctx = binding.Context(0, budgets=BUDGETS)
    yield torch, ctx
    torch.cuda.synchronize()
    ctx.close()


def w64(layers):
    return [{k: f64(v) for k, v in lw.items()} for lw in layers]


def run_dit(env, shape, wdev, x_bits, cond, offsets, down_cus=128):
    torch, ctx = env
    from paper_2608_01785_amd import binding
    from paper_2608_01785_amd.device_data import to_device
    T, B = int(offsets[-1]), len(offsets) - 1
    ws = torch.empty(binding.hs_dit_workspace_size(shape, T, B), dtype=torch.uint8, device="cuda")
    x = to_device(x_bits) if T else torch.empty((0, shape.hidden), dtype=torch.bfloat16, device="cuda")
    y = torch.full((T, shape.hidden), float("nan"), dtype=torch.float32, device="cuda")
    c = torch.from_numpy(np.ascontiguousarray(cond, np.float32)).to("cuda")
    torch.cuda.synchronize()
    binding.hs_dit_forward(ctx, shape, wdev, x, y, c, offsets, down_cus, None, ws)
    torch.cuda.synchronize()
    return y


def _case(shape, n_layers, lengths, seed):
    layers = W.make_dit_weights(shape, n_layers, seed)
    off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    x = W.token_rows(seed + 1, int(off[-1]), shape.hidden)
    cond = W.dit_cond(seed + 2, len(lengths), shape.hidden)
    return layers, off, x, cond


@pytest.mark.parametrize("fmt", ["bf16", "f16"])
def test_dit_tiny_ragged_parity(env, fmt):
    """Lengths span one-row and empty sequences, ragged 128-row query blocks and
    several 256-row GEMM tiles."""
    torch, ctx = env
    from paper_2608_01785_amd.device_data import prepare_dit_f16, upload_weights
    shape = W.DIT_TINY
    lengths = [1, 33, 0, 128, 300, 64, 257]
    layers, off, x, cond = _case(shape, 2, lengths, 91)
    wdev = upload_weights(layers)
    if fmt == "f16":
        wdev = prepare_dit_f16(ctx, wdev)
    log(f"[dit] tiny blocks x2, lengths {lengths}, weights {fmt}")
    got = run_dit(env, shape, wdev, x, cond, off).cpu().numpy().astype(np.float64)
    want = D.dit_forward(f64(x), cond.astype(np.float64), w64(layers), shape, off)
    e = err_ratio(got, want)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL


def test_dit_full_width_parity_and_budgets(env):
    """The bench's block shape (hidden 1024, 16 heads, MLP 4096), two 1024-token
    latents and a ragged one; every budget gives the same bits."""
    torch, ctx = env
    from paper_2608_01785_amd.device_data import prepare_dit_f16, upload_weights
    shape = W.DIT
    lengths = [1024, 257, 1024]
    layers, off, x, cond = _case(shape, 2, lengths, 92)
    wdev = prepare_dit_f16(ctx, upload_weights(layers))
    log(f"[dit] full-width blocks x2, lengths {lengths}")
    ys = [run_dit(env, shape, wdev, x, cond, off, down_cus=256 - b) for b in BUDGETS]
    for y in ys[1:]:
        assert torch.equal(ys[0], y)
    got = ys[0].cpu().numpy().astype(np.float64)
    want = D.dit_forward(f64(x), cond.astype(np.float64), w64(layers), shape, off)
    e = err_ratio(got, want)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL


def test_dit_zero_gates_return_the_input_exactly(env):
    torch, ctx = env
    from paper_2608_01785_amd.device_data import upload_weights
    shape = W.DIT_TINY
    layers, off, x, cond = _case(shape, 2, [70, 130], 93)
    for lw in layers:
        lw["w_ada"][:] = 0
        lw["b_ada"][:] = 0
    got = run_dit(env, shape, upload_weights(layers), x, cond, off).cpu().numpy().astype(np.float64)
    np.testing.assert_array_equal(got, f64(x))


def test_dit_attention_is_bidirectional_and_sequence_local(env):
    torch, ctx = env
    from paper_2608_01785_amd.device_data import upload_weights
    shape = W.DIT_TINY
    layers, off, x, cond = _case(shape, 1, [200, 150], 94)
    wdev = upload_weights(layers)
    y = run_dit(env, shape, wdev, x, cond, off).cpu().numpy()
    x2 = x.copy()
    x2[199] = W.token_rows(95, 1, shape.hidden)[0]   # the last token of sequence 0
    y2 = run_dit(env, shape, wdev, x2, cond, off).cpu().numpy()
    assert np.max(np.abs(y2[0] - y[0])) > 0          # a causal mask would leave row 0 unchanged
    np.testing.assert_array_equal(y2[200:], y[200:])  # sequence 1 sees nothing of sequence 0


def test_dit_token_permutation_permutes_outputs(env):
    torch, ctx = env
    from paper_2608_01785_amd.device_data import upload_weights
    shape = W.DIT_TINY
    layers, off, x, cond = _case(shape, 1, [190], 96)
    wdev = upload_weights(layers)
    perm = np.random.default_rng(97).permutation(190)
    y = run_dit(env, shape, wdev, x, cond, off).cpu().numpy().astype(np.float64)
    yp = run_dit(env, shape, wdev, x[perm], cond, off).cpu().numpy().astype(np.float64)
    assert err_ratio(yp, y[perm]) <= TOL


def test_dit_modulation_batches_across_blocks(env):
    """Nine blocks (the modulation runs for up to eight blocks per launch, so the
    ninth takes a second launch and the first slot again) over eleven sequences,
    one of them empty, at hidden 512 (two 16-byte chunks per lane)."""
    torch, ctx = env
    from paper_2608_01785_amd.device_data import upload_weights
    shape = W.DitShape(512, 8, 64, 1024)
    lengths = [5, 0, 40, 1, 17, 64, 3, 29, 8, 2, 11]
    layers, off, x, cond = _case(shape, 9, lengths, 98)
    log(f"[dit] hidden 512, 9 blocks, {len(lengths)} sequences")
    got = run_dit(env, shape, upload_weights(layers), x, cond, off).cpu().numpy().astype(np.float64)
    want = D.dit_forward(f64(x), cond.astype(np.float64), w64(layers), shape, off)
    e = err_ratio(got, want)
    log(f"  max err / rms = {e:.3e}")
    assert e <= TOL
