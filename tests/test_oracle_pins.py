"""Pins of the float64 reference against closed forms, library routines, invariants
and brute force on tiny inputs.  CPU only.

Each test names the kind of mistake it is there to catch.
"""
import cmath
import math
from types import SimpleNamespace

import numpy as np
import pytest
import scipy.special

from oracle import layer as L
from oracle import partition as P
from paper_2608_01785_amd import workloads as W
from tests.util import f64, weights_f64, as_bf16_f64


def cfg(d=16, hq=4, hkv=2, dh=4, f=12, eps=1e-6, base=10000.0):
    return SimpleNamespace(hidden=d, n_q_heads=hq, n_kv_heads=hkv, head_dim=dh, ffn=f,
                           rms_eps=eps, rope_base=base)


def rand_weights(c, rng, std=0.3, gamma_std=0.1):
    d, f, hq, hkv, dh = c.hidden, c.ffn, c.n_q_heads, c.n_kv_heads, c.head_dim
    return {
        "ln1": 1.0 + gamma_std * rng.standard_normal(d),
        "w_qkv": std * rng.standard_normal(((hq + 2 * hkv) * dh, d)),
        "w_o": std * rng.standard_normal((d, hq * dh)),
        "ln2": 1.0 + gamma_std * rng.standard_normal(d),
        "w_gate_up": std * rng.standard_normal((2 * f, d)),
        "w_down": std * rng.standard_normal((d, f)),
    }


# ----------------------------------------------------------------------------- RMSNorm

@pytest.mark.parametrize("c", [1.0, -2.5, 1e-3, 0.0])
def test_rmsnorm_constant_row_closed_form(c):
    # Catches eps outside the root, a missing mean (sum instead), or a dropped gamma.
    d, eps = 64, 1e-6
    gamma = np.linspace(0.5, 1.5, d)
    y = L.rms_norm(np.full((1, d), c), gamma, eps)
    expect = gamma * c / math.sqrt(c * c + eps)
    np.testing.assert_allclose(y[0], expect, rtol=1e-14, atol=0)


def test_rmsnorm_output_rms():
    # RMS(y / gamma) = sqrt(ms / (ms + eps)) for any row.
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 48)) * np.array([1e-3, 0.1, 1, 10, 100])[:, None]
    gamma = 1 + 0.1 * rng.standard_normal(48)
    eps = 1e-6
    y = L.rms_norm(x, gamma, eps)
    ms = np.mean(x * x, axis=1)
    got = np.sqrt(np.mean((y / gamma) ** 2, axis=1))
    np.testing.assert_allclose(got, np.sqrt(ms / (ms + eps)), rtol=1e-13)


# ----------------------------------------------------------------------------- SiLU / softmax

def test_silu_matches_library_logistic():
    z = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(L.silu(z), z * scipy.special.expit(z), rtol=1e-13, atol=1e-300)
    assert L.silu(np.array([0.0]))[0] == 0.0


def test_softmax_rows_library_shift_and_sum():
    rng = np.random.default_rng(1)
    s = rng.standard_normal((7, 33)) * 5
    p = L.softmax_rows(s)
    np.testing.assert_allclose(p, scipy.special.softmax(s, axis=-1), rtol=1e-13)
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=1e-14)
    np.testing.assert_allclose(L.softmax_rows(s + 123.0), p, rtol=1e-12)
    # Max subtraction: logits near 1000 would overflow exp() without it.
    big = np.array([[1000.0, 999.0, -np.inf]])
    pb = L.softmax_rows(big)
    assert np.all(np.isfinite(pb))
    np.testing.assert_allclose(pb[0, :2], [1 / (1 + math.e ** -1), 1 / (1 + math.e)], rtol=1e-13)
    assert pb[0, 2] == 0.0


# ----------------------------------------------------------------------------- RoPE

@pytest.mark.parametrize("dh", [2, 8, 64])
def test_rope_is_complex_rotation(dh):
    # Independent formulation: pair (j, j+dh/2) as the complex number x_j + i x_{j+dh/2},
    # multiplied by exp(i * pos * base^(-2j/dh)).  Catches sign, pairing and frequency errors.
    rng = np.random.default_rng(dh)
    T, H, base = 9, 3, 10000.0
    x = rng.standard_normal((T, H, dh))
    pos = rng.integers(0, 5000, size=T)
    y = L.rope(x, pos, base)
    half = dh // 2
    for t in range(T):
        for h in range(H):
            for j in range(half):
                z = complex(x[t, h, j], x[t, h, j + half])
                w = z * cmath.exp(1j * pos[t] * base ** (-2.0 * j / dh))
                assert abs(y[t, h, j] - w.real) < 1e-12 * max(1.0, abs(z))
                assert abs(y[t, h, j + half] - w.imag) < 1e-12 * max(1.0, abs(z))


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(3)
    dh = 16
    q = rng.standard_normal((1, 1, dh))
    k = rng.standard_normal((1, 1, dh))
    np.testing.assert_array_equal(L.rope(q, np.array([0]), 1e4), q)
    r = L.rope(q, np.array([1234]), 1e4)
    np.testing.assert_allclose(np.linalg.norm(r), np.linalg.norm(q), rtol=1e-13)
    # q(p) . k(p') depends on p - p' only.
    dots = []
    for p0 in (0, 17, 4000):
        qa = L.rope(q, np.array([p0 + 5]), 1e4)
        ka = L.rope(k, np.array([p0]), 1e4)
        dots.append(float(np.sum(qa * ka)))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-10)


# ----------------------------------------------------------------------------- attention

def test_attention_single_key_returns_value():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((1, 4, 8))
    k = rng.standard_normal((1, 2, 8))
    v = rng.standard_normal((1, 2, 8))
    o = L.attention_one_sequence(q, k, v, 0)
    for h in range(4):
        np.testing.assert_array_equal(o[0, h], v[0, h // 2])


def test_attention_identical_keys_give_causal_running_mean():
    # All keys equal -> uniform weights over the visible prefix.  Catches an off-by-one
    # in the causal mask (diagonal excluded or one future key included) and prefix offsets.
    rng = np.random.default_rng(5)
    ctx, Lq, dh = 3, 6, 8
    q = rng.standard_normal((Lq, 2, dh))
    k = np.tile(rng.standard_normal((1, 1, dh)), (ctx + Lq, 1, 1))
    v = rng.standard_normal((ctx + Lq, 1, dh))
    o = L.attention_one_sequence(q, k, v, ctx)
    for i in range(Lq):
        mean = v[: ctx + i + 1, 0].mean(axis=0)
        np.testing.assert_allclose(o[i, 0], mean, rtol=1e-12)
        np.testing.assert_allclose(o[i, 1], mean, rtol=1e-12)


def test_attention_two_keys_logistic_weight():
    # Two visible keys with scores 0 and a*b/sqrt(dh): weights are the logistic function.
    # Catches a missing or wrong 1/sqrt(dh) scale.
    dh, a, b = 4, 3.0, 1.5
    q = np.zeros((2, 1, dh)); q[1, 0, 0] = a
    k = np.zeros((2, 1, dh)); k[1, 0, 0] = b
    v = np.zeros((2, 1, dh)); v[0, 0, 1] = 1.0; v[1, 0, 2] = 1.0
    o = L.attention_one_sequence(q, k, v, 0)
    w1 = scipy.special.expit(a * b / math.sqrt(dh))
    np.testing.assert_allclose(o[1, 0], [0, 1 - w1, w1, 0], rtol=1e-14, atol=1e-16)
    np.testing.assert_allclose(o[0, 0], v[0, 0])


def test_attention_gqa_groups_are_contiguous():
    # KV head g serves query heads g*G .. g*G+G-1 (not h % Hkv).
    Lq, hq, hkv, dh = 5, 6, 3, 4
    rng = np.random.default_rng(6)
    q = rng.standard_normal((Lq, hq, dh))
    k = rng.standard_normal((Lq, hkv, dh))
    v = np.zeros((Lq, hkv, dh))
    for g in range(hkv):
        v[:, g, :] = g + 1.0
    o = L.attention_one_sequence(q, k, v, 0)
    for h in range(hq):
        np.testing.assert_allclose(o[:, h, :], h // (hq // hkv) + 1.0, rtol=1e-14)


# ----------------------------------------------------------------------------- whole layer

def brute_force_layer(x, w, c, offsets, ctx_lens=None, pk=None, pv=None):
    """Element-by-element loops with math.* scalars (tiny inputs only)."""
    T, d = len(x), c.hidden
    hq, hkv, dh, f = c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn
    B = len(offsets) - 1
    ctx = [0] * B if ctx_lens is None else list(ctx_lens)

    def norm(row, g):
        ms = sum(v * v for v in row) / d
        r = 1.0 / math.sqrt(ms + c.rms_eps)
        return [row[j] * r * g[j] for j in range(d)]

    def matvec(W, vec):
        return [sum(W[o][i] * vec[i] for i in range(len(vec))) for o in range(len(W))]

    def rot(vec, p):
        half = dh // 2
        out = list(vec)
        for j in range(half):
            th = p * c.rope_base ** (-2.0 * j / dh)
            out[j] = vec[j] * math.cos(th) - vec[j + half] * math.sin(th)
            out[j + half] = vec[j + half] * math.cos(th) + vec[j] * math.sin(th)
        return out

    y = []
    for b in range(B):
        rows = list(range(offsets[b], offsets[b + 1]))
        qs, ks, vs = [], [], []
        for i, t in enumerate(rows):
            n = norm(list(x[t]), w["ln1"])
            qkv = matvec(w["w_qkv"], n)
            if w.get("b_qkv") is not None:
                qkv = [v + w["b_qkv"][o] for o, v in enumerate(qkv)]
            p = ctx[b] + i
            qs.append([rot(qkv[h * dh:(h + 1) * dh], p) for h in range(hq)])
            ks.append([rot(qkv[(hq + g) * dh:(hq + g + 1) * dh], p) for g in range(hkv)])
            vs.append([qkv[(hq + hkv + g) * dh:(hq + hkv + g + 1) * dh] for g in range(hkv)])
        allk = [[list(pk[b][j][g]) for g in range(hkv)] for j in range(ctx[b])] + ks
        allv = [[list(pv[b][j][g]) for g in range(hkv)] for j in range(ctx[b])] + vs
        for i, t in enumerate(rows):
            o = []
            for h in range(hq):
                g = h * hkv // hq
                sc = [sum(qs[i][h][e] * allk[j][g][e] for e in range(dh)) / math.sqrt(dh)
                      for j in range(ctx[b] + i + 1)]
                mx = max(sc)
                ex = [math.exp(s - mx) for s in sc]
                den = sum(ex)
                o += [sum(ex[j] * allv[j][g][e] for j in range(len(ex))) / den for e in range(dh)]
            hres = [x[t][j] + v for j, v in enumerate(matvec(w["w_o"], o))]
            m = norm(hres, w["ln2"])
            gu = matvec(w["w_gate_up"], m)
            a = [gu[j] / (1 + math.exp(-gu[j])) * gu[f + j] for j in range(f)]
            y.append([hres[j] + v for j, v in enumerate(matvec(w["w_down"], a))])
    return np.array(y)


def test_layer_matches_brute_force_loops():
    # Catches transposed projections, a wrong q/k/v split, GQA index, misplaced residuals.
    c = cfg(d=12, hq=4, hkv=2, dh=6, f=10)
    rng = np.random.default_rng(7)
    w = rand_weights(c, rng)
    off = [0, 3, 8]
    x = rng.standard_normal((8, 12))
    got, _, _ = L.layer_forward(x, w, c, off)
    ref = brute_force_layer(x, w, c, off)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)


def test_layer_with_qkv_bias_matches_brute_force_loops():
    c = cfg(d=8, hq=2, hkv=1, dh=4, f=6)
    rng = np.random.default_rng(18)
    w = rand_weights(c, rng)
    w["b_qkv"] = rng.standard_normal((c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim)
    off, ctx = [0, 2, 5], [3, 1]
    pk = [rng.standard_normal((n, 1, 4)) for n in ctx]
    pv = [rng.standard_normal((n, 1, 4)) for n in ctx]
    x = rng.standard_normal((5, 8))
    got, _, _ = L.layer_forward(x, w, c, off, ctx, pk, pv)
    ref = brute_force_layer(x, w, c, off, ctx, pk, pv)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)


def test_qkv_bias_alone_gives_rotated_bias_keys_and_bias_values():
    # With W_qkv = 0 every row's key is RoPE(b_k) at its position and its value is b_v.
    c = cfg(d=8, hq=2, hkv=1, dh=4, f=6)
    rng = np.random.default_rng(19)
    w = rand_weights(c, rng)
    w["w_qkv"] = np.zeros_like(w["w_qkv"])
    b = rng.standard_normal((c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim)
    w["b_qkv"] = b
    x = rng.standard_normal((5, 8))
    _, k, v = L.layer_forward(x, w, c, [0, 5])
    bk, bv = b[8:12], b[12:16]
    for t in range(5):
        th = t * c.rope_base ** (-2.0 * np.arange(2) / 4)
        exp = np.concatenate([bk[:2] * np.cos(th) - bk[2:] * np.sin(th), bk[2:] * np.cos(th) + bk[:2] * np.sin(th)])
        np.testing.assert_allclose(k[t, 0], exp, rtol=1e-13, atol=1e-13)
        np.testing.assert_array_equal(v[t, 0], bv)
    w0 = dict(w, w_qkv=rand_weights(c, rng)["w_qkv"])
    y_none, _, _ = L.layer_forward(x, dict(w0, b_qkv=None), c, [0, 5])
    y_zero, _, _ = L.layer_forward(x, dict(w0, b_qkv=np.zeros_like(b)), c, [0, 5])
    np.testing.assert_array_equal(y_none, y_zero)


def test_layer_with_prefix_matches_brute_force_loops():
    c = cfg(d=8, hq=2, hkv=1, dh=4, f=6)
    rng = np.random.default_rng(8)
    w = rand_weights(c, rng)
    off, ctx = [0, 2, 5], [3, 1]
    pk = [rng.standard_normal((n, 1, 4)) for n in ctx]
    pv = [rng.standard_normal((n, 1, 4)) for n in ctx]
    x = rng.standard_normal((5, 8))
    got, _, _ = L.layer_forward(x, w, c, off, ctx, pk, pv)
    ref = brute_force_layer(x, w, c, off, ctx, pk, pv)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)


def test_stack_chains_layers_like_brute_force_loops():
    # Catches a stack that feeds the original x (or the previous layer's input)
    # to every layer, reuses one layer's weights, or drops the last layer: the
    # brute-force loops are applied layer after layer, each on the previous
    # layer's output.
    c = cfg(d=12, hq=4, hkv=2, dh=6, f=10)
    rng = np.random.default_rng(21)
    layers = [rand_weights(c, rng) for _ in range(3)]
    off = [0, 3, 7]
    x = rng.standard_normal((7, 12))
    got, kv = L.stack_forward(x, layers, c, off)
    ref = x
    for w in layers:
        ref = brute_force_layer(ref, w, c, off)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)
    # Layers really differ: two layers are not one layer applied twice.
    twice = brute_force_layer(brute_force_layer(x, layers[0], c, off), layers[0], c, off)
    assert np.max(np.abs(L.stack_forward(x, layers[:2], c, off)[0] - twice)) > 1e-3
    # Keys of layer 1 come from layer 0's output, not from x.
    _, k1, _ = L.layer_forward(L.layer_forward(x, layers[0], c, off)[0], layers[1], c, off)
    np.testing.assert_allclose(kv[1][0], k1, rtol=1e-12, atol=1e-12)


def test_stack_with_per_layer_prefixes_matches_brute_force_loops():
    # Each layer reads its own cached prefix: a stack that handed layer 0's
    # prefix to every layer fails here.
    c = cfg(d=8, hq=2, hkv=1, dh=4, f=6)
    rng = np.random.default_rng(22)
    layers = [rand_weights(c, rng) for _ in range(2)]
    off, ctx = [0, 2, 5], [3, 1]
    pk = [[rng.standard_normal((n, 1, 4)) for n in ctx] for _ in range(2)]
    pv = [[rng.standard_normal((n, 1, 4)) for n in ctx] for _ in range(2)]
    x = rng.standard_normal((5, 8))
    got, _ = L.stack_forward(x, layers, c, off, ctx, pk, pv)
    ref = x
    for li, w in enumerate(layers):
        ref = brute_force_layer(ref, w, c, off, ctx, pk[li], pv[li])
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)
    # The decode step is that stack over one-row sequences.
    kv_lens = [4, 2]
    dk = [[rng.standard_normal((n, 1, 4)) for n in kv_lens] for _ in range(2)]
    dv = [[rng.standard_normal((n, 1, 4)) for n in kv_lens] for _ in range(2)]
    xd = rng.standard_normal((2, 8))
    yd, _ = L.decode_step(xd, layers, c, kv_lens, dk, dv)
    ref = xd
    for li, w in enumerate(layers):
        ref = brute_force_layer(ref, w, c, [0, 1, 2], kv_lens, dk[li], dv[li])
    np.testing.assert_allclose(yd, ref, rtol=1e-10, atol=1e-10)


def test_residual_identity():
    c = cfg()
    rng = np.random.default_rng(9)
    w = rand_weights(c, rng)
    w["w_o"][:] = 0
    w["w_down"][:] = 0
    x = rng.standard_normal((7, c.hidden))
    y, _, _ = L.layer_forward(x, w, c, [0, 7])
    np.testing.assert_array_equal(y, x)


def test_causal_invariance():
    c = cfg()
    rng = np.random.default_rng(10)
    w = rand_weights(c, rng)
    x = rng.standard_normal((12, c.hidden))
    y1, _, _ = L.layer_forward(x, w, c, [0, 12])
    x2 = x.copy()
    x2[7:] += rng.standard_normal((5, c.hidden))
    y2, _, _ = L.layer_forward(x2, w, c, [0, 12])
    np.testing.assert_allclose(y2[:7], y1[:7], rtol=1e-13, atol=1e-13)
    assert np.max(np.abs(y2[7:] - y1[7:])) > 1e-3


def test_sequence_permutation_equivariance():
    c = cfg()
    rng = np.random.default_rng(11)
    w = rand_weights(c, rng)
    lens = [3, 5, 2]
    x = rng.standard_normal((10, c.hidden))
    y, _, _ = L.layer_forward(x, w, c, [0, 3, 8, 10])
    perm = [2, 0, 1]
    segs = [x[0:3], x[3:8], x[8:10]]
    xp = np.concatenate([segs[p] for p in perm])
    offp = np.concatenate([[0], np.cumsum([lens[p] for p in perm])])
    yp, _, _ = L.layer_forward(xp, w, c, offp)
    ysegs = [y[0:3], y[3:8], y[8:10]]
    np.testing.assert_allclose(yp, np.concatenate([ysegs[p] for p in perm]), rtol=1e-13, atol=1e-13)


def test_gqa_equals_mha_with_duplicated_kv_weights():
    c = cfg(d=16, hq=4, hkv=2, dh=4, f=8)
    rng = np.random.default_rng(12)
    w = rand_weights(c, rng)
    x = rng.standard_normal((6, 16))
    y, _, _ = L.layer_forward(x, w, c, [0, 6])
    dh, hq, hkv = 4, 4, 2
    wq = w["w_qkv"][: hq * dh]
    wk = w["w_qkv"][hq * dh:(hq + hkv) * dh].reshape(hkv, dh, 16)
    wv = w["w_qkv"][(hq + hkv) * dh:].reshape(hkv, dh, 16)
    wk_full = np.repeat(wk, hq // hkv, axis=0).reshape(hq * dh, 16)
    wv_full = np.repeat(wv, hq // hkv, axis=0).reshape(hq * dh, 16)
    w2 = dict(w, w_qkv=np.concatenate([wq, wk_full, wv_full]))
    y2, _, _ = L.layer_forward(x, w2, cfg(d=16, hq=4, hkv=4, dh=4, f=8), [0, 6])
    np.testing.assert_allclose(y2, y, rtol=1e-13, atol=1e-13)


def test_chunked_prefill_equals_whole_sequence():
    c = cfg()
    rng = np.random.default_rng(13)
    w = rand_weights(c, rng)
    x = rng.standard_normal((11, c.hidden))
    y, _, _ = L.layer_forward(x, w, c, [0, 11])
    _, k0, v0 = L.layer_forward(x[:4], w, c, [0, 4])
    y1, _, _ = L.layer_forward(x[4:], w, c, [0, 7], [4], [k0], [v0])
    np.testing.assert_allclose(y1, y[4:], rtol=1e-12, atol=1e-12)


def test_decode_equals_prefill_row():
    c = cfg()
    rng = np.random.default_rng(14)
    layers = [rand_weights(c, rng) for _ in range(2)]
    x = rng.standard_normal((6, c.hidden))
    y, kv = L.stack_forward(x, layers, c, [0, 6])
    # Cache of the first 5 rows from the prefill, then decode row 5.
    _, kv5 = L.stack_forward(x[:5], layers, c, [0, 5])
    ck = [[kv5[l][0]] for l in range(2)]
    cv = [[kv5[l][1]] for l in range(2)]
    yd, kvd = L.decode_step(x[5:6], layers, c, [5], ck, cv)
    np.testing.assert_allclose(yd[0], y[5], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(kvd[1][0][0], kv[1][0][5], rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------------------------- integer side

def test_plan_metadata_small():
    pos, sid = P.plan_metadata([0, 2, 2, 5], [3, 0, 7])
    assert pos.tolist() == [3, 4, 7, 8, 9]
    assert sid.tolist() == [0, 0, 2, 2, 2]
    with pytest.raises(ValueError):
        P.plan_metadata([1, 2])
    with pytest.raises(ValueError):
        P.plan_metadata([0, 3, 2])


@pytest.mark.parametrize("c", [1, 7, 8, 64, 96, 128, 160, 192, 255, 256])
def test_partition_properties(c):
    xcc, se, cu = P.default_topology()
    sh, dn = P.cu_partition(xcc, se, cu, 8, c)
    popc = lambda ws: sum(bin(w).count("1") for w in ws)
    assert popc(sh) == c and popc(dn) == 256 - c
    assert all((a & b) == 0 for a, b in zip(sh, dn))
    assert all((a | b) == 0xFFFFFFFF for a, b in zip(sh, dn))
    per_xcd = [0] * 8
    for i in range(256):
        if sh[i // 32] >> (i % 32) & 1:
            per_xcd[xcc[i]] += 1
    assert max(per_xcd) - min(per_xcd) <= 1
    if c < 256:  # nested ladder: a larger budget only adds CUs
        sh2, _ = P.cu_partition(xcc, se, cu, 8, c + 1)
        assert all((a & ~b) == 0 for a, b in zip(sh, sh2))


def test_partition_half_split_default_topology():
    # Default topology puts slot j = i // 8 of every XCD at bit i; half the budget takes
    # slots 0..15 of each XCD, i.e. bits 0..127.
    xcc, se, cu = P.default_topology()
    sh, dn = P.cu_partition(xcc, se, cu, 8, 128)
    assert sh == [0xFFFFFFFF] * 4 + [0] * 4
    assert dn == [0] * 4 + [0xFFFFFFFF] * 4


@pytest.mark.parametrize("c", [0, -1, 257])
def test_partition_rejects_out_of_range(c):
    xcc, se, cu = P.default_topology()
    with pytest.raises(P.PartitionError):
        P.cu_partition(xcc, se, cu, 8, c)


# ----------------------------------------------------------------------------- generator

def test_generator_recipe_lengths():
    b = W.thinker_batch(hidden=8)
    assert b.lengths.tolist() == [849, 1901, 953, 1744, 873, 1679, 970, 1546]
    assert b.seq_offsets.tolist() == [0, 849, 2750, 3703, 5447, 6320, 7999, 8969, 10515]
    assert b.n_image.tolist() == [277, 1090, 464, 747, 387, 757, 456, 468]
    kv = W.talker_kv_lens(32, W.SEEDS["talker"]["cache"])
    assert int(kv.sum()) == 17437 and int(kv.min()) == 159 and int(kv.max()) == 1022
    assert int(W.talker_kv_lens(128, W.SEEDS["talker_mixed"]["cache"]).sum()) == 75820


def test_bf16_rounding_is_nearest_even():
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -3.14159, 65504.0], np.float32)
    got = W.bf16_to_f32(W.bf16_bits(vals))
    # 1+2^-8 is a tie -> even (1.0); 1+3*2^-8 tie -> 1+2^-6... (even mantissa)
    assert got[0] == 1.0 and got[1] == 1.0 and got[2] == np.float32(1.0 + 2 ** -6)
    assert got[3] == 1.0
    assert abs(got[4] - -3.140625) < 1e-7
    w = W.make_weights(W.TINY, 1, 1000)[0]
    assert w["w_qkv"].shape == (512, 256) and w["w_gate_up"].shape == (2048, 256)
    assert abs(f64(w["ln1"]).mean() - 1.0) < 0.01
    assert abs(f64(w["w_qkv"]).std() - 0.02) < 0.001


def test_qkv_bias_draw_leaves_other_weights_unchanged():
    plain = W.make_weights(W.TINY, 2, 1000)
    biased = W.make_weights(W.TINY, 2, 1000, qkv_bias_std=0.5)
    for p_, b_ in zip(plain, biased):
        assert "b_qkv" not in p_ and b_["b_qkv"].shape == (W.TINY.qkv_rows,)
        for name in W.WEIGHT_NAMES:
            np.testing.assert_array_equal(p_[name], b_[name])
    assert abs(f64(biased[0]["b_qkv"]).std() - 0.5) < 0.05
    assert not np.array_equal(biased[0]["b_qkv"], biased[1]["b_qkv"])


def test_tiny_workload_layer_is_finite_and_row_local_residual():
    # End-to-end on the tiny workload's real inputs (the parity case of the GPU tests).
    c = W.TINY
    w = weights_f64(W.make_weights(c, 1, W.SEEDS["tiny"]["weights"]))[0]
    b = W.tiny_batch()
    y, k, v = L.layer_forward(f64(b.x), w, c, b.seq_offsets)
    assert y.shape == (224, 256) and np.all(np.isfinite(y))
    # The first row of each sequence attends to itself only: o = v row.
    for s in range(2):
        t = int(b.seq_offsets[s])
        assert np.all(np.isfinite(v[t]))


# ----------------------------------------------------------------------------- multimodal RoPE

def test_mrope_with_equal_components_is_plain_rope():
    import dataclasses
    c = dataclasses.replace(W.TINY, mrope_sections=(8, 12, 12))
    w = weights_f64(W.make_weights(c, 1, 51))[0]
    b = W.random_batch(c.hidden, [40, 7], seed=52, ctx_lens=[0, 0])
    pos = np.concatenate([np.arange(40), np.arange(7)])
    y0, k0, _ = L.layer_forward(f64(b.x), w, c, b.seq_offsets)
    y1, k1, _ = L.layer_forward(f64(b.x), w, c, b.seq_offsets, positions3=np.stack([pos, pos, pos]))
    np.testing.assert_array_equal(y0, y1)
    np.testing.assert_array_equal(k0, k1)


def test_mrope_scores_depend_only_on_per_section_offsets():
    rng = np.random.default_rng(53)
    sec, dh = (16, 24, 24), 128
    q = rng.standard_normal((1, 1, dh))
    k = rng.standard_normal((1, 1, dh))
    pq, pk = np.array([[5], [9], [2]]), np.array([[1], [3], [7]])
    for shift in ([0, 0, 0], [11, -2, 40], [100, 100, 3]):
        s = np.array(shift)[:, None]
        qa = L.rope(q, pq + s, 1e4, sec)
        ka = L.rope(k, pk + s, 1e4, sec)
        base = (L.rope(q, pq, 1e4, sec) * L.rope(k, pk, 1e4, sec)).sum()
        assert abs((qa * ka).sum() - base) < 1e-9 * np.abs(q).sum() * np.abs(k).sum()


def test_mrope_pair_turns_by_its_sections_component():
    sec, dh, base = (4, 8, 4), 32, 1e4
    for j, comp in ((2, 0), (5, 1), (13, 2)):
        x = np.zeros((1, 1, dh))
        x[0, 0, j] = 1.0                                  # (a, b) = (1, 0) in pair j
        pos = np.zeros((3, 1))
        pos[comp, 0] = 7.0
        y = L.rope(x, pos, base, sec)
        ang = 7.0 * base ** (-2.0 * j / dh)
        assert y[0, 0, j] == pytest.approx(np.cos(ang), abs=1e-15)
        assert y[0, 0, j + dh // 2] == pytest.approx(np.sin(ang), abs=1e-15)
        pos_other = np.zeros((3, 1))
        pos_other[(comp + 1) % 3, 0] = 7.0                # another component moves: no turn
        y = L.rope(x, pos_other, base, sec)
        assert y[0, 0, j] == 1.0 and y[0, 0, j + dh // 2] == 0.0


def test_mrope_positions_layout():
    p = W.mrope_positions([70, 5], [40, 0], [10, 3], grid_w=8)
    assert p.shape == (3, 75)
    assert list(p[:, 0]) == [10, 10, 10] and list(p[:, 9]) == [10, 11, 11]    # patch 9: row 1, col 1
    assert list(p[:, 40]) == [18, 18, 18]                                     # text after a 5 x 8 grid
    assert list(p[:, 70]) == [3, 3, 3] and p.max() < 80
