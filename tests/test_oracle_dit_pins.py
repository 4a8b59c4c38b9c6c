"""Pins of the float64 DiT-block reference (oracle/dit.py) against closed forms,
library routines, invariants and brute-force loops on tiny inputs.  CPU only.

Each test names the kind of mistake it is there to catch.
"""
import math
from types import SimpleNamespace

import numpy as np
import pytest
import scipy.special

from oracle import dit as D


def cfg(d=8, heads=2, dh=4, mlp=16, eps=1e-6):
    return SimpleNamespace(hidden=d, n_heads=heads, head_dim=dh, mlp=mlp, ln_eps=eps)


def rand_weights(c, rng, std=0.3):
    d, m, H, dh = c.hidden, c.mlp, c.n_heads, c.head_dim
    return {
        "w_ada": std * rng.standard_normal((6 * d, d)), "b_ada": std * rng.standard_normal(6 * d),
        "w_qkv": std * rng.standard_normal((3 * H * dh, d)), "b_qkv": std * rng.standard_normal(3 * H * dh),
        "w_o": std * rng.standard_normal((d, H * dh)), "b_o": std * rng.standard_normal(d),
        "w_fc1": std * rng.standard_normal((m, d)), "b_fc1": std * rng.standard_normal(m),
        "w_fc2": std * rng.standard_normal((d, m)), "b_fc2": std * rng.standard_normal(d),
    }


# ----------------------------------------------------------------------------- pieces

def test_layer_norm_closed_form():
    # x = a + s u with u of zero mean and unit variance: LN(x) = s u / sqrt(s^2 + eps).
    # Catches a missing mean subtraction, eps outside the root, or a sum for the mean.
    u = np.array([1.0, -1.0, 1.0, -1.0, 1.0, -1.0])
    for a, s in ((3.0, 2.0), (-1e3, 1e-3), (0.0, 1.0)):
        eps = 1e-6
        got = D.layer_norm((a + s * u)[None, :], eps)[0]
        np.testing.assert_allclose(got, s * u / math.sqrt(s * s + eps), rtol=1e-9, atol=1e-12)


def test_layer_norm_of_a_constant_row_is_zero():
    np.testing.assert_array_equal(D.layer_norm(np.full((2, 5), 7.25), 1e-6), np.zeros((2, 5)))


def test_gelu_tanh_identities_and_erf_form():
    # gelu(z) - gelu(-z) = z exactly for the tanh form (catches a sign or a
    # dropped 0.5); within 1e-3 of the exact erf-based GELU (catches a wrong
    # constant such as sqrt(pi / 2)).
    z = np.linspace(-6, 6, 1201)
    np.testing.assert_allclose(D.gelu_tanh(z) - D.gelu_tanh(-z), z, rtol=0, atol=1e-12)
    exact = 0.5 * z * (1.0 + scipy.special.erf(z / math.sqrt(2.0)))
    assert np.max(np.abs(D.gelu_tanh(z) - exact)) < 1e-3
    assert D.gelu_tanh(np.array([0.0]))[0] == 0.0


def test_modulation_matches_loops_and_chunk_order():
    # Catches a transposed W_ada, SiLU applied after the linear map, or a wrong chunk order.
    rng = np.random.default_rng(1)
    B, d = 3, 4
    c = rng.standard_normal((B, d))
    w = rng.standard_normal((6 * d, d))
    b = rng.standard_normal(6 * d)
    mod = D.modulation(c, w, b)
    for bi in range(B):
        for j in range(6 * d):
            s = b[j] + sum((c[bi, k] / (1 + math.exp(-c[bi, k]))) * w[j, k] for k in range(d))
            assert abs(mod[bi, j // d, j % d] - s) < 1e-12


def test_bidirectional_attention_single_key_and_uniform():
    # One key returns its value; identical keys average all values (no causal mask).
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 2, 4))
    k = rng.standard_normal((1, 2, 4))
    v = rng.standard_normal((1, 2, 4))
    np.testing.assert_allclose(D.attention_bidirectional(q, k, v), v, rtol=1e-14)
    L = 5
    q = rng.standard_normal((L, 1, 4))
    k = np.repeat(rng.standard_normal((1, 1, 4)), L, axis=0)
    v = rng.standard_normal((L, 1, 4))
    got = D.attention_bidirectional(q, k, v)
    np.testing.assert_allclose(got, np.repeat(v.mean(axis=0, keepdims=True), L, axis=0), rtol=1e-12)


def test_bidirectional_attention_matches_library_softmax():
    rng = np.random.default_rng(3)
    q, k, v = (rng.standard_normal((6, 2, 4)) for _ in range(3))
    got = D.attention_bidirectional(q, k, v)
    for h in range(2):
        p = scipy.special.softmax(q[:, h] @ k[:, h].T / 2.0, axis=-1)
        np.testing.assert_allclose(got[:, h], p @ v[:, h], rtol=1e-12)


# ----------------------------------------------------------------------------- the block

def brute_block(x, c, w, cf, off):
    """The DiT block written with plain Python loops (tiny shapes only)."""
    T, d = len(x), len(x[0])
    H, dh, m = cf.n_heads, cf.head_dim, cf.mlp
    out = [list(r) for r in x]

    def ln(row):
        mu = sum(row) / d
        var = sum((v - mu) ** 2 for v in row) / d
        return [(v - mu) / math.sqrt(var + cf.ln_eps) for v in row]

    def silu(z):
        return z / (1 + math.exp(-z))

    def gelu(z):
        return 0.5 * z * (1 + math.tanh(math.sqrt(2 / math.pi) * (z + 0.044715 * z ** 3)))

    for b in range(len(off) - 1):
        rows = range(off[b], off[b + 1])
        mod = [w["b_ada"][j] + sum(silu(c[b][k]) * w["w_ada"][j][k] for k in range(d)) for j in range(6 * d)]
        sh1, sc1, g1, sh2, sc2, g2 = (mod[i * d:(i + 1) * d] for i in range(6))
        hs = {t: [ln(out[t])[j] * (1 + sc1[j]) + sh1[j] for j in range(d)] for t in rows}
        qkv = {t: [w["b_qkv"][o] + sum(hs[t][j] * w["w_qkv"][o][j] for j in range(d)) for o in range(3 * H * dh)]
               for t in rows}
        att = {}
        for t in rows:
            o_row = []
            for h in range(H):
                qv = qkv[t][h * dh:(h + 1) * dh]
                scores = [sum(qv[e] * qkv[s][H * dh + h * dh + e] for e in range(dh)) / math.sqrt(dh) for s in rows]
                mx = max(scores)
                ex = [math.exp(sc - mx) for sc in scores]
                tot = sum(ex)
                for e in range(dh):
                    o_row.append(sum(ex[i] / tot * qkv[s][2 * H * dh + h * dh + e] for i, s in enumerate(rows)))
            att[t] = o_row
        for t in rows:
            proj = [w["b_o"][o] + sum(att[t][j] * w["w_o"][o][j] for j in range(H * dh)) for o in range(d)]
            out[t] = [out[t][o] + g1[o] * proj[o] for o in range(d)]
        for t in rows:
            h2 = [ln(out[t])[j] * (1 + sc2[j]) + sh2[j] for j in range(d)]
            a = [gelu(w["b_fc1"][i] + sum(h2[j] * w["w_fc1"][i][j] for j in range(d))) for i in range(m)]
            y = [w["b_fc2"][o] + sum(a[i] * w["w_fc2"][o][i] for i in range(m)) for o in range(d)]
            out[t] = [out[t][o] + g2[o] * y[o] for o in range(d)]
    return np.array(out)


def test_block_matches_brute_force_loops():
    # Catches any dropped term, wrong chunk, transposed weight, missing bias or a causal mask.
    rng = np.random.default_rng(4)
    cf = cfg()
    w = rand_weights(cf, rng)
    off = [0, 3, 4, 7]
    x = rng.standard_normal((7, cf.hidden))
    c = rng.standard_normal((3, cf.hidden))
    got = D.dit_block(x, c, w, cf, off)
    ref = brute_block(x.tolist(), c.tolist(), {k: v.tolist() for k, v in w.items()}, cf, off)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)


def test_stack_chains_blocks_like_brute_force_loops():
    # Catches a stack that feeds the original input to every block.
    rng = np.random.default_rng(5)
    cf = cfg()
    layers = [rand_weights(cf, rng) for _ in range(2)]
    off = [0, 2, 5]
    x = rng.standard_normal((5, cf.hidden))
    c = rng.standard_normal((2, cf.hidden))
    ref = x.tolist()
    for w in layers:
        ref = brute_block(ref, c.tolist(), {k: v.tolist() for k, v in w.items()}, cf, off).tolist()
    np.testing.assert_allclose(D.dit_forward(x, c, layers, cf, off), np.array(ref), rtol=1e-10, atol=1e-10)


def test_zero_gates_make_the_block_the_identity():
    # adaLN-Zero: with W_ada = 0 and b_ada = 0 every gate is 0 and the block returns x exactly.
    rng = np.random.default_rng(6)
    cf = cfg()
    w = rand_weights(cf, rng)
    w["w_ada"][:] = 0.0
    w["b_ada"][:] = 0.0
    x = rng.standard_normal((6, cf.hidden))
    c = rng.standard_normal((2, cf.hidden))
    np.testing.assert_array_equal(D.dit_block(x, c, w, cf, [0, 4, 6]), x)


def test_attention_is_bidirectional():
    # Changing the last token of a sequence changes the first token's output
    # (it would not under a causal mask) and never another sequence's.
    rng = np.random.default_rng(7)
    cf = cfg()
    w = rand_weights(cf, rng)
    off = [0, 4, 9]
    x = rng.standard_normal((9, cf.hidden))
    c = rng.standard_normal((2, cf.hidden))
    y = D.dit_block(x, c, w, cf, off)
    x2 = x.copy()
    x2[3] += rng.standard_normal(cf.hidden)   # not a constant shift, which LN would remove
    y2 = D.dit_block(x2, c, w, cf, off)
    assert np.max(np.abs(y2[0] - y[0])) > 1e-6
    np.testing.assert_array_equal(y2[4:], y[4:])


def test_token_permutation_within_a_sequence_permutes_outputs():
    # No positions inside the block: permuting a sequence's tokens permutes its outputs.
    rng = np.random.default_rng(8)
    cf = cfg()
    w = rand_weights(cf, rng)
    x = rng.standard_normal((6, cf.hidden))
    c = rng.standard_normal((1, cf.hidden))
    perm = np.array([3, 0, 5, 1, 4, 2])
    y = D.dit_block(x, c, w, cf, [0, 6])
    yp = D.dit_block(x[perm], c, w, cf, [0, 6])
    np.testing.assert_allclose(yp, y[perm], rtol=1e-12, atol=1e-12)


def test_conditioning_is_per_sequence():
    # Swapping two sequences together with their conditioning swaps the outputs.
    rng = np.random.default_rng(9)
    cf = cfg()
    w = rand_weights(cf, rng)
    xa, xb = rng.standard_normal((3, cf.hidden)), rng.standard_normal((2, cf.hidden))
    ca, cb = rng.standard_normal(cf.hidden), rng.standard_normal(cf.hidden)
    y1 = D.dit_block(np.vstack([xa, xb]), np.vstack([ca, cb]), w, cf, [0, 3, 5])
    y2 = D.dit_block(np.vstack([xb, xa]), np.vstack([cb, ca]), w, cf, [0, 2, 5])
    np.testing.assert_allclose(y2[:2], y1[3:], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(y2[2:], y1[:3], rtol=1e-12, atol=1e-12)
