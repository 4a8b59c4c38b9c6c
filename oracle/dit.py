"""Float64 reference of a diffusion-transformer (DiT) denoising step.  TEST INFRASTRUCTURE ONLY.

The paper names diffusion transformers among the output-side generators of
omni models: they produce visual content by iterative denoising, a generation
loop distinct from autoregressive decode (§2.1, "Visual generators"), and an
image-output request enters such a generator as its downstream stage (§2.2).
It gives no block formula.  The block below is the adaptive-layer-norm DiT
block with zero-initialised gates ("adaLN-Zero") of the cited DiT design, over
a ragged batch of latent-token sequences (one image or audio chunk each), with
these readings of details the paper leaves open:

* Conditioning: each sequence b has one conditioning vector c_b [d] (the
  timestep and class/text embedding, already embedded).  Per layer,
  (shift1, scale1, gate1, shift2, scale2, gate2) = chunk6(silu(c_b) W_ada^T + b_ada).
* Block: h = LN(x) (1 + scale1) + shift1;  x = x + gate1 * (MHSA(h) W_o^T + b_o);
         h = LN(x) (1 + scale2) + shift2;  x = x + gate2 * (gelu(h W_1^T + b_1) W_2^T + b_2).
  LN has no affine parameters and eps = 1e-6 inside the root; gelu is the
  tanh form 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))).
* Attention is bidirectional within a sequence (every token sees every token
  of its own sequence, none of another), multi-head with Hq = Hkv, scale
  1/sqrt(dh); w_qkv rows are [query heads | key heads | value heads] with a
  bias b_qkv; no rotary embedding (positions enter with the token
  embeddings, before the blocks).
* A step is the block stack: patch embedding, the final projection and the
  sampler's update are outside it.

Everything is evaluated in float64 with no intermediate rounding.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np


def layer_norm(x: np.ndarray, eps: float) -> np.ndarray:
    """(x - mean) / sqrt(var + eps) over the last axis, no affine parameters."""
    x = np.asarray(x, dtype=np.float64)
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def gelu_tanh(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    return 0.5 * z * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (z + 0.044715 * z ** 3)))


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def modulation(c: np.ndarray, w_ada: np.ndarray, b_ada: np.ndarray) -> np.ndarray:
    """[B, 6, d]: shift1, scale1, gate1, shift2, scale2, gate2 of every sequence."""
    c = np.asarray(c, dtype=np.float64)
    m = silu(c) @ np.asarray(w_ada, np.float64).T + np.asarray(b_ada, np.float64)
    return m.reshape(c.shape[0], 6, -1)


def attention_bidirectional(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """q, k, v [L, H, dh] of one sequence; every query attends to every key."""
    L, H, dh = q.shape
    out = np.empty_like(q)
    for h in range(H):
        s = (q[:, h, :] @ k[:, h, :].T) / np.sqrt(dh)
        s = s - np.max(s, axis=-1, keepdims=True)
        p = np.exp(s)
        p = p / np.sum(p, axis=-1, keepdims=True)
        out[:, h, :] = p @ v[:, h, :]
    return out


def dit_block(x: np.ndarray, c: np.ndarray, w: Dict[str, np.ndarray], cfg, seq_offsets: Sequence[int]) -> np.ndarray:
    """One adaLN-Zero block over a packed ragged batch.

    x: [T, d]; c: [B, d] conditioning per sequence; seq_offsets [B + 1]."""
    x = np.asarray(x, dtype=np.float64)
    T, d = x.shape
    H, dh = cfg.n_heads, cfg.head_dim
    off = [int(o) for o in seq_offsets]
    mod = modulation(c, w["w_ada"], w["b_ada"])
    seq = np.empty(T, dtype=np.int64)
    for b in range(len(off) - 1):
        seq[off[b]:off[b + 1]] = b
    shift1, scale1, gate1 = mod[seq, 0], mod[seq, 1], mod[seq, 2]
    shift2, scale2, gate2 = mod[seq, 3], mod[seq, 4], mod[seq, 5]

    h = layer_norm(x, cfg.ln_eps) * (1.0 + scale1) + shift1
    qkv = h @ w["w_qkv"].T + w["b_qkv"]
    q = qkv[:, :H * dh].reshape(T, H, dh)
    k = qkv[:, H * dh:2 * H * dh].reshape(T, H, dh)
    v = qkv[:, 2 * H * dh:].reshape(T, H, dh)
    o = np.zeros((T, H, dh))
    for b in range(len(off) - 1):
        lo, hi = off[b], off[b + 1]
        if hi > lo:
            o[lo:hi] = attention_bidirectional(q[lo:hi], k[lo:hi], v[lo:hi])
    x = x + gate1 * (o.reshape(T, H * dh) @ w["w_o"].T + w["b_o"])

    h = layer_norm(x, cfg.ln_eps) * (1.0 + scale2) + shift2
    a = gelu_tanh(h @ w["w_fc1"].T + w["b_fc1"])
    return x + gate2 * (a @ w["w_fc2"].T + w["b_fc2"])


def dit_forward(x: np.ndarray, c: np.ndarray, layers: List[Dict[str, np.ndarray]], cfg, seq_offsets) -> np.ndarray:
    """The block stack of one denoising step, blocks in order."""
    for w in layers:
        x = dit_block(x, c, w, cfg, seq_offsets)
    return x
