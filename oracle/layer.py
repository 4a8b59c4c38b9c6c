"""Float64 reference of the shared-stage decoder layer.  TEST INFRASTRUCTURE ONLY.

The paper defines the two phases of an autoregressive transformer stage:
prefill processes the input context and builds the key/value cache, decode
re-reads weights and the accumulated cache for every new token (§2.1,
"Autoregressive transformers").  It leaves the model computation of its base
runtime unchanged (§5) and states no layer formula, so the layer below is the
standard pre-norm decoder layer, with these readings of unstated details:

* RMSNorm: ``x / sqrt(mean(x^2) + eps) * gamma``, eps inside the root.
* No biases, except an optional bias ``b_qkv`` [(Hq + 2 Hkv) dh] added to the
  QKV projection before RoPE (the thinker's model family carries one there;
  the paper is silent).  Residual after attention and after the FFN.  No
  final norm.
* ``w_qkv`` rows are [query heads | key heads | value heads], ``head_dim``
  rows per head; query head ``h`` reads key/value head ``h // (Hq / Hkv)``.
* RoPE rotates the pairs (j, j + dh/2), j < dh/2, by ``pos * base^(-2j/dh)``;
  positions restart at 0 per sequence and are offset by the cached prefix
  length.  Image/video-patch rows use the same 1-D positions as text rows,
  unless multimodal positions are given: then every row has a temporal,
  height and width position, the pairs are split into consecutive sections
  of ``cfg.mrope_sections`` pairs, and pair j turns by its section's
  component (the sectioned multimodal RoPE of the Qwen2-VL family; the paper
  does not define one).
* Attention scale ``1/sqrt(dh)``; causal alignment is bottom-right: row ``i``
  of a chunk behind ``c`` cached rows sees keys ``0 .. c + i``; sequences never
  see each other.
* SwiGLU: ``silu(m Wg^T) * (m Wu^T)``, ``w_gate_up`` rows are [gate | up].
* Decode is the single-row case of prefill with the cached length as prefix.

Everything is evaluated in float64 with no intermediate rounding; the inputs
are the exact bfloat16 values the GPU receives.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise RMSNorm: x / sqrt(mean_j x_j^2 + eps) * gamma."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gamma, dtype=np.float64)


def rope_angles(pos: np.ndarray, head_dim: int, base: float) -> np.ndarray:
    """theta[t, j] = pos[t] * base^(-2j/dh) for j < dh/2 (float64)."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = np.power(float(base), -2.0 * j / head_dim)
    return np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]


def rope_angles_sectioned(pos3: np.ndarray, head_dim: int, base: float, sections) -> np.ndarray:
    """theta[t, j] = pos3[c(j), t] * base^(-2j/dh), c(j) the section (0, 1, 2) holding pair j."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = np.power(float(base), -2.0 * j / head_dim)
    comp = np.repeat(np.arange(3), [int(n) for n in sections])       # [dh/2]
    p = np.asarray(pos3, dtype=np.float64)[comp, :].T                # [T, dh/2]
    return p * inv_freq[None, :]


def rope(x: np.ndarray, pos: np.ndarray, base: float, sections=None) -> np.ndarray:
    """Rotate-half RoPE on x[T, H, dh]: (a, b) -> (a cos - b sin, b cos + a sin).

    pos is [T], or [3, T] with ``sections`` (pairs per temporal / height / width section)."""
    x = np.asarray(x, dtype=np.float64)
    dh = x.shape[-1]
    half = dh // 2
    if sections is not None:
        th = rope_angles_sectioned(pos, dh, base, sections)[:, None, :]
    else:
        th = rope_angles(pos, dh, base)[:, None, :]      # [T, 1, dh/2]
    c, s = np.cos(th), np.sin(th)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Softmax over the last axis with max subtraction; -inf entries get weight 0."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attention_one_sequence(q: np.ndarray, k: np.ndarray, v: np.ndarray, ctx: int) -> np.ndarray:
    """Causal grouped-query attention for one sequence.

    q: [L, Hq, dh] (rows at positions ctx .. ctx+L-1); k, v: [ctx+L, Hkv, dh]
    (cached prefix followed by the chunk's own rows).  Returns [L, Hq, dh].
    """
    L, hq, dh = q.shape
    n_keys, hkv, _ = k.shape
    assert n_keys == ctx + L and hq % hkv == 0
    group = hq // hkv
    scale = 1.0 / np.sqrt(dh)
    rows = ctx + np.arange(L)[:, None]
    cols = np.arange(n_keys)[None, :]
    masked = cols > rows                                  # key after the query's position
    out = np.empty((L, hq, dh), dtype=np.float64)
    for h in range(hq):
        g = h // group
        s = (q[:, h, :] @ k[:, g, :].T) * scale
        s[masked] = -np.inf
        out[:, h, :] = softmax_rows(s) @ v[:, g, :]
    return out


def layer_forward(x: np.ndarray, w: Dict[str, np.ndarray], cfg, seq_offsets: Sequence[int],
                  ctx_lens: Optional[Sequence[int]] = None,
                  prefix_k: Optional[List[np.ndarray]] = None,
                  prefix_v: Optional[List[np.ndarray]] = None,
                  positions3: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One pre-norm decoder layer over a packed ragged batch.

    x: [T, d] float64; w: float64 weights ('ln1', 'w_qkv', 'w_o', 'ln2',
    'w_gate_up', 'w_down', optional 'b_qkv'); seq_offsets: [B+1]; ctx_lens: [B] cached rows per
    sequence (None = no prefix); prefix_k/v: per sequence [ctx_b, Hkv, dh].
    ``positions3`` [3, T], if given, are the rows' multimodal RoPE positions
    (``cfg.mrope_sections`` splits the pairs).  Returns (y [T, d], k_new [T, Hkv, dh], v_new [T, Hkv, dh]).
    """
    x = np.asarray(x, dtype=np.float64)
    T, d = x.shape
    hq, hkv, dh = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    off = [int(o) for o in seq_offsets]
    B = len(off) - 1
    ctx = [0] * B if ctx_lens is None else [int(c) for c in ctx_lens]

    pos = np.empty(T, dtype=np.int64)
    for b in range(B):
        pos[off[b]:off[b + 1]] = ctx[b] + np.arange(off[b + 1] - off[b])

    n = rms_norm(x, w["ln1"], cfg.rms_eps)
    qkv = n @ w["w_qkv"].T
    if w.get("b_qkv") is not None:
        qkv = qkv + np.asarray(w["b_qkv"], dtype=np.float64)
    q = qkv[:, : hq * dh].reshape(T, hq, dh)
    k = qkv[:, hq * dh: (hq + hkv) * dh].reshape(T, hkv, dh)
    v = qkv[:, (hq + hkv) * dh:].reshape(T, hkv, dh)
    if positions3 is not None:
        q = rope(q, positions3, cfg.rope_base, cfg.mrope_sections)
        k = rope(k, positions3, cfg.rope_base, cfg.mrope_sections)
    else:
        q = rope(q, pos, cfg.rope_base)
        k = rope(k, pos, cfg.rope_base)

    o = np.zeros((T, hq, dh), dtype=np.float64)
    for b in range(B):
        lo, hi = off[b], off[b + 1]
        if hi == lo:
            continue
        if ctx[b] > 0:
            kb = np.concatenate([np.asarray(prefix_k[b], np.float64), k[lo:hi]], axis=0)
            vb = np.concatenate([np.asarray(prefix_v[b], np.float64), v[lo:hi]], axis=0)
        else:
            kb, vb = k[lo:hi], v[lo:hi]
        o[lo:hi] = attention_one_sequence(q[lo:hi], kb, vb, ctx[b])

    h = x + o.reshape(T, hq * dh) @ w["w_o"].T
    m = rms_norm(h, w["ln2"], cfg.rms_eps)
    f = cfg.ffn
    gu = m @ w["w_gate_up"].T
    a = silu(gu[:, :f]) * gu[:, f:]
    y = h + a @ w["w_down"].T
    return y, k, v


def stack_forward(x: np.ndarray, layers: List[Dict[str, np.ndarray]], cfg, seq_offsets,
                  ctx_lens=None, prefix_k=None, prefix_v=None, positions3=None):
    """Layers applied in order; the output is the residual stream (no final norm).

    prefix_k/v, if given, are per layer lists of per-sequence prefixes.
    Returns (y, [(k_new, v_new) per layer]).
    """
    kv = []
    for li, w in enumerate(layers):
        pk = None if prefix_k is None else prefix_k[li]
        pv = None if prefix_v is None else prefix_v[li]
        x, k, v = layer_forward(x, w, cfg, seq_offsets, ctx_lens, pk, pv, positions3)
        kv.append((k, v))
    return x, kv


def decode_step(x: np.ndarray, layers, cfg, kv_lens, cache_k, cache_v, positions3=None):
    """One decode step: every row is a one-row sequence behind kv_lens[b] cached rows.

    cache_k/v: per layer, per sequence [kv_len_b, Hkv, dh].  The new row sits
    at position kv_lens[b] and attends to kv_lens[b] + 1 keys.  Returns
    (y [B, d], [(k_new [B, Hkv, dh], v_new) per layer]).  positions3 [3, B]: the new rows'
    multimodal RoPE positions (cfg.mrope_sections splits the pairs).
    """
    B = len(kv_lens)
    off = np.arange(B + 1)
    return stack_forward(x, layers, cfg, off, kv_lens, cache_k, cache_v, positions3=positions3)

