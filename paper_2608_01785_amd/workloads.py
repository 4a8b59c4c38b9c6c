"""Seeded synthetic inputs for the shared-stage layer and the talker decode step.

This module only draws random numbers and rounds them to bfloat16. It holds
none of the layer's arithmetic, so both the HIP path and the CPU reference can
consume its output without sharing any of the method's code.

Workloads (shapes of the omni-model traffic described in the paper's
motivation, §3.3, and its evaluation, §6.1; the paper's datasets are not
available, so every value is drawn from the recipes below):

* ``tiny``      - one decoder layer, hidden 256, 4 query / 2 key-value heads,
                  head_dim 64, FFN 1024; two sequences of 96 and 128 rows.
* ``thinker``   - four layers, hidden 3584, 28 / 4 heads, head_dim 128,
                  FFN 18944; eight prefill requests, lengths uniform in
                  [256, 2048], 30-70 % image-patch rows first, then text rows.
* ``talker``    - sixteen layers, hidden 1024, 16 / 16 heads, head_dim 64,
                  FFN 4096; a decode batch whose cached lengths are uniform in
                  [128, 1024].
* ``thinker_mixed`` - one layer, hidden 4096, 32 / 8 heads, head_dim 128,
                  FFN 14336; four 2048-row prefill chunks behind cached
                  prefixes of 0/2048/4096/6144 rows, plus 64 single-row decode
                  sequences behind 4096 cached rows.

Weights are N(0, 0.02); RMSNorm gains are 1 + N(0, 0.02); the optional QKV
bias (models of the Qwen2 family carry one) is N(0, sigma) with sigma chosen
by the caller; token embeddings and
cached keys/values are N(0, 1).  All values are drawn in float32 with NumPy's
PCG64 generator and rounded with round-to-nearest-even: to bfloat16 for
weights and token rows, to IEEE half for cached keys/values.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

# ----------------------------------------------------------------------------
# bfloat16 helpers (bit manipulation only)
# ----------------------------------------------------------------------------


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return raw uint16 bits.

    Inputs are finite by construction (the generators below never produce
    NaN or infinity).
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Expand raw bfloat16 bits to float32 (exact)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def f16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to IEEE half (nearest even); return raw uint16 bits."""
    return np.ascontiguousarray(a, dtype=np.float32).astype(np.float16).view(np.uint16)


def f16_to_f32(bits: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(bits, dtype=np.uint16).view(np.float16).astype(np.float32)


# ----------------------------------------------------------------------------
# Layer shapes
# ----------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class LayerShape:
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    mrope_sections: tuple = (0, 0, 0)   # temporal / height / width rotary pairs; zeros: plain RoPE

    @property
    def qkv_rows(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def params_per_layer(self) -> int:
        d, f = self.hidden, self.ffn
        return self.qkv_rows * d + d * self.n_q_heads * self.head_dim + 2 * f * d + d * f


TINY = LayerShape(256, 4, 2, 64, 1024)
THINKER = LayerShape(3584, 28, 4, 128, 18944)
TALKER = LayerShape(1024, 16, 16, 64, 4096)
THINKER_MIXED = LayerShape(4096, 32, 8, 128, 14336)

# Per-workload seeds: weights, token rows, lengths, decode caches.
SEEDS = {
    "tiny": dict(weights=1000, tokens=2000, lengths=3000, cache=4000),
    "thinker": dict(weights=1001, tokens=2001, lengths=3001, cache=4001),
    "talker": dict(weights=1003, tokens=2003, lengths=3003, cache=4003),
    "talker_mixed": dict(weights=1003, tokens=2004, lengths=3004, cache=4004),
    "thinker_mixed": dict(weights=1004, tokens=2004, lengths=3004, cache=5004),
}


# ----------------------------------------------------------------------------
# Weights
# ----------------------------------------------------------------------------

WEIGHT_NAMES = ("ln1", "w_qkv", "w_o", "ln2", "w_gate_up", "w_down")


def weight_shapes(s: LayerShape) -> Dict[str, tuple]:
    d, f = s.hidden, s.ffn
    return {
        "ln1": (d,),
        "w_qkv": (s.qkv_rows, d),
        "w_o": (d, s.n_q_heads * s.head_dim),
        "ln2": (d,),
        "w_gate_up": (2 * f, d),
        "w_down": (d, f),
    }


def make_weights(s: LayerShape, n_layers: int, seed: int, std: float = 0.02,
                 qkv_bias_std: float = 0.0) -> List[Dict[str, np.ndarray]]:
    """Per-layer dict of raw bf16 bits, drawn layer by layer in WEIGHT_NAMES order.

    ``w_qkv`` rows are [query heads | key heads | value heads], ``head_dim``
    rows each; ``w_gate_up`` rows are [gate | up]. Matrices are [out, in].
    With ``qkv_bias_std`` > 0 each layer also gets ``b_qkv`` [qkv_rows],
    N(0, qkv_bias_std), drawn afterwards from a generator of its own so that
    the other weights do not depend on whether biases are drawn.
    """
    rng = np.random.default_rng(seed)
    shapes = weight_shapes(s)
    layers = []
    for _ in range(n_layers):
        lw = {}
        for name in WEIGHT_NAMES:
            shp = shapes[name]
            v = rng.standard_normal(shp, dtype=np.float32)
            v *= np.float32(std)
            if name.startswith("ln"):
                v += np.float32(1.0)
            lw[name] = bf16_bits(v)
            del v
        layers.append(lw)
    if qkv_bias_std > 0.0:
        brng = np.random.default_rng([seed, 1])
        for lw in layers:
            v = brng.standard_normal(s.qkv_rows, dtype=np.float32)
            v *= np.float32(qkv_bias_std)
            lw["b_qkv"] = bf16_bits(v)
    return layers


# ----------------------------------------------------------------------------
# Ragged prefill batches
# ----------------------------------------------------------------------------


@dataclasses.dataclass
class PrefillBatch:
    lengths: np.ndarray          # int32 [B] query rows per sequence
    seq_offsets: np.ndarray      # int32 [B+1] packed row offsets
    ctx_lens: Optional[np.ndarray]  # int32 [B] cached rows before the chunk, or None
    n_image: np.ndarray          # int32 [B] leading image/video-patch rows (label only)
    x: np.ndarray                # uint16 [T, d] bf16 bits

    @property
    def n_tokens(self) -> int:
        return int(self.seq_offsets[-1])

    @property
    def n_seqs(self) -> int:
        return int(self.lengths.shape[0])


def _offsets(lengths: np.ndarray) -> np.ndarray:
    off = np.zeros(len(lengths) + 1, dtype=np.int32)
    off[1:] = np.cumsum(lengths, dtype=np.int64).astype(np.int32)
    return off


def draw_lengths(seed: int, n: int, lo: int, hi: int, frac_lo: float = 0.3, frac_hi: float = 0.7):
    """Lengths uniform in [lo, hi] and the leading image-row count per request."""
    rng = np.random.default_rng(seed)
    lengths = rng.integers(lo, hi, size=n, endpoint=True).astype(np.int32)
    frac = rng.uniform(frac_lo, frac_hi, size=n)
    n_img = np.floor(frac * lengths + 0.5).astype(np.int32)
    return lengths, n_img


def token_rows(seed: int, n_rows: int, hidden: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return bf16_bits(rng.standard_normal((n_rows, hidden), dtype=np.float32))


def tiny_batch(hidden: int = TINY.hidden, seed: int = SEEDS["tiny"]["tokens"],
               lengths=(96, 128)) -> PrefillBatch:
    lengths = np.asarray(lengths, dtype=np.int32)
    off = _offsets(lengths)
    return PrefillBatch(lengths, off, None, np.zeros_like(lengths), token_rows(seed, int(off[-1]), hidden))


def thinker_batch(hidden: int = THINKER.hidden, n_requests: int = 8,
                  seeds: Dict[str, int] = SEEDS["thinker"]) -> PrefillBatch:
    lengths, n_img = draw_lengths(seeds["lengths"], n_requests, 256, 2048)
    off = _offsets(lengths)
    return PrefillBatch(lengths, off, None, n_img, token_rows(seeds["tokens"], int(off[-1]), hidden))


def mrope_positions(lengths, n_img, ctx_lens=None, grid_w: int = 32) -> np.ndarray:
    """Multimodal RoPE positions [3, T] of packed sequences whose first n_img[b] rows are
    image patches: patch i sits at (t, h, w) = (s, s + i // grid_w, s + i % grid_w) with
    s = ctx_lens[b]; the text rows after it continue from the largest position + 1 with three
    equal components (the layout of the Qwen2-VL family)."""
    lengths = [int(n) for n in lengths]
    ctx = [0] * len(lengths) if ctx_lens is None else [int(c) for c in ctx_lens]
    out = np.zeros((3, sum(lengths)), np.int32)
    t0 = 0
    for n, k, s in zip(lengths, [int(i) for i in n_img], ctx):
        k = min(k, n)
        i = np.arange(k)
        out[0, t0:t0 + k] = s
        out[1, t0:t0 + k] = s + i // grid_w
        out[2, t0:t0 + k] = s + i % grid_w
        nxt = s + (max((k - 1) // grid_w, min(k, grid_w) - 1) + 1 if k else 0)
        out[:, t0 + k:t0 + n] = nxt + np.arange(n - k)
        t0 += n
    return out


def random_batch(hidden: int, lengths, seed: int, ctx_lens=None) -> PrefillBatch:
    lengths = np.asarray(lengths, dtype=np.int32)
    off = _offsets(lengths)
    ctx = None if ctx_lens is None else np.asarray(ctx_lens, dtype=np.int32)
    return PrefillBatch(lengths, off, ctx, np.zeros_like(lengths), token_rows(seed, int(off[-1]), hidden))


# ----------------------------------------------------------------------------
# Key/value caches
# ----------------------------------------------------------------------------


@dataclasses.dataclass
class CacheContents:
    """Cached keys/values in logical order: per layer, per slot, [ctx, Hkv, dh] fp16 bits."""
    k: List[List[np.ndarray]]
    v: List[List[np.ndarray]]


def make_cache(s: LayerShape, n_layers: int, ctx_lens, seed: int) -> CacheContents:
    rng = np.random.default_rng(seed)
    ks, vs = [], []
    for _ in range(n_layers):
        kl, vl = [], []
        for c in ctx_lens:
            shp = (int(c), s.n_kv_heads, s.head_dim)
            kl.append(f16_bits(rng.standard_normal(shp, dtype=np.float32)))
            vl.append(f16_bits(rng.standard_normal(shp, dtype=np.float32)))
        ks.append(kl)
        vs.append(vl)
    return CacheContents(ks, vs)


@dataclasses.dataclass
class DecodeBatch:
    kv_lens: np.ndarray   # int32 [B] cached rows before the step
    x: np.ndarray         # uint16 [B, d]
    cache: Optional[CacheContents]


def talker_kv_lens(batch: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(128, 1024, size=batch, endpoint=True).astype(np.int32)


def talker_batch(s: LayerShape, n_layers: int, batch: int, seeds: Dict[str, int],
                 step: int = 0, with_cache: bool = True) -> DecodeBatch:
    """Decode rows for one talker step.

    Step ``step`` draws fresh N(0, 1) rows with seed (tokens seed, step); the
    cache prefix is drawn from the cache seed (after the kv lengths).
    """
    kv = talker_kv_lens(batch, seeds["cache"])
    x = bf16_bits(np.random.default_rng([seeds["tokens"], step]).standard_normal(
        (batch, s.hidden), dtype=np.float32))
    cache = make_cache(s, n_layers, kv, seeds["cache"] + 7919) if with_cache else None
    return DecodeBatch(kv, x, cache)


def thinker_mixed_layout(n_chunks: int = 4, chunk: int = 2048, n_decode: int = 64, decode_ctx: int = 4096):
    """Lengths and cached-prefix lengths of the mixed chunked-prefill + decode step."""
    lengths = [chunk] * n_chunks + [1] * n_decode
    ctx = [chunk * i for i in range(n_chunks)] + [decode_ctx] * n_decode
    return np.asarray(lengths, np.int32), np.asarray(ctx, np.int32)


# ----------------------------------------------------------------------------
# Diffusion-transformer (DiT) denoising step: the image / audio generator
# downstream stage
# ----------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class DitShape:
    hidden: int
    n_heads: int
    head_dim: int
    mlp: int
    ln_eps: float = 1e-6

    @property
    def params_per_layer(self) -> int:
        d, m = self.hidden, self.mlp
        return 6 * d * d + 3 * d * d + d * d + 2 * m * d


DIT_TINY = DitShape(256, 4, 64, 1024)
DIT = DitShape(1024, 16, 64, 4096)

DIT_WEIGHT_NAMES = ("w_ada", "b_ada", "w_qkv", "b_qkv", "w_o", "b_o", "w_fc1", "b_fc1", "w_fc2", "b_fc2")

SEEDS["dit"] = dict(weights=1005, tokens=2005, lengths=3005, cond=4005)


def dit_weight_shapes(s: DitShape) -> Dict[str, tuple]:
    d, m = s.hidden, s.mlp
    return {"w_ada": (6 * d, d), "b_ada": (6 * d,), "w_qkv": (3 * d, d), "b_qkv": (3 * d,),
            "w_o": (d, d), "b_o": (d,), "w_fc1": (m, d), "b_fc1": (m,), "w_fc2": (d, m), "b_fc2": (d,)}


def make_dit_weights(s: DitShape, n_layers: int, seed: int, std: float = 0.02) -> List[Dict[str, np.ndarray]]:
    """Per-layer dict of bf16 bits, drawn layer by layer in DIT_WEIGHT_NAMES order, all N(0, std)."""
    rng = np.random.default_rng(seed)
    shapes = dit_weight_shapes(s)
    layers = []
    for _ in range(n_layers):
        lw = {}
        for name in DIT_WEIGHT_NAMES:
            v = rng.standard_normal(shapes[name], dtype=np.float32)
            v *= np.float32(std)
            lw[name] = bf16_bits(v)
            del v
        layers.append(lw)
    return layers


def dit_cond(seed: int, n_seqs: int, hidden: int) -> np.ndarray:
    """Per-sequence conditioning vectors, N(0, 1) float32 (the embedded timestep and class)."""
    return np.random.default_rng(seed).standard_normal((n_seqs, hidden), dtype=np.float32)
