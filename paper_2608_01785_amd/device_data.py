"""Device-side placement of seeded inputs (data layout only, no layer arithmetic).

Moves generator output (raw bf16 bits) into torch device tensors and builds
key/value caches in the layout the library expects:

* K: fp16 [n_slots, max_ctx, Hkv, dh]   (token-major)
* V: fp16 [n_slots, Hkv, dh, max_ctx]   (dimension-major)
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np
import torch


def to_device(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 bf16 bits -> torch.bfloat16 device tensor (same shape)."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to(device)


def to_bits(t: torch.Tensor) -> np.ndarray:
    """torch.bfloat16 tensor -> uint16 bf16 bits on the host."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def to_device_f16(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 fp16 bits -> torch.float16 device tensor."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.float16).to(device)


def f16_bits_of(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def upload_weights(layers: List[Dict[str, np.ndarray]], device="cuda") -> List[Dict[str, torch.Tensor]]:
    return [{k: to_device(v, device) for k, v in lw.items()} for lw in layers]


def prepare_f16(ctx, layers_dev: List[Dict[str, torch.Tensor]]) -> List[Dict[str, object]]:
    """fp16 panel-major copies of the projection matrices (the library's converter); gains stay bf16.

    Each copy is a flat buffer holding [K / 32][N][32] for an [N, K] matrix.
    """
    from paper_2608_01785_amd import binding
    out = []
    for lw in layers_dev:
        d = {"ln1": lw["ln1"], "ln2": lw["ln2"], "format": binding.HS_WEIGHTS_F16}
        for name in binding.MATRICES:
            n, k = lw[name].shape
            dst = torch.empty((k // 32, n, 32), dtype=torch.float16, device=lw[name].device)
            binding.hs_convert_weights_f16(ctx, lw[name], dst, n, k)
            d[name] = dst
        out.append(d)
    torch.cuda.synchronize()
    return out


class DeviceCache:
    """Per-layer K/V device tensors for n_slots sequences of up to max_ctx positions."""

    def __init__(self, n_layers: int, n_slots: int, max_ctx: int, n_kv_heads: int, head_dim: int,
                 device="cuda", fill: Optional[float] = None):
        assert max_ctx % 64 == 0
        self.n_slots, self.max_ctx = n_slots, max_ctx
        self.hkv, self.dh = n_kv_heads, head_dim
        mk = (lambda shape: torch.full(shape, fill, dtype=torch.float16, device=device)) if fill is not None \
            else (lambda shape: torch.empty(shape, dtype=torch.float16, device=device))
        self.k = [mk((n_slots, max_ctx, n_kv_heads, head_dim)) for _ in range(n_layers)]
        self.v = [mk((n_slots, n_kv_heads, head_dim, max_ctx)) for _ in range(n_layers)]

    def as_arg(self):
        return (self.k, self.v, self.n_slots, self.max_ctx)

    def load_prefix(self, layer: int, slot: int, k_bits: np.ndarray, v_bits: np.ndarray) -> None:
        """Place logical [n, Hkv, dh] rows at positions 0..n-1 of a slot."""
        n = k_bits.shape[0]
        if n == 0:
            return
        self.k[layer][slot, :n] = to_device_f16(k_bits, self.k[layer].device)
        self.v[layer][slot, :, :, :n] = to_device_f16(v_bits, self.v[layer].device).permute(1, 2, 0)

    def fill_random(self, layer: int, slot: int, n: int, gen: torch.Generator) -> None:
        """Seeded N(0, 1) rows (torch's device generator, rounded to fp16) at positions 0..n-1."""
        if n == 0:
            return
        dev = self.k[layer].device
        kv = torch.randn((2, n, self.hkv, self.dh), generator=gen, device=dev, dtype=torch.float32)
        self.k[layer][slot, :n] = kv[0].to(torch.float16)
        self.v[layer][slot, :, :, :n] = kv[1].to(torch.float16).permute(1, 2, 0)

    def rows(self, layer: int, slot: int, start: int, stop: int):
        """Logical [stop - start, Hkv, dh] K and V rows as fp16 bits on the host."""
        k = f16_bits_of(self.k[layer][slot, start:stop])
        v = f16_bits_of(self.v[layer][slot, :, :, start:stop].permute(2, 0, 1))
        return k, v
