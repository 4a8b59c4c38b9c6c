"""Device-side placement of seeded inputs (data layout only, no layer arithmetic).

Moves generator output (raw bf16 bits) into torch device tensors and builds
key/value caches in the layout the library expects (fp16, per layer):

* K: [n_slots, Hkv, max_ctx, dh]              (key rows of a head contiguous)
* V: [n_slots, Hkv, max_ctx / 32, dh, 32]     (values transposed in 32-key tiles)
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
        if lw.get("b_qkv") is not None:
            d["b_qkv"] = lw["b_qkv"]
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

    TILE = 32  # keys per value tile

    def __init__(self, n_layers: int, n_slots: int, max_ctx: int, n_kv_heads: int, head_dim: int,
                 device="cuda", fill: Optional[float] = None):
        assert max_ctx % 64 == 0
        self.n_slots, self.max_ctx = n_slots, max_ctx
        self.hkv, self.dh = n_kv_heads, head_dim
        mk = (lambda shape: torch.full(shape, fill, dtype=torch.float16, device=device)) if fill is not None \
            else (lambda shape: torch.empty(shape, dtype=torch.float16, device=device))
        self.k = [mk((n_slots, n_kv_heads, max_ctx, head_dim)) for _ in range(n_layers)]
        self.v = [mk((n_slots, n_kv_heads, max_ctx // self.TILE, head_dim, self.TILE)) for _ in range(n_layers)]

    def as_arg(self):
        return (self.k, self.v, self.n_slots, self.max_ctx)

    def _put(self, layer: int, slot: int, k: torch.Tensor, v: torch.Tensor) -> None:
        """Store logical [n, Hkv, dh] fp16 rows at positions 0..n-1 (later positions untouched)."""
        n, T = k.shape[0], self.TILE
        self.k[layer][slot, :, :n] = k.permute(1, 0, 2)
        full = n // T
        vt = v.permute(1, 0, 2)  # [Hkv, n, dh]
        if full:
            self.v[layer][slot, :, :full] = vt[:, :full * T].reshape(self.hkv, full, T, self.dh).transpose(2, 3)
        if n % T:
            self.v[layer][slot, :, full, :, :n % T] = vt[:, full * T:].transpose(1, 2)

    def load_prefix(self, layer: int, slot: int, k_bits: np.ndarray, v_bits: np.ndarray) -> None:
        """Place logical [n, Hkv, dh] rows at positions 0..n-1 of a slot."""
        if k_bits.shape[0] == 0:
            return
        dev = self.k[layer].device
        self._put(layer, slot, to_device_f16(k_bits, dev), to_device_f16(v_bits, dev))

    def fill_random(self, layer: int, slot: int, n: int, gen: torch.Generator) -> None:
        """Seeded N(0, 1) rows (torch's device generator, rounded to fp16) at positions 0..n-1."""
        if n == 0:
            return
        dev = self.k[layer].device
        kv = torch.randn((2, n, self.hkv, self.dh), generator=gen, device=dev, dtype=torch.float32)
        self._put(layer, slot, kv[0].to(torch.float16), kv[1].to(torch.float16))

    def rows(self, layer: int, slot: int, start: int, stop: int):
        """Logical [stop - start, Hkv, dh] K and V rows as fp16 bits on the host."""
        k = f16_bits_of(self.k[layer][slot, :, start:stop].permute(1, 0, 2))
        v_all = self.v[layer][slot].transpose(2, 3).reshape(self.hkv, self.max_ctx, self.dh)
        v = f16_bits_of(v_all[:, start:stop].permute(1, 0, 2))
        return k, v


class PagedCache(DeviceCache):
    """A pool of n_pages pages of page_size positions per layer, plus a block table.

    Sequence b's position p lives in page table[b, p // page_size] at position
    p % page_size; a page is a slot of the DeviceCache layout.
    """

    def __init__(self, n_layers: int, n_pages: int, page_size: int, n_kv_heads: int, head_dim: int,
                 table: np.ndarray, device="cuda", fill: Optional[float] = None):
        super().__init__(n_layers, n_pages, page_size, n_kv_heads, head_dim, device, fill)
        self.page_size = page_size
        self.table = np.ascontiguousarray(table, dtype=np.int32)

    def as_arg(self):
        return (self.k, self.v, self.n_slots, self.max_ctx, self.table)

    def load_prefix(self, layer: int, seq: int, k_bits: np.ndarray, v_bits: np.ndarray) -> None:
        """Place logical [n, Hkv, dh] rows at positions 0..n-1 of sequence `seq`."""
        P = self.page_size
        for j in range(0, k_bits.shape[0], P):
            super().load_prefix(layer, int(self.table[seq, j // P]), k_bits[j:j + P], v_bits[j:j + P])

    def rows(self, layer: int, seq: int, start: int, stop: int):
        """Logical [stop - start, Hkv, dh] K and V rows of sequence `seq` as fp16 bits on the host."""
        P, ks, vs = self.page_size, [], []
        p = start
        while p < stop:
            j, lo = divmod(p, P)
            hi = min(stop - j * P, P)
            k, v = super().rows(layer, int(self.table[seq, j]), lo, hi)
            ks.append(k)
            vs.append(v)
            p = j * P + hi
        return np.concatenate(ks), np.concatenate(vs)


def prepare_dit_f16(ctx, layers_dev: List[Dict[str, torch.Tensor]]) -> List[Dict[str, object]]:
    """The DiT projections (w_qkv, w_o, w_fc1, w_fc2) as fp16 panel-major copies; the
    modulation matrix and the biases stay bf16."""
    from paper_2608_01785_amd import binding
    out = []
    for lw in layers_dev:
        d = {k: v for k, v in lw.items() if k not in binding.DIT_MATRICES}
        d["format"] = binding.HS_WEIGHTS_F16
        for name in binding.DIT_MATRICES:
            n, k = lw[name].shape
            dst = torch.empty((k // 32, n, 32), dtype=torch.float16, device=lw[name].device)
            binding.hs_convert_weights_f16(ctx, lw[name], dst, n, k)
            d[name] = dst
        out.append(d)
    torch.cuda.synchronize()
    return out
