"""Integer side of the hot path: batch metadata and the CU partition.  TEST INFRASTRUCTURE ONLY.

Batch metadata.  The shared stage runs one batch B of mixed requests per
scheduling step (Algorithm 1, step 4).  Rows of the batch are packed: request
b owns rows [seq_offsets[b], seq_offsets[b+1]) and sits behind ctx_lens[b]
cached rows, so its row i is at position ctx_lens[b] + i.

CU partition.  The downstream stage receives the complement of the shared
stage's allocation, s_down = S_tot - s_shared (§4.4, "Complementary downstream
headroom"; Algorithm 1, step 3), and both stages hold pre-built complementary
ladders whose counts always sum to the physical total (§5).  The paper does not
say which units make up a given count; the reading taken here is a balanced
spread over the chip's XCDs, which matters because work-groups are handed to
XCDs round-robin:

* budget c must satisfy 1 <= c <= n_cus;
* XCD x (of n_xcc) receives s_x = c // n_xcc + (1 if x < c % n_xcc else 0)
  shared CUs;
* within an XCD the mask bits are ordered by (cu index within its shader
  engine, shader engine, bit), i.e. round-robin over shader engines, and the
  first s_x of them are shared;
* every other bit is the downstream mask.

The topology is a per-bit table (xcc, se, cu) of length n_cus.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np


class PartitionError(ValueError):
    pass


def plan_metadata(seq_offsets: Sequence[int], ctx_lens: Optional[Sequence[int]] = None):
    """Per-row position and sequence id for a packed ragged batch.

    Returns (pos int32[T], seq_id int32[T]).  Raises ValueError when the
    offsets do not start at 0 or decrease.
    """
    off = [int(o) for o in seq_offsets]
    if len(off) < 2 or off[0] != 0:
        raise ValueError("offsets must start at 0 and hold B+1 entries")
    B = len(off) - 1
    ctx = [0] * B if ctx_lens is None else [int(c) for c in ctx_lens]
    pos, sid = [], []
    for b in range(B):
        if off[b + 1] < off[b]:
            raise ValueError("offsets must be non-decreasing")
        if ctx[b] < 0:
            raise ValueError("cached lengths must be non-negative")
        for i in range(off[b + 1] - off[b]):
            pos.append(ctx[b] + i)
            sid.append(b)
    return np.asarray(pos, dtype=np.int32), np.asarray(sid, dtype=np.int32)


def default_topology(n_cus: int = 256, n_xcc: int = 8, n_se: int = 4):
    """Bit i -> XCD i % n_xcc, slot j = i // n_xcc -> (se = j % n_se, cu = j // n_se)."""
    xcc = [i % n_xcc for i in range(n_cus)]
    se = [(i // n_xcc) % n_se for i in range(n_cus)]
    cu = [(i // n_xcc) // n_se for i in range(n_cus)]
    return xcc, se, cu


def cu_partition(xcc: Sequence[int], se: Sequence[int], cu: Sequence[int], n_xcc: int,
                 c: int) -> Tuple[List[int], List[int]]:
    """Return (shared_words[8], down_words[8]) as 32-bit mask words."""
    n = len(xcc)
    if not (1 <= c <= n):
        raise PartitionError(f"budget {c} outside [1, {n}]")
    if n > 256:
        raise PartitionError("at most 256 CUs")
    shared_bits = set()
    for x in range(n_xcc):
        want = c // n_xcc + (1 if x < c % n_xcc else 0)
        bits = [i for i in range(n) if xcc[i] == x]
        bits.sort(key=lambda i: (cu[i], se[i], i))
        if len(bits) < want:
            raise PartitionError(f"XCD {x} has {len(bits)} CUs, {want} requested")
        shared_bits.update(bits[:want])
    shared = [0] * 8
    down = [0] * 8
    for i in range(n):
        if i in shared_bits:
            shared[i // 32] |= 1 << (i % 32)
        else:
            down[i // 32] |= 1 << (i % 32)
    return shared, down
