"""Shared helpers of the GPU tests: skip logic, device buffers, tolerance."""
import sys

import numpy as np
import pytest

TOL = 2e-2  # max |gpu - reference| <= 2e-2 * rms(reference), per output tensor


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_01785_amd import binding  # fails loudly if the library is missing
    binding.lib()
    return torch


def workspace(torch, cfg, T, B, max_pos):
    from paper_2608_01785_amd import binding
    n = binding.hs_workspace_size(cfg, T, B, max_pos)
    return torch.empty(n, dtype=torch.uint8, device="cuda")


def err_ratio(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert np.all(np.isfinite(got)), "non-finite GPU output"
    return float(np.max(np.abs(got - ref)) / np.sqrt(np.mean(ref * ref)))
