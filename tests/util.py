"""Test helpers: conversions between the generator's bf16 bits and float64."""
import numpy as np

from paper_2608_01785_amd.workloads import bf16_to_f32, bf16_bits, f16_to_f32


def f64(bits):
    """bf16 bits -> float64."""
    return bf16_to_f32(bits).astype(np.float64)


def h64(bits):
    """fp16 bits -> float64."""
    return f16_to_f32(bits).astype(np.float64)


def weights_f64(layers):
    return [{k: f64(v) for k, v in lw.items()} for lw in layers]


def as_bf16_f64(a):
    """Round float values to bf16 and return them as float64 (exactly representable)."""
    return f64(bf16_bits(np.asarray(a, dtype=np.float32)))


def rel_err(got, ref):
    """max |got - ref| / rms(ref)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    return float(np.max(np.abs(got - ref))) / rms
