"""Helpers shared by the GPU tests: moving seeded arrays to the device and
the comparison rule against the oracle."""
from __future__ import annotations

import numpy as np
import torch

from paper_2410_19123_amd import workloads as wl

# Floating-point tolerance of the layer outputs (bf16 inputs, fp32
# accumulation), relative to the fp64 oracle:
#   max |y - ref| <= 2e-2 * max |ref|  and  sum |y - ref| / sum |ref| <= 5e-3.
MAX_REL = 2e-2
L1_REL = 5e-3


def dev():
    return torch.device("cuda:0")


def to_dev(a: np.ndarray) -> torch.Tensor:
    from paper_2410_19123_amd import _lib
    return _lib.to_device(a, dev())


def from_dev(t: torch.Tensor) -> np.ndarray:
    from paper_2410_19123_amd import _lib
    return _lib.from_device(t)


def as_f64(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:
        return wl.bf16_bits_to_f32(a).astype(np.float64)
    return a.astype(np.float64)


def close(got: np.ndarray, ref: np.ndarray, what: str = ""):
    """Assert the tolerance above; returns (max_rel, l1_rel)."""
    got = as_f64(got) if got.dtype != np.float64 else got
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    err = np.abs(got - ref)
    scale = np.abs(ref).max()
    max_rel = float(err.max() / scale) if scale > 0 else float(err.max())
    l1 = float(err.sum() / np.abs(ref).sum()) if scale > 0 else float(err.sum())
    assert max_rel <= MAX_REL, f"{what}: max rel err {max_rel:.3e}"
    assert l1 <= L1_REL, f"{what}: normalized L1 err {l1:.3e}"
    return max_rel, l1


def weights_to_dev(wg, wu, wd):
    return to_dev(wg), to_dev(wu), to_dev(wd)
