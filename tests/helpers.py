"""Shared checks for the GPU parity tests."""
import sys

import numpy as np

from paper_2504_14489_amd.device import bits_to_f32

# bf16 outputs against the fp64 oracle: per call, over every compared element
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def say(*a):
    """Names the case about to run on the GPU (flushed, so a fault leaves it)."""
    print(*a, file=sys.stderr, flush=True)


def assert_close(got_bits: np.ndarray, ref: np.ndarray, what: str):
    got = bits_to_f32(got_bits).astype(np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - ref)
    mx, mean = float(err.max(initial=0.0)), float(err.mean()) if err.size else 0.0
    assert mx <= MAX_ABS and mean <= MEAN_ABS, f"{what}: max-abs {mx:.3g} mean-abs {mean:.3g}"
    return mx, mean
