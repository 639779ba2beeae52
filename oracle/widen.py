"""Exact widening of stored inputs to float64 (oracle; test infrastructure only)."""

import numpy as np


def widen(a: np.ndarray, dtype: str) -> np.ndarray:
    """float32 values, or bfloat16 given as uint16 bit patterns, to float64.

    A bfloat16 value is the upper half of a float32 word, so shifting its 16 bits
    into the top of a 32-bit word reproduces it exactly; float32 -> float64 is
    exact as well.
    """
    if dtype == "f64":                          # values computed by the oracle itself
        return np.asarray(a, np.float64)
    if dtype == "f32":
        return np.asarray(a, np.float32).astype(np.float64)
    if dtype == "bf16":
        w = np.asarray(a, np.uint16).astype(np.uint32) << np.uint32(16)
        return w.view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")
