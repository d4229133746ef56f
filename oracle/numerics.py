"""Small float64 helpers of the oracle (test infrastructure only)."""
from __future__ import annotations

import numpy as np


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 value (ties to even), returned as float64.

    bfloat16 keeps 8 significant bits. With x = m * 2**e and 0.5 <= |m| < 1,
    the rounded value is rint(m * 2**8) * 2**(e - 8); ``np.rint`` rounds half
    to even. Normal range only (the workloads never reach bf16 subnormals or
    overflow); zeros and NaN pass through.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(m * 256.0), e - 8)


def logsumexp(s: np.ndarray, axis: int = -1) -> np.ndarray:
    mx = np.max(s, axis=axis, keepdims=True)
    return (mx + np.log(np.sum(np.exp(s - mx), axis=axis, keepdims=True))).squeeze(axis)


def softmax(s: np.ndarray, axis: int = -1) -> np.ndarray:
    mx = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - mx)
    return e / np.sum(e, axis=axis, keepdims=True)
