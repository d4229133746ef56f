"""Shared test utilities: array conversion between the generators, torch and the oracle, and the
row-normwise relative error used by the parity bars."""
import numpy as np
import torch

import synth


def dev_tensor(x: np.ndarray, dtype: str = None, device="cuda"):
    """numpy array (bf16 stored as uint16 bits) -> device tensor of the workload dtype."""
    if x.dtype == np.uint16:
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to(device)


def f64(x: np.ndarray, dtype: str) -> np.ndarray:
    return synth.to_f64(x, dtype)


def row_rel_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per row (last axis): max|got - ref| / max|ref|."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.abs(got - ref).max(axis=-1)
    den = np.abs(ref).max(axis=-1)
    return num / np.maximum(den, 1e-300)


def tol_for(dtype: str) -> float:
    return 1e-5 if dtype == "f32" else 2e-3


def assert_faithful_bf16(got: np.ndarray, exact: np.ndarray, row_tol: float = 1e-3):
    """``got`` (bf16 values) must lie within one bf16 ulp of ``exact`` plus ``row_tol`` times the row's
    largest magnitude. The ulp covers the nearest-even decision of the final rounding, which may fall either
    way when the two sides compute the pre-rounding value in different precisions; the row term covers
    upstream rounding points (LayerNorm output rounded to bf16) whose decisions may differ the same way."""
    got = np.asarray(got, dtype=np.float64)
    exact = np.asarray(exact, dtype=np.float64)
    _, e = np.frexp(np.abs(exact))
    ulp = np.ldexp(1.0, e - 8)          # spacing of bf16 values at |exact| (8 significant bits)
    scale = np.abs(exact).max(axis=-1, keepdims=True)
    err = np.abs(got - exact)
    bad = err > ulp + row_tol * scale
    assert not bad.any(), f"{bad.sum()} values off by more than one bf16 ulp + {row_tol} of the row scale; " \
                          f"worst {err[bad].max()}"
