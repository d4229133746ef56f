"""Shared test utilities: array conversion between the generators, torch and the oracle, and the
row-normwise relative error used by the parity bars."""
import numpy as np
import torch

import oracle
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


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    """Spacing of bf16 values (8 significant bits) at |x|."""
    _, e = np.frexp(np.abs(np.asarray(x, dtype=np.float64)))
    return np.ldexp(1.0, e - 8)


# GPU LayerNorm in fp32 (mean, variance and scale over d <= 8192 elements) stays well within this relative
# distance of the float64 value; an LN output closer than this to a bf16 rounding midpoint may round either way
LN_AMBIGUOUS_REL = 2.0 ** -20


def z_tolerance(x: np.ndarray, A: np.ndarray, ln_eps: float = 1e-5) -> np.ndarray:
    """Per-element bound [rows, H, d] on |z_gpu - z_exact| for bf16 head states z = round(x + SiLU(A LN(x) + b)).

    z_exact is the oracle's value before its rounding point, computed from its own bf16-rounded LN output.
    * one bf16 ulp of z: the final nearest-even decision may fall either way (the GPU evaluates the
      pre-rounding value in fp32);
    * 2^-20 of the row's largest |x| + 1: the fp32 evaluation of x and of the GEMM before that rounding;
    * the LN outputs n_i within LN_AMBIGUOUS_REL of a bf16 midpoint may be rounded the other way by the GPU,
      moving A_h n by |A_h[:, i]| ulp(n_i) each, times max SiLU' < 1.1.
    """
    x = np.asarray(x, dtype=np.float64)
    A = np.asarray(A, dtype=np.float64)
    n = oracle.layer_norm(x, ln_eps)
    nr = oracle.round_bf16(n)
    ulp_n = bf16_ulp(n)
    amb = (0.5 * ulp_n - np.abs(n - nr)) <= LN_AMBIGUOUS_REL * np.abs(n)
    w = np.where(amb, ulp_n, 0.0)                          # [rows, d]
    flip = np.stack([w @ np.abs(A[h]).T for h in range(A.shape[0])], axis=1)   # [rows, H, d]
    floor = 2.0 ** -20 * (np.abs(x).max(axis=-1) + 1.0)
    return 1.1 * flip + floor[:, None, None]


def assert_z_bf16(got: np.ndarray, exact: np.ndarray, extra_tol: np.ndarray):
    """``got`` (bf16 values) within one bf16 ulp of ``exact`` plus ``extra_tol`` (same shape, see z_tolerance)."""
    got = np.asarray(got, dtype=np.float64)
    exact = np.asarray(exact, dtype=np.float64)
    err = np.abs(got - exact)
    lim = bf16_ulp(exact) + extra_tol
    bad = err > lim
    assert not bad.any(), f"{bad.sum()} of {bad.size} values off by more than their bound; worst excess " \
                          f"{(err - lim)[bad].max():.3e}, worst error {err[bad].max():.3e}"
