"""ctypes declarations of libspecroll.so (the C ABI in include/specroll.h).

Loading fails loudly when the built library is missing: there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspecroll.so")

SR_OK, SR_ERR_INVALID, SR_ERR_UNSUPPORTED, SR_ERR_WORKSPACE, SR_ERR_HIP = 0, 1, 2, 3, 4
SR_F32, SR_BF16 = 0, 1
SR_MAX_TREE = 128

_p = C.c_void_p
_i32p = C.POINTER(C.c_int32)


class HeadsDesc(C.Structure):
    _fields_ = [("B", C.c_int32), ("d", C.c_int32), ("H", C.c_int32), ("V", C.c_int32), ("T", C.c_int32),
                ("max_children", C.c_int32), ("dtype", C.c_int32), ("clip_norm", C.c_float),
                ("ln_eps", C.c_float)]


class AttnDesc(C.Structure):
    _fields_ = [("B", C.c_int32), ("T", C.c_int32), ("Hq", C.c_int32), ("Hkv", C.c_int32), ("D", C.c_int32),
                ("block_size", C.c_int32), ("max_blocks", C.c_int32), ("num_blocks", C.c_int32),
                ("dtype", C.c_int32), ("scale", C.c_float)]


class AcceptDesc(C.Structure):
    _fields_ = [("B", C.c_int32), ("T", C.c_int32), ("V", C.c_int32), ("max_depth", C.c_int32),
                ("logit_dtype", C.c_int32), ("temperature", C.c_float), ("top_p", C.c_float)]


class BudgetDesc(C.Structure):
    _fields_ = [("c_peak", C.c_int32), ("n_min", C.c_int32), ("n_max", C.c_int32), ("n_alloc", C.c_int32),
                ("alloc", _i32p)]


class CommitDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("B", C.c_int32), ("T", C.c_int32), ("Hkv", C.c_int32),
                ("D", C.c_int32), ("block_size", C.c_int32), ("max_blocks", C.c_int32),
                ("num_blocks", C.c_int32), ("max_depth", C.c_int32), ("dtype", C.c_int32)]


class ReflexDesc(C.Structure):
    _fields_ = [("R", C.c_int32), ("V", C.c_int32), ("d", C.c_int32), ("B", C.c_int32), ("H", C.c_int32),
                ("n_p_rows", C.c_int32), ("n_q_rows", C.c_int32), ("max_cand", C.c_int32), ("support", C.c_int32),
                ("n_boundary", C.c_int32), ("p_dtype", C.c_int32), ("w_dtype", C.c_int32),
                ("temperature", C.c_float), ("w_dist", C.c_float), ("w_cov", C.c_float), ("sev_tv", C.c_float),
                ("sev_out", C.c_float), ("w_min", C.c_float), ("eps", C.c_float), ("rho", C.c_float * 8),
                ("rank", C.c_int32)]


class ReflexGateDesc(C.Structure):
    _fields_ = [("rank", C.c_int32), ("z_delta", C.c_float), ("eps", C.c_float), ("m_floor", C.c_float),
                ("alpha_min", C.c_float * 8), ("alpha_max", C.c_float * 8), ("n_fb_min", C.c_int32 * 8),
                ("n_align_min", C.c_int32 * 8)]


# name -> (restype, argtypes)
SIGNATURES = {
    "sr_last_error": (C.c_char_p, []),
    "sr_version": (C.c_char_p, []),
    "sr_kernel_names": (C.c_char_p, []),
    "sr_heads_propose_workspace": (C.c_size_t, [C.POINTER(HeadsDesc)]),
    "sr_heads_propose": (C.c_int, [C.POINTER(HeadsDesc), _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p,
                                   _p, C.c_size_t, _p]),
    "sr_tree_build_workspace": (C.c_size_t, [C.POINTER(HeadsDesc)]),
    "sr_tree_build": (C.c_int, [C.POINTER(HeadsDesc), _p, _p, _p, _p, _p, _p, _p, C.c_size_t, _p]),
    "sr_tree_verify_attn_workspace": (C.c_size_t, [C.POINTER(AttnDesc)]),
    "sr_tree_verify_attn": (C.c_int, [C.POINTER(AttnDesc), _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p,
                                      C.c_size_t, _p]),
    "sr_tree_verify_attn_noalloc": (C.c_int, [C.POINTER(AttnDesc), _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p]),
    "sr_tree_accept_workspace": (C.c_size_t, [C.POINTER(AcceptDesc)]),
    "sr_tree_accept": (C.c_int, [C.POINTER(AcceptDesc), _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p,
                                 C.c_size_t, _p]),
    "sr_tree_budget": (C.c_int, [C.POINTER(BudgetDesc), C.c_int32, _i32p, _i32p, _i32p, C.c_int32, _i32p]),
    "sr_commit_path": (C.c_int, [C.POINTER(CommitDesc), _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p]),
    "sr_reflex_feedback": (C.c_int, [C.POINTER(ReflexDesc), _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p,
                                     _p, _p]),
    "sr_heads_propose_reflex": (C.c_int, [C.POINTER(HeadsDesc), C.POINTER(ReflexGateDesc), _p, _p, _p, _p, _p, _p,
                                          _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, _p, C.c_size_t, _p]),
    "sr_prof_begin": (C.c_int, [C.c_char_p]),
    "sr_prof_end": (C.c_int, [C.POINTER(C.c_double), _i32p]),
}

_lib = None


def lib() -> C.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_04962_amd.build` "
                               "(there is no fallback implementation)")
        h = C.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(h, name)
            f.restype = res
            f.argtypes = args
        _lib = h
    return _lib


def last_error() -> str:
    return lib().sr_last_error().decode()


class SpecRollError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where} failed with status {status}: {last_error()}")


def check(status: int, where: str) -> None:
    if status != SR_OK:
        raise SpecRollError(status, where)
