"""sr_tree_verify_attn_noalloc (the allocation-free variant of the tree-verify attention, for callers that cannot
allocate device memory) against sr_tree_verify_attn with a caller workspace: same kernels and plan, so the
outputs must agree bit for bit. Two calls in a row on one GPU share its scratch array; the second is smaller and
must not see the first's counters or recomputation list."""
import ctypes as C

import numpy as np
import pytest
import torch

import paper_2608_04962_amd as sr
from paper_2608_04962_amd import _lib
import synth
from helpers import dev_tensor, f64, row_rel_err


def _tensors(inp):
    return {k: dev_tensor(inp[k]) for k in ("q", "k_cache", "v_cache", "k_tree", "v_tree", "block_table", "ctx_len",
                                            "parents")}


def _noalloc(t, scale):
    B, T, Hq, D = t["q"].shape
    out = torch.empty((B, T, Hq, D), dtype=torch.float32, device="cuda")
    lse = torch.empty((B, T, Hq), dtype=torch.float32, device="cuda")
    desc = sr.attn_desc(t["q"], t["k_cache"], t["block_table"], scale)
    st = _lib.lib().sr_tree_verify_attn_noalloc(
        C.byref(desc), t["q"].data_ptr(), t["k_cache"].data_ptr(), t["v_cache"].data_ptr(),
        t["block_table"].data_ptr(), t["ctx_len"].data_ptr(), t["k_tree"].data_ptr(), t["v_tree"].data_ptr(),
        t["parents"].data_ptr(), out.data_ptr(), lse.data_ptr(), C.c_void_p(torch.cuda.current_stream().cuda_stream))
    _lib.check(st, "sr_tree_verify_attn_noalloc")
    return out, lse


def _with_workspace(t, scale):
    return sr.tree_verify_attn(t["q"], t["k_cache"], t["v_cache"], t["block_table"], t["ctx_len"], t["k_tree"],
                               t["v_tree"], t["parents"], scale=scale)


def _scale_v(inp, traj, factor):
    inp = dict(inp)
    vc = synth.to_f64(inp["v_cache"], "bf16")
    pages = inp["block_table"][traj, :-(-int(inp["ctx_len"][traj]) // 16)]
    vc[pages] *= factor
    inp["v_cache"] = synth.as_dtype(vc.astype(np.float32), "bf16")
    return inp


@pytest.mark.gpu
def test_noalloc_matches_workspace_call_twice():
    # first call: 48 trajectories of the 7B attention shape with 1-8k-token contexts (split prefixes, partials
    # in the scratch array) and one trajectory whose V needs the fp32 recomputation; second call: a smaller,
    # different shape with no such values
    big = synth.scaled(synth.SHAPE_7B, B=48)
    small = synth.scaled(synth.SHAPE_7B, B=5, T=12, depth=4, Hq=8, Hkv=2, ctx=("uniform", 1, 5000))
    inputs = [_scale_v(synth.attn_inputs(big, seed=0), 3, 1.0e5), synth.attn_inputs(small, seed=1)]
    for inp in inputs:
        print(f"[noalloc] {inp['cfg'].name} B={inp['cfg'].B} T={inp['cfg'].T}", flush=True)
        t = _tensors(inp)
        o1, l1 = _noalloc(t, inp["scale"])
        torch.cuda.synchronize()
        o2, l2 = _with_workspace(t, inp["scale"])
        torch.cuda.synchronize()
        assert torch.equal(o1, o2) and torch.equal(l1, l2)
        assert torch.isfinite(o1).all()


def test_noalloc_rejects_requests_beyond_its_scratch():
    # 1024 trajectories of 64 rows with 16k-token contexts need ~3.2 GB of partials: refused on the host,
    # before anything touches a device
    d = _lib.AttnDesc(1024, 64, 8, 8, 128, 16, 1024, 100000, _lib.SR_BF16, 0.088)
    need = _lib.lib().sr_tree_verify_attn_workspace(C.byref(d))
    assert need > 256 << 20
    fake = C.c_void_p(1 << 20)    # never dereferenced: the size check fails first
    st = _lib.lib().sr_tree_verify_attn_noalloc(C.byref(d), *([fake] * 9), None, None)
    assert st == _lib.SR_ERR_UNSUPPORTED
    assert "scratch" in _lib.last_error()
