"""CPU checks of the C ABI: the library loads, exports every function include/specroll.h declares,
and rejects malformed calls on the host before anything is enqueued (no GPU needed)."""
import ctypes as C
import os
import re

import pytest

import paper_2608_04962_amd as sr
from paper_2608_04962_amd import _lib

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "specroll.h")


def _declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(sr_[a-z_]+)\s*\(", txt)))


def test_library_loads_and_reports_version():
    assert "gfx950" in sr.version()
    assert "sr_tree_attn" in sr.kernel_names()


def test_every_declared_function_is_exported_and_bound():
    names = _declared_functions()
    assert {"sr_heads_propose", "sr_tree_build", "sr_tree_verify_attn", "sr_tree_accept"} <= set(names)
    h = C.CDLL(_lib.LIB_PATH)
    for n in names:
        assert hasattr(h, n), n
        assert n in _lib.SIGNATURES, f"{n} has no binding"


def test_struct_layouts_match_header():
    # the descriptors are plain int32/float fields in header order
    assert C.sizeof(_lib.HeadsDesc) == 9 * 4
    assert C.sizeof(_lib.AttnDesc) == 10 * 4
    assert C.sizeof(_lib.AcceptDesc) == 7 * 4
    assert C.sizeof(_lib.CommitDesc) == 10 * 4
    assert C.sizeof(_lib.BudgetDesc) == 4 * 4 + C.sizeof(C.c_void_p)
    assert C.sizeof(_lib.ReflexDesc) == (12 + 7 + 8 + 1) * 4
    assert C.sizeof(_lib.ReflexGateDesc) == (4 + 8 * 4) * 4


def _call_heads(desc, **ptrs):
    args = [ptrs.get(k) for k in ("hidden", "corr", "act", "A", "bias", "W", "parents", "root", "u", "logits", "z",
                                  "tokens", "cl")]
    return _lib.lib().sr_heads_propose(C.byref(desc), *args, ptrs.get("ws"), ptrs.get("wsb", 0), None)


@pytest.mark.parametrize("field,value", [("B", 0), ("d", 96), ("H", 0), ("T", 0), ("T", 129),
                                         ("max_children", 8), ("dtype", 7), ("clip_norm", 0.0),
                                         ("V", 4099), ("V", 4), ("V", 0)])
def test_heads_descriptor_rejected(field, value):
    desc = _lib.HeadsDesc(2, 256, 2, 512, 8, 2, _lib.SR_F32, 1.0, 1e-5)
    setattr(desc, field, value)
    st = _call_heads(desc)
    assert st == _lib.SR_ERR_INVALID
    assert _lib.last_error()


def test_heads_null_pointer_and_small_workspace_rejected():
    desc = _lib.HeadsDesc(2, 256, 2, 512, 8, 2, _lib.SR_F32, 1.0, 1e-5)
    assert _call_heads(desc) == _lib.SR_ERR_INVALID
    assert "null" in _lib.last_error()
    fake = C.c_void_p(1 << 20)   # never dereferenced: the workspace check fails first
    ptrs = {k: fake for k in ("hidden", "A", "bias", "W", "parents", "root", "u", "tokens", "cl")}
    st = _call_heads(desc, ws=None, wsb=0, **ptrs)
    assert st == _lib.SR_ERR_WORKSPACE
    need = _lib.lib().sr_heads_propose_workspace(C.byref(desc))
    assert need > 0
    st = _call_heads(desc, ws=fake, wsb=need - 1, **ptrs)
    assert st == _lib.SR_ERR_WORKSPACE


@pytest.mark.parametrize("field,value", [("Hq", 6), ("D", 96), ("block_size", 32), ("max_blocks", 0),
                                         ("T", 200), ("dtype", 3)])
def test_attn_descriptor_rejected(field, value):
    desc = _lib.AttnDesc(2, 8, 4, 4, 64, 16, 10, 20, _lib.SR_F32, 0.125)
    desc.Hkv = 4
    if field == "Hq":
        desc.Hkv = 4
    setattr(desc, field, value)
    st = _lib.lib().sr_tree_verify_attn(C.byref(desc), *([None] * 10), None, 0, None)
    assert st == _lib.SR_ERR_INVALID


@pytest.mark.parametrize("field,value", [("V", 12), ("V", 1 << 20), ("temperature", 0.0), ("max_depth", -1),
                                         ("T", 0), ("top_p", 0.0), ("top_p", 1.5), ("top_p", float("nan"))])
def test_accept_descriptor_rejected(field, value):
    desc = _lib.AcceptDesc(2, 8, 512, 3, _lib.SR_F32, 1.0, 1.0)
    setattr(desc, field, value)
    st = _lib.lib().sr_tree_accept(C.byref(desc), *([None] * 11), None, 0, None)
    assert st == _lib.SR_ERR_INVALID


def test_workspace_queries_are_consistent():
    d = _lib.AttnDesc(128, 32, 28, 4, 128, 16, 512, 40000, _lib.SR_BF16, 0.088)
    ws = _lib.lib().sr_tree_verify_attn_workspace(C.byref(d))
    assert ws > 0 and ws % 256 == 0
    d1 = _lib.AttnDesc(2, 8, 4, 2, 64, 16, 10, 20, _lib.SR_F32, 0.125)   # one chunk: no partials
    assert _lib.lib().sr_tree_verify_attn_workspace(C.byref(d1)) == 0
    # bf16 runs persistent blocks that take work items from a counter, followed by the count and list of items
    # to recompute with fp32 V and the longest-first item list with its length: 3 + 2 n_items words in
    # 256-byte slots
    d2 = _lib.AttnDesc(2, 8, 4, 2, 64, 16, 10, 20, _lib.SR_BF16, 0.125)   # 2 x 2 (trajectory, KV head) items
    assert _lib.lib().sr_tree_verify_attn_workspace(C.byref(d2)) == 256
    d3 = _lib.AttnDesc(128, 32, 28, 4, 128, 16, 512, 40000, _lib.SR_F32, 0.088)
    n_items = 128 * 4 * 2                                               # 224 rows: one group; 256-page chunks
    assert _lib.lib().sr_tree_verify_attn_workspace(C.byref(d)) == \
        _lib.lib().sr_tree_verify_attn_workspace(C.byref(d3)) + (3 + 2 * n_items) * 4 // 256 * 256 + 256
    assert _lib.lib().sr_tree_accept_workspace(C.byref(_lib.AcceptDesc(2, 8, 512, 3, 0, 1.0, 1.0))) == 0


def test_prof_hook_host_side():
    _lib.check(_lib.lib().sr_prof_begin(b"sr_tree_attn"), "begin")
    assert sr.prof_end() == (0.0, 0)


@pytest.mark.parametrize("field,value", [("n_layers", 0), ("n_layers", 70000), ("B", 0), ("T", 0), ("T", 129),
                                         ("D", 4), ("dtype", 5), ("block_size", 0), ("max_depth", -1),
                                         ("max_depth", 200), ("num_blocks", 0)])
def test_commit_descriptor_rejected(field, value):
    desc = _lib.CommitDesc(2, 4, 8, 2, 64, 16, 10, 40, 3, _lib.SR_BF16)
    setattr(desc, field, value)
    fake = C.c_void_p(1 << 20)    # never dereferenced: the descriptor check fails first
    st = _lib.lib().sr_commit_path(C.byref(desc), *([fake] * 10), None)
    assert st == _lib.SR_ERR_INVALID
    assert _lib.last_error()


def test_commit_pointer_checks():
    desc = _lib.CommitDesc(2, 4, 8, 2, 64, 16, 10, 40, 3, _lib.SR_BF16)
    fake = C.c_void_p(1 << 20)
    args = [fake] * 10
    args[0] = None                                      # acc_nodes with max_depth > 0
    assert _lib.lib().sr_commit_path(C.byref(desc), *args, None) == _lib.SR_ERR_INVALID
    args = [fake] * 10
    args[3] = C.c_void_p((1 << 20) + 8)                 # misaligned k_tree
    assert _lib.lib().sr_commit_path(C.byref(desc), *args, None) == _lib.SR_ERR_INVALID
    args = [fake] * 10
    args[9] = args[6]                                   # new_ctx_len == ctx_len
    assert _lib.lib().sr_commit_path(C.byref(desc), *args, None) == _lib.SR_ERR_INVALID
    assert "overlap" in _lib.last_error()


@pytest.mark.parametrize("c_peak,n_min,n_max,alloc", [
    (512, 1, 10, (5, 4, 0)), (300, 3, 17, (1, 6, 2, 9)), (64, 1, 5, (0, 3)), (7, 1, 128, (100, 100)), (50, 2, 9, ())])
def test_tree_budget_host_rule_matches_oracle(c_peak, n_min, n_max, alloc):
    """sr_tree_budget is host-only integer logic, so its parity with the oracle runs here, bit-exact."""
    import oracle
    for live in list(range(1, 2 * c_peak + 3)) + [10 ** 6]:
        got = sr.tree_budget(live, c_peak, n_min, n_max, alloc)
        n_t, counts, parents = oracle.tree_budget(live, c_peak, n_min, n_max, alloc)
        assert got == (n_t, counts, parents.tolist()), live


def test_tree_budget_rejections():
    lib = _lib.lib()
    al = (C.c_int32 * 3)(5, 4, 0)
    out = [C.c_int32() for _ in range(2)]
    par = (C.c_int32 * 10)()
    good = _lib.BudgetDesc(512, 1, 10, 3, al)
    args = lambda live, cap: (live, C.byref(out[0]), None, par, cap, C.byref(out[1]))  # noqa: E731
    assert lib.sr_tree_budget(C.byref(good), *args(1, 10)) == _lib.SR_OK
    assert (out[0].value, out[1].value) == (10, 10)
    assert lib.sr_tree_budget(C.byref(good), *args(0, 10)) == _lib.SR_ERR_INVALID
    assert lib.sr_tree_budget(C.byref(good), *args(1, 9)) == _lib.SR_ERR_INVALID     # capacity below the tree
    assert lib.sr_tree_budget(C.byref(good), *args(200, 3)) == _lib.SR_OK             # 512 // 200 = 2 nodes
    assert (out[0].value, out[1].value) == (2, 2) and par[:2] == [-1, 0]
    for bad in (_lib.BudgetDesc(0, 1, 10, 3, al), _lib.BudgetDesc(512, 0, 10, 3, al),
                _lib.BudgetDesc(512, 4, 3, 3, al), _lib.BudgetDesc(512, 1, 129, 3, al),
                _lib.BudgetDesc(512, 1, 10, 3, None), _lib.BudgetDesc(512, 1, 10, 2, (C.c_int32 * 2)(3, -1))):
        assert lib.sr_tree_budget(C.byref(bad), *args(1, 200)) == _lib.SR_ERR_INVALID


def _reflex_desc(**over):
    d = _lib.ReflexDesc(4, 512, 256, 2, 2, 4, 4, 3, 48, 4, _lib.SR_F32, _lib.SR_F32, 1.0, 0.15, 1.25, 0.3, 0.7,
                        0.03, 1e-6, (C.c_float * 8)(0.85, 0.9, 0.95, 0.95, 0.95, 0.95, 0.95, 0.95), 0)
    for k, v in over.items():
        setattr(d, k, v)
    return d


@pytest.mark.parametrize("field,value", [("R", 0), ("V", 12), ("V", 1 << 20), ("d", 12), ("d", 16384), ("H", 9),
                                         ("support", 0), ("support", 65), ("max_cand", 49), ("max_cand", 0),
                                         ("n_boundary", 0), ("p_dtype", 4), ("temperature", 0.0), ("eps", 0.0),
                                         ("w_cov", -1.0), ("n_p_rows", 0)])
def test_reflex_descriptor_rejected(field, value):
    fake = C.c_void_p(1 << 20)
    st = _lib.lib().sr_reflex_feedback(C.byref(_reflex_desc(**{field: value})), *([fake] * 11), None, None, None,
                                       None, None)
    assert st == _lib.SR_ERR_INVALID
    assert _lib.last_error()


def test_reflex_rho_and_pointer_checks():
    fake = C.c_void_p(1 << 20)
    d = _reflex_desc()
    d.rho[1] = 1.0
    tail = (None, None, None, None, None)
    assert _lib.lib().sr_reflex_feedback(C.byref(d), *([fake] * 11), *tail) == _lib.SR_ERR_INVALID
    args = [fake] * 11
    args[9] = None                                           # memory
    assert _lib.lib().sr_reflex_feedback(C.byref(_reflex_desc()), *args, *tail) == _lib.SR_ERR_INVALID
    args = [fake] * 11
    args[8] = C.c_void_p((1 << 20) + 4)                      # misaligned W
    assert _lib.lib().sr_reflex_feedback(C.byref(_reflex_desc()), *args, *tail) == _lib.SR_ERR_INVALID
    # alignment with rank > 0 needs P and the stored sketches
    assert _lib.lib().sr_reflex_feedback(C.byref(_reflex_desc(rank=24)), *([fake] * 11), None, None, None, fake,
                                         None) == _lib.SR_ERR_INVALID


@pytest.mark.parametrize("change", ["rank", "eps", "alpha", "count", "H", "P"])
def test_heads_reflex_gate_rejected(change):
    hd = _lib.HeadsDesc(2, 256, 2, 512, 8, 2, _lib.SR_F32, 1.0, 1e-5)
    g = sr.reflex_gate_desc(rank=4)
    fake = C.c_void_p(1 << 20)
    P = fake
    if change == "rank":
        g.rank = 65
    elif change == "eps":
        g.eps = 0.0
    elif change == "alpha":
        g.alpha_min[1] = 0.5
    elif change == "count":
        g.n_fb_min[0] = -1
    elif change == "H":
        hd.H = 9
        hd.max_children = 2
    else:
        P = None
    need = _lib.lib().sr_heads_propose_workspace(C.byref(_lib.HeadsDesc(2, 256, 2, 512, 8, 2, _lib.SR_F32, 1.0, 1e-5)))
    st = _lib.lib().sr_heads_propose_reflex(C.byref(hd), C.byref(g), *([fake] * 9), fake, fake, P, None, None,
                                            fake, fake, None, None, fake, need, None)
    assert st == _lib.SR_ERR_INVALID, change
    assert _lib.last_error()
