"""GPU parity on randomly drawn valid shapes (fixed seed): every call of the step against the float64 oracle
with the same bars as the dedicated tests, over shapes no single test pins -- tree sizes 1..128 with varied
depth, 1..8 query heads per KV head, D 64/128, head widths 64..512, vocabularies that are any multiple of 8,
fp32 and bf16, temperatures and nucleus thresholds."""
import numpy as np
import pytest

import synth
import test_gpu_accept as TC
import test_gpu_attn as TA
import test_gpu_heads as TH

pytestmark = pytest.mark.gpu


def _topology(rng, T):
    depth = int(rng.integers(1, min(6, T - 1) + 1)) if T > 1 else 1
    return dict(T=T, depth=depth, parents=None if T > 1 else (-1,))


@pytest.mark.parametrize("round_", range(12))
def test_random_shapes(round_):
    rng = np.random.default_rng(9000 + round_)
    # tree-verify attention (App. B.1 Eq. (nodep))
    T = int(rng.choice([1, 2, 5, 8, 16, 31, 32, 48, 64, 96, 128]))
    Hkv, G, D = int(rng.choice([1, 2, 4, 8])), int(rng.integers(1, 9)), int(rng.choice([64, 128]))
    dt, B = str(rng.choice(["bf16", "f32"])), int(rng.integers(1, 7))
    lo = int(rng.integers(0, 2000))
    hi = lo + int(rng.integers(0, 3000))
    cfg = synth.scaled(synth.SHAPE_7B, dtype=dt, B=B, Hq=Hkv * G, Hkv=Hkv, D=D, ctx=("uniform", lo, hi),
                       **_topology(rng, T))
    print(f"[random {round_}] attention B={B} T={T} Hkv={Hkv} G={G} D={D} {dt} ctx=[{lo},{hi}]", flush=True)
    TA._check(synth.attn_inputs(cfg, seed=1000 + round_),
              nodes=None if B * T * Hkv * G <= 2048 else TA._sample_nodes(cfg, 4, round_))
    # heads and the fused tree (Sec. 3.2 Eq. (heads); App. B.1 Eq. (slotq))
    T = int(rng.choice([1, 2, 8, 16, 32, 64]))
    H, d = int(rng.integers(1, 6)), int(rng.choice([64, 128, 256, 512]))
    B, V, dt = int(rng.integers(1, 40)), 8 * int(rng.integers(max(8, T), 2500)), str(rng.choice(["bf16", "f32"]))
    cfg = synth.scaled(synth.SHAPE_7B, dtype=dt, B=B, H=H, d=d, V=V, active_frac=float(rng.random()),
                       **_topology(rng, T))
    print(f"[random {round_}] heads B={B} T={T} H={H} d={d} V={V} {dt}", flush=True)
    inp = synth.heads_inputs(cfg, seed=2000 + round_)
    tok, cl, lg, z = TH._gpu_heads(inp)
    ref = TH._oracle_heads(inp)
    if dt == "bf16":
        TH._check_z(inp, z, ref)
    else:
        assert TH.row_rel_err(z.reshape(-1, d), ref["z"].reshape(-1, d)).max() <= 1e-5
    lerr = TH.row_rel_err(lg.reshape(-1, V), ref["logits"].reshape(-1, V)).max()
    assert lerr <= (2e-3 if dt == "bf16" else 1e-5), lerr
    TH._check_fused_tree(inp, tok, cl, lg, range(B))
    # acceptance walk (App. B.2), plain and nucleus
    T, B = int(rng.choice([1, 2, 3, 8, 16, 32, 64, 100, 128])), int(rng.integers(1, 30))
    V, dt = 8 * int(rng.integers(max(2, T), 4000)), str(rng.choice(["bf16", "f32"]))
    top_p, temp = float(rng.choice([1.0, 1.0, 0.95, 0.6])), float(rng.choice([1.0, 0.7, 1.5]))
    cfg = synth.scaled(synth.SHAPE_7B, dtype=dt, B=B, V=V, **_topology(rng, T))
    print(f"[random {round_}] accept B={B} T={T} V={V} {dt} top_p={top_p} temperature={temp}", flush=True)
    TC._compare(synth.accept_inputs(cfg, seed=3000 + round_, target_std=float(rng.choice([0.5, 4.0, 8.0]))),
                temperature=temp, top_p=top_p)
