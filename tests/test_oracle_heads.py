"""Pins of the heads oracle (Sec. 3.2 Eq. (heads); App. C future-token proposer) against
library routines, closed forms and hand-computed values."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth


def test_round_bf16_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(200000) * np.exp(rng.uniform(-20, 20, 200000))).astype(np.float32)
    # exact halfway cases: 1 + 2^-8 (tie -> even 1.0), 1 + 3*2^-8 (tie -> 1 + 2^-6)
    ties = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 3 * (1 + 2 ** -8)], dtype=np.float32)
    x = np.concatenate([x, ties])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x.astype(np.float64)), ref)
    assert oracle.round_bf16(np.float64(1 + 2 ** -8)) == 1.0
    assert oracle.round_bf16(np.float64(1 + 3 * 2 ** -8)) == 1 + 2 ** -6


def test_generator_bf16_storage_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(100000).astype(np.float32) * 7
    bits = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(bits, ref)
    np.testing.assert_array_equal(synth.bf16_bits_to_f32(bits),
                                  torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_clip_correction_norm_direction_and_gates():
    rng = np.random.default_rng(2)
    d = rng.standard_normal((4, 64)) * 0.5          # norm ~4 > 1: clipped
    d[1] *= 1e-3                                      # norm ~4e-3 < 1: untouched
    d[3] = 0.0                                        # zero vector stays zero
    act = np.array([1, 1, 0, 1], dtype=np.uint8)
    out = oracle.clip_correction(d, act, 1.0)
    assert math.isclose(np.linalg.norm(out[0]), 1.0, rel_tol=1e-12)
    np.testing.assert_allclose(out[0] / np.linalg.norm(out[0]), d[0] / np.linalg.norm(d[0]), rtol=1e-12)
    np.testing.assert_array_equal(out[1], d[1])
    assert not out[2].any() and not out[3].any()


def test_layer_norm_and_silu_match_torch():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 300)) * 3 + 2
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (300,), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.layer_norm(x, 1e-5), ref, rtol=1e-12, atol=1e-12)
    n = oracle.layer_norm(x, 0.0)
    np.testing.assert_allclose(n.mean(-1), 0, atol=1e-12)
    np.testing.assert_allclose(n.var(-1), 1, rtol=1e-12)
    a = rng.standard_normal(1000) * 6
    np.testing.assert_allclose(oracle.silu(a), torch.nn.functional.silu(torch.from_numpy(a)).numpy(), rtol=1e-13)


def test_heads_hand_example():
    # x = (1, 3): mean 2, variance 1 -> LN(x) = (-1, 1) with eps = 0.
    # A = I, b = 0 -> z = x + SiLU(LN(x)) = (1 - 0.2689414213699951, 3 + 0.7310585786300049).
    # W = [[1,0],[0,1],[1,1]] -> logits = (z0, z1, z0 + z1).
    hidden = np.array([[1.0, 3.0]])
    A = np.eye(2)[None]
    bias = np.zeros((1, 2))
    W = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    out = oracle.heads_forward(hidden, None, None, A, bias, W, ln_eps=0.0)
    z = np.array([0.7310585786300049, 3.7310585786300049])
    np.testing.assert_allclose(out["z"][0, 0], z, rtol=1e-14)
    np.testing.assert_allclose(out["logits"][0, 0], [z[0], z[1], z[0] + z[1]], rtol=1e-14)


def test_heads_zero_weights_reduce_to_residual():
    # SiLU(0) = 0, so with A = 0 and b = 0 every head returns the corrected hidden state itself.
    rng = np.random.default_rng(4)
    B, d, H, V = 3, 32, 3, 50
    hidden = rng.standard_normal((B, d))
    corr = rng.standard_normal((B, d))
    act = np.array([1, 0, 1], dtype=np.uint8)
    out = oracle.heads_forward(hidden, corr, act, np.zeros((H, d, d)), np.zeros((H, d)),
                               rng.standard_normal((V, d)), clip_norm=0.5)
    for h in range(H):
        np.testing.assert_array_equal(out["z"][:, h], out["x"])
    np.testing.assert_array_equal(out["x"][1], hidden[1])
    assert math.isclose(np.linalg.norm(out["x"][0] - hidden[0]), 0.5, rel_tol=1e-12)


def test_heads_match_torch_module_composition():
    rng = np.random.default_rng(5)
    B, d, H, V = 4, 48, 3, 97
    hidden = rng.standard_normal((B, d))
    corr = rng.standard_normal((B, d)) * 0.3
    act = np.array([1, 1, 0, 1], dtype=np.uint8)
    A = rng.standard_normal((H, d, d)) * 0.1
    bias = rng.standard_normal((H, d)) * 0.1
    W = rng.standard_normal((V, d)) * 0.1
    out = oracle.heads_forward(hidden, corr, act, A, bias, W, clip_norm=1.0, ln_eps=1e-5)
    th = torch.from_numpy(hidden)
    tc = torch.from_numpy(corr)
    norms = tc.norm(dim=1, keepdim=True)
    tx = th + tc * torch.clamp(1.0 / norms, max=1.0) * torch.from_numpy(act).double()[:, None]
    tn = torch.nn.functional.layer_norm(tx, (d,), eps=1e-5)
    for h in range(H):
        tz = tx + torch.nn.functional.silu(torch.nn.functional.linear(tn, torch.from_numpy(A[h]), torch.from_numpy(bias[h])))
        np.testing.assert_allclose(out["z"][:, h], tz.numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(out["logits"][:, h], torch.nn.functional.linear(tz, torch.from_numpy(W)).numpy(),
                                   rtol=1e-11, atol=1e-11)


def test_heads_rounding_points_are_bf16():
    rng = np.random.default_rng(6)
    B, d, H, V = 2, 64, 2, 30
    out = oracle.heads_forward(rng.standard_normal((B, d)), None, None, rng.standard_normal((H, d, d)) * .05,
                               rng.standard_normal((H, d)) * .05, rng.standard_normal((V, d)),
                               round_fn=oracle.round_bf16)
    for key in ("n", "z"):
        v = out[key]
        np.testing.assert_array_equal(v, torch.from_numpy(v).float().to(torch.bfloat16).double().numpy())
