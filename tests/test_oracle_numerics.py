"""Pins of the oracle's scalar numerics against library routines and hand values."""
import numpy as np
import pytest
import torch

from oracle import numerics


def test_round_bf16_hand_values():
    r = numerics.round_bf16
    one = 1.0
    assert r(one + 2.0 ** -8) == one                       # tie -> even (1.0)
    assert r(one + 3 * 2.0 ** -8) == one + 2.0 ** -6       # tie -> even (odd neighbour rejected)
    assert r(one + 2.0 ** -8 + 2.0 ** -20) == one + 2.0 ** -7
    assert r(-3.0) == -3.0
    assert r(0.0) == 0.0
    assert np.isinf(r(3.5e38))
    assert np.isnan(r(np.nan))


def test_round_bf16_matches_torch_conversion():
    # torch converts float32 -> bfloat16 with round-to-nearest-even; on values
    # that are exact in float32 that is the same rounding as ours.
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(200000) * np.exp(rng.uniform(-20, 20, 200000))).astype(np.float32)
    ours = numerics.round_bf16(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ours, ref)


def test_layernorm_matches_torch(torch_cpu):
    rng = np.random.default_rng(1)
    x = rng.standard_normal((37, 48)) * 3 + 1
    g, b = rng.standard_normal(48), rng.standard_normal(48)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (48,), torch.from_numpy(g),
                                         torch.from_numpy(b), eps=1e-5).numpy()
    np.testing.assert_allclose(numerics.layernorm(x, g, b), ref, rtol=1e-12, atol=1e-12)


def test_activations_match_torch(torch_cpu):
    x = np.linspace(-9, 9, 1001)
    t = torch.from_numpy(x)
    np.testing.assert_allclose(numerics.silu(x), torch.nn.functional.silu(t).numpy(), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(numerics.gelu(x), torch.nn.functional.gelu(t).numpy(), rtol=1e-13, atol=1e-15)


def test_softmax_matches_torch_and_is_shift_invariant(torch_cpu):
    rng = np.random.default_rng(2)
    s = rng.standard_normal((5, 17)) * 10
    ref = torch.softmax(torch.from_numpy(s), -1).numpy()
    np.testing.assert_allclose(numerics.softmax(s), ref, rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(numerics.softmax(s + 123.0), ref, rtol=1e-12, atol=1e-16)
    np.testing.assert_allclose(numerics.softmax(s).sum(-1), 1.0, rtol=1e-14)


def test_linear_convention():
    # V' = V W^T + b with W stored [out, in]
    x = np.array([[1.0, 2.0]])
    w = np.array([[1.0, 0.0], [0.0, 1.0], [1.0, 1.0]])
    assert numerics.linear(x, w, np.array([0.5, 0, 0])).tolist() == [[1.5, 2.0, 3.0]]
