"""Pins for the oracle's rotary embedding and key re-rotation."""
import numpy as np
import torch
from transformers.models.llama.modeling_llama import apply_rotary_pos_emb

import oracle


def test_hand_worked_case():
    # hd = 4, theta = 100: frequencies 100^0 = 1 and 100^(-1/2) = 0.1.
    x = np.array([[[1.0, 0.0, 0.0, 0.0]]])
    y = oracle.rotate(x, [1], 100.0)[0, 0]
    np.testing.assert_allclose(y, [np.cos(1.0), 0.0, np.sin(1.0), 0.0], atol=1e-15)
    x = np.array([[[0.0, 1.0, 0.0, 0.0]]])
    y = oracle.rotate(x, [10], 100.0)[0, 0]
    np.testing.assert_allclose(y, [0.0, np.cos(1.0), 0.0, np.sin(1.0)], atol=1e-15)


def test_position_zero_is_identity_bitwise():
    x = np.random.default_rng(0).standard_normal((5, 3, 16))
    assert np.array_equal(oracle.rotate(x, np.zeros(5, int), 1e4), x)


def test_composition_and_pair_norms():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((6, 2, 64))
    a = rng.integers(0, 5000, size=6)
    b = rng.integers(0, 12000, size=6)
    two_steps = oracle.rotate(oracle.rotate(x, a, 1e6), b, 1e6)
    np.testing.assert_allclose(two_steps, oracle.rotate(x, a + b, 1e6), atol=1e-11)
    y = oracle.rotate(x, b, 1e4)
    pair = lambda z: z[..., :32] ** 2 + z[..., 32:] ** 2
    np.testing.assert_allclose(pair(y), pair(x), rtol=1e-12)


def test_rerotation_moves_a_cached_key_to_its_new_position():
    rng = np.random.default_rng(2)
    k_raw = rng.standard_normal((4, 2, 32))
    cached = oracle.rotate(k_raw, np.arange(4), 1e4)          # encoded at 0..3
    moved = oracle.rerotate(cached, 300, 1e4)                 # unit now starts at 300
    np.testing.assert_allclose(moved, oracle.rotate(k_raw, 300 + np.arange(4), 1e4), atol=1e-12)


def test_matches_transformers_rotate_half():
    rng = np.random.default_rng(3)
    hd, theta = 64, 1e4
    x = rng.standard_normal((7, 3, hd))
    pos = rng.integers(0, 4000, size=7)
    c, s = oracle.rope_cos_sin(pos, hd, theta)
    cos = torch.as_tensor(np.concatenate([c, c], axis=1))[None]
    sin = torch.as_tensor(np.concatenate([s, s], axis=1))[None]
    xt = torch.as_tensor(x).transpose(0, 1)[None]               # [1][H][n][hd]
    ref, _ = apply_rotary_pos_emb(xt, xt, cos, sin)
    np.testing.assert_allclose(oracle.rotate(x, pos, theta), ref[0].transpose(0, 1).numpy(),
                               atol=1e-13)
