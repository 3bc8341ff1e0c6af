"""Pins of the oracle's bfloat16 rounding and RoPE (Eq. 3) against things
other than the oracle itself: torch's float32->bfloat16 cast, the textbook
2-D rotation matrix, HuggingFace's Qwen2 rotary embedding, and the algebraic
properties Eq. 3 states (relative-offset dot products, composition)."""
import math

import numpy as np
import pytest
import torch

from oracle import numerics, rope


def test_bf16_rounding_matches_torch_cast():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(100),
        # exact ties of the 16 dropped bits, both parities of the kept lsb
        (np.arange(1000, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
        (np.arange(1000, dtype=np.uint32) << 16 | 0x7FFF).view(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 1e-40, -1e-40, 3.4e38], np.float32),
    ])
    ours = numerics.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.isnan(numerics.bf16_bits_to_f32(numerics.f32_to_bf16_bits(np.float32(np.nan))))


def test_inv_freq_closed_form():
    w = rope.inv_freq(1e4, 4)
    assert w[0] == 1.0
    assert abs(w[1] - 0.01) < 1e-17
    w = rope.inv_freq(1e6, 128)
    assert w[0] == 1.0 and abs(w[32] - 1e-3) < 1e-15


@pytest.mark.parametrize("p", [0, 1, 7, 1000])
def test_rotation_matches_textbook_matrix(p):
    """d = 4, theta = 1e4: pairs (0,2) turn by p rad, pairs (1,3) by 0.01 p rad,
    each as the 2-D rotation matrix [[cos, -sin], [sin, cos]]."""
    x = np.array([1.0, 2.0, 3.0, 4.0])
    y = rope.apply_at_positions(x[None, :], [p], 1e4, dtype=np.float64)[0]
    for (i, j), a in (((0, 2), p * 1.0), ((1, 3), p * 0.01)):
        R = np.array([[math.cos(a), -math.sin(a)], [math.sin(a), math.cos(a)]])
        assert np.allclose(y[[i, j]], R @ x[[i, j]], rtol=0, atol=1e-12)


def test_zero_offset_is_identity_exactly():
    c, s = rope.angle_table(1e6, 128, [0, 0])
    assert np.all(c == 1.0) and np.all(s == 0.0)
    x = np.random.default_rng(1).standard_normal((3, 128))
    assert np.array_equal(rope.rotate(x, c[0], s[0]), x)


def test_matches_huggingface_qwen2_rotary():
    from transformers.models.qwen2 import modeling_qwen2 as m
    from transformers import Qwen2Config

    d, theta = 64, 1e4
    cfg = Qwen2Config(hidden_size=4 * d, num_attention_heads=4, num_key_value_heads=2,
                      rope_theta=theta, max_position_embeddings=4096)
    emb = m.Qwen2RotaryEmbedding(cfg)
    pos = torch.arange(0, 160, dtype=torch.long)[None, :]
    x = torch.randn(1, 2, 160, d, dtype=torch.float64, generator=torch.Generator().manual_seed(0))
    cos, sin = emb(x.float(), pos)
    q_hf, _ = m.apply_rotary_pos_emb(x, x, cos.double(), sin.double())
    ours = rope.apply_at_positions(x.numpy(), np.arange(160), theta, axis=-2)
    # HF builds its frequencies in float32: allow its angle error at p < 160
    assert np.allclose(ours, q_hf.numpy(), rtol=0, atol=2e-5 * float(x.abs().max()))


def test_relative_offset_property_eq3():
    """q'_s . k'_t = q_s^T R^(t-s) k_t (the property Eq. 3 states)."""
    rng = np.random.default_rng(2)
    d, theta = 128, 1e6
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    for s_, t in ((3, 50), (50, 1050), (30000, 12)):
        lhs = rope.apply_at_positions(q[None], [s_], theta, dtype=np.float64)[0] @ \
            rope.apply_at_positions(k[None], [t], theta, dtype=np.float64)[0]
        rhs = q @ rope.apply_at_positions(k[None], [t - s_], theta, dtype=np.float64)[0]
        assert abs(lhs - rhs) < 1e-9 * np.linalg.norm(q) * np.linalg.norm(k)


def test_composition_and_norm():
    """R^a R^b = R^(a+b) and |R x| = |x| (float64 tables)."""
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 128))
    for a, b in ((50, 1000), (-32000, 17), (12345, -12345)):
        ab = rope.apply_at_positions(rope.apply_at_positions(x, [a] * 5, 1e6, dtype=np.float64),
                                     [b] * 5, 1e6, dtype=np.float64)
        direct = rope.apply_at_positions(x, [a + b] * 5, 1e6, dtype=np.float64)
        assert np.max(np.abs(ab - direct)) < 1e-10 * np.max(np.abs(x))
        assert np.allclose(np.linalg.norm(ab, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)


def test_reuse_at_new_position_with_float32_table():
    """A key cached at 50 and corrected by R^1000 equals the key rotated at 1050
    (the Sec. 3.2 example), up to the float32 rounding of the tables."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((1, 128))
    cached = rope.apply_at_positions(x, [50], 1e6)
    c, s = rope.angle_table(1e6, 128, [1000])
    moved = rope.rotate(cached, c[0], s[0])
    direct = rope.apply_at_positions(x, [1050], 1e6, dtype=np.float64)
    assert np.max(np.abs(moved - direct)) < 4 * 2.0**-24 * 4 * np.max(np.abs(x))
