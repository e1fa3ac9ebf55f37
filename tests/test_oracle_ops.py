"""Pins of the oracle's building blocks against closed forms, special cases
and independent library implementations (CPU only)."""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import model as om

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_rms_norm_hand_values():
    # rms([3, 4]) = sqrt((9 + 16) / 2) = sqrt(12.5)
    y = om.rms_norm(np.array([[3.0, 4.0]]), np.array([1.0, 1.0]), 0.0)
    r = math.sqrt(12.5)
    assert np.allclose(y, [[3 / r, 4 / r]], rtol=0, atol=1e-15)
    # gain scales per column, eps enters under the square root
    y = om.rms_norm(np.array([[1.0, -1.0, 1.0, -1.0]]), np.array([2.0, 1.0, 0.5, 0.0]), 3.0)
    assert np.allclose(y, [[1.0, -0.5, 0.25, 0.0]], atol=1e-15)  # 1/sqrt(1+3) = 0.5
    assert np.all(om.rms_norm(np.zeros((2, 8)), np.ones(8), 1e-6) == 0)


def test_rms_norm_matches_torch():
    rng = np.random.default_rng(0)
    x, g = rng.standard_normal((5, 64)), rng.standard_normal(64)
    ref = torch.nn.functional.rms_norm(torch.tensor(x), (64,), torch.tensor(g), eps=1e-6).numpy()
    assert np.allclose(om.rms_norm(x, g, 1e-6), ref, rtol=1e-13, atol=1e-13)


def test_silu_hand_values():
    assert om.silu(np.float64(0.0)) == 0.0
    assert abs(om.silu(np.float64(1.0)) - 0.7310585786300049) < 1e-15   # 1/(1+e^-1)
    assert abs(om.silu(np.float64(-2.0)) - (-0.23840584404423515)) < 1e-15


def test_rope_closed_form_d4():
    # d = 4, theta = 10000: pairs (0, 2) and (1, 3), frequencies 1 and 1/100.
    x = np.zeros((1, 1, 4))
    x[0, 0, 0] = 1.0
    y = om.rope(x, np.array([1.0]), 1e4)[0, 0]
    assert np.allclose(y, [math.cos(1), 0, math.sin(1), 0], atol=1e-15)
    x = np.zeros((1, 1, 4))
    x[0, 0, 3] = 1.0
    y = om.rope(x, np.array([50.0]), 1e4)[0, 0]
    # (x1, x3) = (0, 1) rotated by 0.5 rad -> (-sin 0.5, cos 0.5)
    assert np.allclose(y, [0, -math.sin(0.5), 0, math.cos(0.5)], atol=1e-15)


def test_rope_properties():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((3, 2, 128))
    k = rng.standard_normal((3, 2, 128))
    assert np.allclose(om.rope(q, np.zeros(3), 1e6), q, atol=0)            # position 0: identity
    pos = np.array([5.0, 900.0, 7000.0])
    assert np.allclose(np.linalg.norm(om.rope(q, pos, 1e6), axis=-1), np.linalg.norm(q, axis=-1))
    # q.k depends only on the position difference
    a = np.sum(om.rope(q, pos, 1e6) * om.rope(k, pos - 3, 1e6), axis=-1)
    b = np.sum(om.rope(q, pos + 1000, 1e6) * om.rope(k, pos + 997, 1e6), axis=-1)
    assert np.allclose(a, b, atol=1e-9)


def test_rope_matches_transformers_rotate_half():
    from transformers.models.qwen2 import modeling_qwen2 as mq
    rng = np.random.default_rng(2)
    T, nh, d, theta = 7, 3, 64, 1e4
    x = rng.standard_normal((T, nh, d))
    pos = np.arange(100, 100 + T, dtype=np.float64)
    inv = 1.0 / theta ** (np.arange(0, d, 2) / d)
    emb = np.concatenate([pos[:, None] * inv[None], pos[:, None] * inv[None]], -1)
    cos, sin = torch.tensor(np.cos(emb))[None], torch.tensor(np.sin(emb))[None]
    xt = torch.tensor(x.transpose(1, 0, 2))[None]            # [1, heads, T, d]
    ref, _ = mq.apply_rotary_pos_emb(xt, xt, cos, sin)
    assert np.allclose(om.rope(x, pos, theta), ref[0].numpy().transpose(1, 0, 2), atol=1e-12)


def test_attention_single_key_returns_value():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 2, 16))
    K = rng.standard_normal((1, 1, 16))
    V = rng.standard_normal((1, 1, 16))
    out = om.attention(q, K, V, np.array([0]))
    assert np.allclose(out[0, 0], V[0, 0]) and np.allclose(out[0, 1], V[0, 0])


def test_attention_zero_query_averages_visible_values():
    rng = np.random.default_rng(4)
    K = rng.standard_normal((1, 6, 8))
    V = rng.standard_normal((1, 6, 8))
    out = om.attention(np.zeros((2, 1, 8)), K, V, np.array([2, 5]))
    assert np.allclose(out[0, 0], V[0, :3].mean(0)) and np.allclose(out[1, 0], V[0].mean(0))


def test_attention_is_causal():
    rng = np.random.default_rng(5)
    q = rng.standard_normal((3, 4, 8))
    K, V = rng.standard_normal((2, 10, 8)), rng.standard_normal((2, 10, 8))
    pos = np.array([4, 5, 6])
    base = om.attention(q, K, V, pos)
    K2, V2 = K.copy(), V.copy()
    K2[:, 7:] = 1e3
    V2[:, 7:] = -1e3
    assert np.array_equal(om.attention(q, K2, V2, pos), base)


def test_gqa_reduces_to_mha_on_repeated_heads():
    rng = np.random.default_rng(6)
    q = rng.standard_normal((4, 6, 8))
    K, V = rng.standard_normal((2, 9, 8)), rng.standard_normal((2, 9, 8))
    pos = np.array([5, 6, 7, 8])
    gqa = om.attention(q, K, V, pos)
    mha = om.attention(q, np.repeat(K, 3, axis=0), np.repeat(V, 3, axis=0), pos)
    assert np.allclose(gqa, mha, atol=1e-14)


def test_attention_matches_torch_sdpa():
    rng = np.random.default_rng(7)
    T, nq, nkv, d, S = 5, 8, 2, 32, 40
    q = rng.standard_normal((T, nq, d))
    K, V = rng.standard_normal((nkv, S, d)), rng.standard_normal((nkv, S, d))
    pos = np.arange(S - T, S)
    mask = torch.tensor(np.arange(S)[None, :] <= pos[:, None])
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q.transpose(1, 0, 2))[None], torch.tensor(K)[None], torch.tensor(V)[None],
        attn_mask=mask, enable_gqa=True)[0].numpy().transpose(1, 0, 2)
    assert np.allclose(om.attention(q, K, V, pos), ref, atol=1e-12)


def test_greedy_ties_to_lowest_index_and_rejects_nan():
    assert om.greedy(np.array([0.5, 2.0, -1.0, 2.0])) == 1
    assert om.greedy(np.array([3.0, 3.0])) == 0
    with pytest.raises(FloatingPointError):
        om.greedy(np.array([0.0, np.nan, 1.0]))
    with pytest.raises(FloatingPointError):
        om.greedy(np.array([0.0, np.inf]))


def test_top2_margin():
    assert om.top2_margin(np.array([1.0, 4.0, 3.5])) == 0.5
    assert om.top2_margin(np.array([2.0, 2.0])) == 0.0


def test_verify_block_figure4_example():
    """Figure 4(b): candidates A B C D; target agrees on A B, predicts X."""
    g = json.load(open(os.path.join(GOLDEN, "fig4_token_flow.json")))
    sym = g["symbols"]
    cands = [sym[c] for c in g["candidates"]]
    t = [sym[c] for c in g["target_greedy_after_root_and_prefix"]]
    a, corr = om.verify_block(t, cands, len(cands))
    assert a == g["expected_accepted_len"]
    assert corr == sym[g["expected_correction"]]
    committed = cands[:a] + [corr]
    assert committed == [sym[c] for c in g["expected_committed"]]


def test_verify_block_edge_cases():
    assert om.verify_block([7, 8, 9], [7, 8], 2) == (2, 9)       # full acceptance: bonus token
    assert om.verify_block([7, 8, 9], [1, 8], 2) == (0, 7)       # wrong first candidate
    assert om.verify_block([5], [], 0) == (0, 5)                 # K1 step
