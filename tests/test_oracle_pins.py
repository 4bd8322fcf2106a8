"""Pins of the oracle's per-row math against what mathematics and library routines fix.

None of these re-types the oracle's own formula: each compares with a closed form, a
hand-worked value, brute force in plain Python, or an independent library routine.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle.model import attend_segment, rmsnorm, rope, round_storage, silu


# ----------------------------------------------------------------------------- storage rounding
def test_bf16_rounding_matches_torch_rne():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
                        [0.0, -0.0, 1.0, -1.0, 65504.0, 1e-30]])
    # exact ties between two bf16 values: low 16 bits = 0x8000, both parities of bit 16
    ties = (np.arange(0x3F800000, 0x3F800000 + 64 * 0x10000, 0x10000, dtype=np.uint32) | 0x8000)
    x = np.concatenate([x, ties.view(np.float32).astype(np.float64)])
    want = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    got = round_storage(x, "bf16")
    assert np.array_equal(got, want)


def test_f32_rounding_is_ieee_single():
    x = np.array([1.0 + 2.0 ** -30, 1.0 / 3.0, math.pi])
    got = round_storage(x, "f32")
    assert got[0] == 1.0
    assert got[1] == float(np.float32(1.0) / np.float32(3.0))
    assert got[2] == 3.1415927410125732


# ----------------------------------------------------------------------------- RMSNorm
def test_rmsnorm_hand_value():
    # x = (3, 4): mean of squares 12.5, rms sqrt(12.5); gain (1, 2), eps 0
    y = rmsnorm(np.array([3.0, 4.0]), np.array([1.0, 2.0]), 0.0)
    r = math.sqrt(12.5)
    assert y == pytest.approx([3.0 / r, 8.0 / r], rel=1e-15)


def test_rmsnorm_constant_row_closed_form():
    for c in (0.5, -3.0, 1e-3):
        g = np.linspace(0.5, 2.0, 16)
        y = rmsnorm(np.full(16, c), g, 1e-6)
        assert np.allclose(y, g * c / math.sqrt(c * c + 1e-6), rtol=1e-14, atol=0)


def test_rmsnorm_matches_torch_library():
    rng = np.random.default_rng(2)
    x, g = rng.standard_normal((5, 64)), rng.standard_normal(64)
    want = torch.nn.functional.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g), eps=1e-6).numpy()
    assert np.allclose(rmsnorm(x, g, 1e-6), want, rtol=1e-13, atol=1e-15)


# ----------------------------------------------------------------------------- RoPE
def test_rope_position_zero_is_identity():
    u = np.random.default_rng(3).standard_normal((3, 2, 8))
    assert np.array_equal(rope(u, np.zeros(3, dtype=int), 10000.0), u)


def test_rope_hd2_is_plane_rotation():
    # hd = 2: one pair (0, 1), frequency theta^0 = 1, so the angle is the position itself
    for p in (1, 2, 7):
        got = rope(np.array([[[1.0, 0.0]]]), np.array([p]), 10000.0)[0, 0]
        assert got == pytest.approx([math.cos(p), math.sin(p)], abs=1e-15)
        got = rope(np.array([[[0.0, 1.0]]]), np.array([p]), 10000.0)[0, 0]
        assert got == pytest.approx([-math.sin(p), math.cos(p)], abs=1e-15)


def test_rope_hd4_pairs_first_and_second_half():
    # hd = 4, theta = 10000: pair (0, 2) turns by p, pair (1, 3) by p * 10000^(-1/2) = p / 100
    p = 3
    u = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    a, b = p, p / 100.0
    want = [1 * math.cos(a) - 3 * math.sin(a), 2 * math.cos(b) - 4 * math.sin(b),
            3 * math.cos(a) + 1 * math.sin(a), 4 * math.cos(b) + 2 * math.sin(b)]
    assert rope(u, np.array([p]), 10000.0)[0, 0] == pytest.approx(want, abs=1e-14)


def test_rope_preserves_norm_and_depends_on_relative_position():
    rng = np.random.default_rng(4)
    q, k = rng.standard_normal((1, 1, 128)), rng.standard_normal((1, 1, 128))
    for m, n, d in ((5, 2, 11), (100, 40, 250), (0, 0, 282)):
        qm, kn = rope(q, np.array([m]), 1e4), rope(k, np.array([n]), 1e4)
        assert np.linalg.norm(qm) == pytest.approx(np.linalg.norm(q), rel=1e-13)
        s1 = float(np.sum(qm * kn))
        s2 = float(np.sum(rope(q, np.array([m + d]), 1e4) * rope(k, np.array([n + d]), 1e4)))
        assert s1 == pytest.approx(s2, rel=1e-11, abs=1e-11)


# ----------------------------------------------------------------------------- SiLU
def test_silu_closed_forms():
    assert silu(np.array([0.0]))[0] == 0.0
    assert silu(np.array([1.0]))[0] == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)
    z = np.linspace(-8, 8, 101)
    assert np.allclose(silu(z), torch.nn.functional.silu(torch.from_numpy(z)).numpy(), rtol=1e-14, atol=1e-16)


# ----------------------------------------------------------------------------- attention
def _brute_attention(q, pos, keys, values, scale):
    """Plain Python loops, float64, math.exp."""
    out = []
    for i in range(len(q)):
        sc = [scale * sum(q[i][d] * keys[j][d] for d in range(len(q[i]))) for j in range(pos[i] + 1)]
        mx = max(sc)
        w = [math.exp(s - mx) for s in sc]
        tot = sum(w)
        out.append([sum(w[j] * values[j][d] for j in range(len(w))) / tot for d in range(len(values[0]))])
    return np.array(out)


@pytest.mark.parametrize("n,pos0,hd", [(1, 0, 4), (1, 6, 8), (5, 0, 4), (4, 3, 8), (3, 9, 2)])
def test_attention_brute_force(n, pos0, hd):
    rng = np.random.default_rng(10 + n + pos0)
    kv = pos0 + n
    q, k, v = rng.standard_normal((n, hd)), rng.standard_normal((kv, hd)), rng.standard_normal((kv, hd))
    pos = np.arange(pos0, pos0 + n)
    got = attend_segment(q, pos, k, v, 1 / math.sqrt(hd))
    want = _brute_attention(q.tolist(), pos.tolist(), k.tolist(), v.tolist(), 1 / math.sqrt(hd))
    assert np.allclose(got, want, rtol=1e-13, atol=1e-14)


def test_attention_single_key_returns_its_value():
    rng = np.random.default_rng(5)
    v = rng.standard_normal((1, 16))
    got = attend_segment(rng.standard_normal((1, 16)), np.array([0]), rng.standard_normal((1, 16)), v, 0.25)
    assert np.array_equal(got, v)


def test_attention_zero_query_averages_visible_values():
    rng = np.random.default_rng(6)
    v = rng.standard_normal((7, 8))
    got = attend_segment(np.zeros((3, 8)), np.array([2, 4, 6]), rng.standard_normal((7, 8)), v, 1.0)
    for i, p in enumerate((2, 4, 6)):
        assert np.allclose(got[i], v[: p + 1].mean(axis=0), rtol=1e-14)


def test_attention_prefill_matches_torch_sdpa_causal():
    rng = np.random.default_rng(7)
    n, hd = 12, 16
    q, k, v = (rng.standard_normal((n, hd)) for _ in range(3))
    got = attend_segment(q, np.arange(n), k, v, 1 / math.sqrt(hd))
    T = lambda a: torch.from_numpy(a)[None, None]
    want = torch.nn.functional.scaled_dot_product_attention(T(q), T(k), T(v), is_causal=True)[0, 0].numpy()
    assert np.allclose(got, want, rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------------------- argmax
def test_argmax_takes_lowest_index_on_ties():
    z = np.array([[0.0, 2.0, 2.0, 1.0], [5.0, 5.0, 5.0, 5.0], [-1.0, -3.0, -1.0, -2.0]])
    assert list(oracle.OracleModel.argmax(z)) == [1, 0, 0]
