"""Pins of the oracle's components against library routines, closed forms and brute force.

None of these re-types the oracle's formula: each compares it with an
independent implementation (torch's bf16 conversion, rms_norm, silu and
scaled_dot_product_attention) or with values fixed by mathematics.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle.accept import accept_length, argmax_lowest, top2_gap
from oracle.bf16 import BF16_MAX, bf16_bits, from_bf16_bits, round_bf16
from oracle.decoder import attention, rms_norm, rope, silu


# ----------------------------------------------------------------------- bf16
def _torch_bf16(x32: np.ndarray) -> np.ndarray:
    return torch.from_numpy(x32).to(torch.bfloat16).to(torch.float64).numpy()


def test_bf16_matches_torch_on_random_fp32_bit_patterns():
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 2 ** 32, size=400_000, dtype=np.uint64).astype(np.uint32)
    x32 = bits.view(np.float32)
    ours = round_bf16(x32.astype(np.float64))
    ref = _torch_bf16(x32)
    nan = np.isnan(x32)
    assert np.isnan(ours[nan]).all()
    np.testing.assert_array_equal(ours[~nan], ref[~nan])


def test_bf16_edge_cases_match_torch():
    specials = [0.0, -0.0, np.inf, -np.inf, 1.0, -1.0,
                1.0 + 2 ** -8,            # exact tie -> even (1.0)
                1.0 + 3 * 2 ** -8,        # tie -> even (1 + 2^-6)
                1.0 + 2 ** -8 + 2 ** -20,  # just above the tie -> up
                2 ** -126, 2 ** -127, 2 ** -133, 2 ** -134, 3 * 2 ** -134, 2 ** -149,
                BF16_MAX, 3.3895313892515355e38, 3.4e38, 3.4028234663852886e38,
                65504.0, 1e-40, -1e-40, 0.1, 1 / 3]
    x32 = np.array(specials, dtype=np.float32)
    np.testing.assert_array_equal(round_bf16(x32.astype(np.float64)), _torch_bf16(x32))


def test_bf16_float64_inputs_round_to_nearest_neighbour():
    # Brute force: the result is one of the two bf16 neighbours and the nearer one.
    rng = np.random.default_rng(1)
    x = rng.standard_normal(20000) * np.exp2(rng.integers(-30, 30, 20000))
    r = round_bf16(x)
    r32 = r.astype(np.float32)
    assert (r32.astype(np.float64) == r).all()
    assert ((r32.view(np.uint32) & 0xFFFF) == 0).all()          # representable in bf16
    up = from_bf16_bits(bf16_bits(r).astype(np.int64) + 1)       # next value away from 0
    dn = from_bf16_bits(bf16_bits(r).astype(np.int64) - 1)
    err = np.abs(x - r)
    assert (err <= np.abs(x - up) + 0).all() and (err <= np.abs(x - dn) + 0).all()


def test_bf16_bits_roundtrip():
    b = np.arange(0, 2 ** 16, dtype=np.uint32).astype(np.uint16)
    v = from_bf16_bits(b)
    fin = np.isfinite(v)
    np.testing.assert_array_equal(bf16_bits(v[fin]), b[fin])


# -------------------------------------------------------------------- RMSNorm
def test_rms_norm_matches_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((7, 96)) * 3
    g = 1 + 0.1 * rng.standard_normal(96)
    ref = F.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-6).numpy()
    np.testing.assert_allclose(rms_norm(x, g, 1e-6), ref, rtol=1e-13, atol=1e-13)


def test_rms_norm_constant_row_gives_gain():
    x = np.full((1, 8), -5.0)
    g = np.arange(1, 9, dtype=np.float64)
    np.testing.assert_allclose(rms_norm(x, g, 0.0), -g[None], rtol=1e-15)


# ----------------------------------------------------------------------- RoPE
def test_rope_identity_at_position_zero():
    x = np.random.default_rng(3).standard_normal((1, 3, 16))
    np.testing.assert_array_equal(rope(x, np.array([0]), 10000.0), x)


def test_rope_explicit_angles_d4():
    # D = 4: pairs (0,2) and (1,3); angles p*base^0 and p*base^(-1/2).
    x = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    p, base = 3.0, 100.0
    a0, a1 = p * 1.0, p / 10.0
    want = [1 * math.cos(a0) - 3 * math.sin(a0), 2 * math.cos(a1) - 4 * math.sin(a1),
            3 * math.cos(a0) + 1 * math.sin(a0), 4 * math.cos(a1) + 2 * math.sin(a1)]
    np.testing.assert_allclose(rope(x, np.array([p]), base)[0, 0], want, rtol=1e-14)


def test_rope_scores_depend_only_on_relative_position():
    rng = np.random.default_rng(4)
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    s = [float(np.sum(rope(q, np.array([m]), 1e4) * rope(k, np.array([m - 7]), 1e4)))
         for m in (7, 100, 5000, 65000)]
    np.testing.assert_allclose(s, s[0], rtol=1e-9)
    n = np.linalg.norm(rope(q, np.array([12345]), 1e4))
    assert abs(n - np.linalg.norm(q)) < 1e-12


# ---------------------------------------------------------------------- SwiGLU
def test_silu_matches_torch():
    a = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(silu(a), F.silu(torch.from_numpy(a)).numpy(), rtol=1e-14, atol=1e-300)
    assert silu(np.array([0.0]))[0] == 0.0


# ------------------------------------------------------------------- attention
def _sdpa_reference(q, K, V, q_pos, group):
    """torch's scaled_dot_product_attention with an explicit position mask."""
    n, Hq, D = q.shape
    S = K.shape[1]
    Kr = torch.from_numpy(np.repeat(K, group, axis=0))     # [Hq, S, D]
    Vr = torch.from_numpy(np.repeat(V, group, axis=0))
    qt = torch.from_numpy(q.transpose(1, 0, 2).copy())     # [Hq, n, D]
    mask = torch.from_numpy(np.arange(S)[None, :] <= np.asarray(q_pos)[:, None])
    o = F.scaled_dot_product_attention(qt[None], Kr[None], Vr[None], attn_mask=mask[None, None])
    return o[0].numpy().transpose(1, 0, 2)


@pytest.mark.parametrize("n,S0,Hq,Hkv,D", [(1, 37, 4, 2, 16), (5, 100, 8, 2, 32), (9, 16, 4, 1, 8)])
def test_attention_matches_sdpa(n, S0, Hq, Hkv, D):
    rng = np.random.default_rng(n * 100 + S0)
    q = rng.standard_normal((n, Hq, D))
    K = rng.standard_normal((Hkv, S0 + n, D))
    V = rng.standard_normal((Hkv, S0 + n, D))
    pos = S0 + np.arange(n)
    np.testing.assert_allclose(attention(q, K, V, pos, Hq // Hkv), _sdpa_reference(q, K, V, pos, Hq // Hkv),
                               rtol=1e-12, atol=1e-12)


def test_attention_closed_forms():
    rng = np.random.default_rng(5)
    D = 16
    V = rng.standard_normal((2, 5, D))
    K = rng.standard_normal((2, 5, D))
    # position 0 sees only key 0: output is v_0 of its kv head
    q = rng.standard_normal((1, 4, D))
    o = attention(q, K, V, np.array([0]), 2)
    np.testing.assert_allclose(o[0, 1], V[0, 0], rtol=1e-15)
    np.testing.assert_allclose(o[0, 3], V[1, 0], rtol=1e-15)
    # zero query: uniform weights over the visible keys 0..3
    o = attention(np.zeros((1, 4, D)), K, V, np.array([3]), 2)
    np.testing.assert_allclose(o[0, 2], V[1, :4].mean(axis=0), rtol=1e-13)
    # scale 1/sqrt(D): score gap ln 3 gives weights 1/4 and 3/4
    K2 = np.zeros((1, 2, D)); K2[0, 1, 0] = 1.0
    q2 = np.zeros((1, 1, D)); q2[0, 0, 0] = math.log(3.0) * math.sqrt(D)
    V2 = np.zeros((1, 2, D)); V2[0, 0, 1] = 1.0; V2[0, 1, 2] = 1.0
    o = attention(q2, K2, V2, np.array([1]), 1)
    np.testing.assert_allclose(o[0, 0, 1:3], [0.25, 0.75], rtol=1e-14)


# -------------------------------------------------------------- argmax / accept
def test_argmax_ties_go_to_lowest_id():
    z = np.zeros((4, 10))
    z[0, [3, 7]] = 5.0
    z[1, :] = -1.0
    z[2, 9] = 1.0
    z[3, [0, 9]] = 2.0
    np.testing.assert_array_equal(argmax_lowest(z), [3, 0, 9, 0])
    with pytest.raises(ValueError):
        argmax_lowest(np.array([[0.0, np.nan]]))


def test_accept_length_brute_force():
    rng = np.random.default_rng(6)
    for _ in range(2000):
        n = int(rng.integers(0, 7))
        g = rng.integers(0, 3, size=n + 1)
        d = rng.integers(0, 3, size=n)
        want = 0
        while want < n and all(d[m] == g[m] for m in range(want + 1)):
            want += 1
        assert accept_length(d, g) == want


def test_top2_gap():
    z = np.array([[1.0, 5.0, 4.5, -3.0], [2.0, 2.0, 0.0, 1.0]])
    np.testing.assert_allclose(top2_gap(z), [0.5, 0.0])
