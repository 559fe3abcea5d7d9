"""Pins for the oracle's rotary rebinding (Eq. (4), Eq. (5), Eq. (12)).

Each test checks the oracle against something other than itself: closed forms,
transformers' own (M-)RoPE routines run in float64 as library references, and the
defining properties of a rotation (pair norms, relative-position scores,
composition, axis isolation).
"""
import math

import numpy as np
import pytest
import torch

from oracle import inv_freq, pair_axis, rotate_keys

RNG = np.random.default_rng(7)


def test_inv_freq_closed_forms():
    f = inv_freq(1e6, 64)
    assert f[0] == 1.0
    assert f[16] == pytest.approx(1e-3, rel=1e-15)        # 1e6^(-32/64)
    g = inv_freq(1e4, 128)
    assert g[32] == pytest.approx(1e-2, rel=1e-15)        # 1e4^(-64/128)
    ratio = g[1:] / g[:-1]
    assert np.allclose(ratio, 1e4 ** (-2 / 128), rtol=1e-13, atol=0)


def test_pair_axis_sectioned_explicit():
    assert pair_axis(64, (8, 12, 12), False).tolist() == [0] * 8 + [1] * 12 + [2] * 12
    assert pair_axis(8, (1, 2, 1), False).tolist() == [0, 1, 1, 2]
    with pytest.raises(ValueError):
        pair_axis(64, (8, 12, 11), False)


def test_pair_axis_interleaved_plain_mod3():
    # [22, 21, 21] over 64 pairs is exactly "pair i -> axis i mod 3".
    assert pair_axis(128, (22, 21, 21), True).tolist() == [i % 3 for i in range(64)]


@pytest.mark.parametrize("sections", [(24, 20, 20), (22, 21, 21), (16, 24, 24), (24, 22, 18), (20, 18, 26)])
def test_pair_axis_interleaved_matches_qwen3vl(sections):
    from transformers.models.qwen3_vl.modeling_qwen3_vl import Qwen3VLTextRotaryEmbedding
    P = 64
    # Tag each axis' frequency slot with its axis id; the library's interleave
    # picks, per pair, which axis' slot survives.
    freqs = torch.stack([torch.full((1, 1, P), float(a)) for a in range(3)])
    picked = Qwen3VLTextRotaryEmbedding.apply_interleaved_mrope(None, freqs, list(sections))
    assert picked[0, 0].long().tolist() == pair_axis(128, sections, True).tolist()


def test_quarter_and_half_turn_closed_form():
    # theta = 4, d = 4: inv_freq = [1, 1/2].  At position pi on every axis, pair 0
    # (x0, x2) turns by pi and pair 1 (x1, x3) by pi/2:
    #   y = [-x0, -x3, -x2, x1].
    invf = inv_freq(4.0, 4)
    assert invf.tolist() == [1.0, 0.5]
    axis = pair_axis(4, (2, 0, 0), False)
    x = np.array([1.5, -2.0, 0.25, 3.0])
    y = rotate_keys(x, np.full(3, math.pi), invf, axis)
    assert np.allclose(y, [-1.5, -3.0, -0.25, -2.0], atol=1e-15)
    # A quarter turn of e_0 lands on e_{d/2} (positive orientation).
    y = rotate_keys(np.array([1.0, 0, 0, 0]), np.full(3, math.pi / 2), invf, axis)
    assert np.allclose(y, [0, 0, 1, 0], atol=1e-15)


def _hf_cos_sin(pos, invf):
    """cos/sin in the library's [3, 1, S, D] layout for per-axis positions pos [S, 3]."""
    fr = torch.from_numpy(pos.T[:, :, None] * invf[None, None, :])     # [3, S, P]
    emb = torch.cat([fr, fr], dim=-1)[:, None]                          # [3, 1, S, D]
    return emb.cos(), emb.sin()


@pytest.mark.parametrize("D,sections", [(128, (16, 24, 24)), (64, (8, 12, 12))])
def test_matches_qwen2vl_mrope(D, sections):
    from transformers.models.qwen2_vl.modeling_qwen2_vl import apply_multimodal_rotary_pos_emb
    S = 37
    x = RNG.standard_normal((1, 2, S, D))
    pos = RNG.uniform(0, 5000, size=(S, 3))
    invf = inv_freq(1e6, D)
    cos, sin = _hf_cos_sin(pos, invf)
    xt = torch.from_numpy(x)
    _, ref = apply_multimodal_rotary_pos_emb(xt, xt, cos, sin, list(sections), unsqueeze_dim=1)
    ours = rotate_keys(x, pos[None, None], invf, pair_axis(D, sections, False))
    assert np.allclose(ours, ref.numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("sections", [(24, 20, 20), (22, 21, 21)])
def test_matches_qwen3vl_interleaved(sections):
    from transformers.models.qwen3_vl.modeling_qwen3_vl import (Qwen3VLTextRotaryEmbedding,
                                                                 apply_rotary_pos_emb)
    D, S = 128, 29
    x = RNG.standard_normal((1, 3, S, D))
    pos = RNG.uniform(0, 9000, size=(S, 3))
    invf = inv_freq(5e6, D)
    fr = torch.from_numpy(pos.T[:, None, :, None] * invf)                 # [3, 1, S, P]
    fr_t = Qwen3VLTextRotaryEmbedding.apply_interleaved_mrope(None, fr, list(sections))
    emb = torch.cat([fr_t, fr_t], dim=-1)
    xt = torch.from_numpy(x)
    _, ref = apply_rotary_pos_emb(xt, xt, emb.cos(), emb.sin())
    ours = rotate_keys(x, pos[None, None], invf, pair_axis(D, sections, True))
    assert np.allclose(ours, ref.numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("interleaved,sections", [(False, (16, 24, 24)), (True, (22, 21, 21))])
def test_text_positions_reduce_to_textbook_rope(interleaved, sections):
    """With t = h = w = p (the text rule), M-RoPE is plain 1-D RoPE.

    Reference: transformers' Llama rotary embedding (its own inv_freq, cos/sin
    and rotate_half), computed in float32 by the library, so the tolerance is
    set by float32 angles at positions below 64.
    """
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding, apply_rotary_pos_emb
    D, S, theta = 128, 64, 1e4
    cfg = LlamaConfig(hidden_size=2 * D, num_attention_heads=2, head_dim=D, rope_theta=theta)
    rot = LlamaRotaryEmbedding(config=cfg)
    x = RNG.standard_normal((1, 1, S, D))
    p = np.arange(S, dtype=np.float64)
    cos, sin = rot(torch.zeros(1, S, D), torch.arange(S)[None])
    _, ref = apply_rotary_pos_emb(torch.from_numpy(x).float(), torch.from_numpy(x).float(), cos, sin)
    ours = rotate_keys(x, np.stack([p, p, p], 1)[None, None], inv_freq(theta, D),
                       pair_axis(D, sections, interleaved))
    assert np.allclose(ours, ref.double().numpy(), rtol=0, atol=2e-5)


def test_pair_norms_preserved():
    D = 128
    invf, axis = inv_freq(1e6, D), pair_axis(D, (16, 24, 24), False)
    x = RNG.standard_normal((50, D))
    pos = RNG.uniform(-1e4, 1e4, size=(50, 3))
    y = rotate_keys(x, pos, invf, axis)
    P = D // 2
    nx = np.hypot(x[:, :P], x[:, P:])
    ny = np.hypot(y[:, :P], y[:, P:])
    assert np.allclose(ny, nx, rtol=1e-14, atol=0)


@pytest.mark.parametrize("interleaved,sections", [(False, (16, 24, 24)), (True, (22, 21, 21))])
def test_scores_depend_only_on_coordinate_differences(interleaved, sections):
    """Eq. (5): <R(p)q, R(p')k> is unchanged when both positions move by one offset per axis."""
    D = 128
    invf, axis = inv_freq(1e6, D), pair_axis(D, sections, interleaved)
    q = RNG.standard_normal(D)
    k = RNG.standard_normal((20, D))
    pq = RNG.uniform(0, 3000, 3)
    pk = RNG.uniform(0, 3000, (20, 3))
    shift = RNG.uniform(-500, 500, 3)
    s0 = rotate_keys(k, pk, invf, axis) @ rotate_keys(q, pq, invf, axis)
    s1 = rotate_keys(k, pk + shift, invf, axis) @ rotate_keys(q, pq + shift, invf, axis)
    assert np.allclose(s0, s1, rtol=1e-9, atol=1e-9)
    # and equal to <q, R(p' - p) k>
    s2 = rotate_keys(k, pk - pq, invf, axis) @ q
    assert np.allclose(s0, s2, rtol=1e-9, atol=1e-9)


def test_composition_and_rebinding_a_stale_key():
    D = 128
    invf, axis = inv_freq(1e6, D), pair_axis(D, (16, 24, 24), False)
    k_raw = RNG.standard_normal((10, D))
    p_orig = RNG.integers(0, 48, (10, 3)).astype(np.float64)
    p_new = RNG.uniform(1000, 1003, (10, 3))
    stale = rotate_keys(k_raw, p_orig, invf, axis)                   # Eq. (4)
    via_stale = rotate_keys(stale, p_new - p_orig, invf, axis)
    direct = rotate_keys(k_raw, p_new, invf, axis)                    # Eq. (12)
    assert np.allclose(via_stale, direct, rtol=0, atol=1e-11)
    # identity rotation at position 0
    assert np.array_equal(rotate_keys(k_raw, np.zeros((10, 3)), invf, axis), k_raw)


@pytest.mark.parametrize("interleaved,sections", [(False, (16, 24, 24)), (True, (24, 20, 20))])
def test_each_axis_moves_only_its_pairs(interleaved, sections):
    D = 128
    P = D // 2
    invf, axis = inv_freq(1e6, D), pair_axis(D, sections, interleaved)
    x = RNG.standard_normal(D)
    base = np.array([3.0, 7.0, 11.0])
    y0 = rotate_keys(x, base, invf, axis)
    for a in range(3):
        p = base.copy()
        p[a] += 1.25
        y = rotate_keys(x, p, invf, axis)
        changed = ~np.isclose(y, y0, rtol=0, atol=1e-15)
        mask = np.concatenate([axis == a, axis == a])
        assert changed[mask].all() and not changed[~mask].any()
    assert P == len(axis)


@pytest.mark.parametrize("interleaved,sections,theta", [(True, (24, 20, 20), 5e6), (False, (16, 24, 24), 1e6)])
def test_float64_error_within_derived_bound_of_50_digit_reference(interleaved, sections, theta):
    """The oracle against the rotation evaluated to 50 significant digits.

    The reference takes theta^(-2i/d), the product with the position and the
    cosine and sine in mpmath, from the same float64 inputs.  The oracle's
    error budget per output, with u = 2^-53:
      * inv_freq: 2i/d is exact for a power-of-two d; the power adds at most
        ~1 ulp, so the angle carries |angle| * 2u;
      * the product pos * inv_freq rounds once: |angle| * u more;
      * cos and sin: at most ~1 ulp each, so u in absolute terms;
      * a*c - b*s: two products and a difference, 3u * (|a| + |b|).
    Total: (|lo| + |hi|) * ((3 |angle| + 1) u + 3u).  The test allows twice that.
    A wrong angle, axis, orientation or frequency is off by many orders more.
    """
    import mpmath
    mpmath.mp.dps = 50
    D = 128
    P = D // 2
    invf, axis = inv_freq(theta, D), pair_axis(D, sections, interleaved)
    x = RNG.standard_normal((6, D))
    pos = np.concatenate([RNG.uniform(0, 12000, (4, 3)), [[1e-3, 0.5, 3.0]], [[9999.75, 9998.5, 9997.25]]])
    y = rotate_keys(x, pos, invf, axis)
    u = 2.0 ** -53
    th = mpmath.mpf(theta)
    for n in range(x.shape[0]):
        for i in range(P):
            ang = mpmath.mpf(pos[n, axis[i]]) * th ** (-mpmath.mpf(2 * i) / D)
            c, s = mpmath.cos(ang), mpmath.sin(ang)
            lo, hi = mpmath.mpf(x[n, i]), mpmath.mpf(x[n, i + P])
            ref_lo, ref_hi = lo * c - hi * s, hi * c + lo * s
            bound = 2 * (abs(x[n, i]) + abs(x[n, i + P])) * ((3 * float(abs(ang)) + 1) * u + 3 * u)
            assert abs(float(y[n, i] - ref_lo)) <= bound, (n, i)
            assert abs(float(y[n, i + P] - ref_hi)) <= bound, (n, i)


@pytest.mark.parametrize("interleaved,sections", [(False, (2, 3, 3)), (True, (3, 3, 2))])
def test_equals_exponential_of_the_rotation_generator(interleaved, sections):
    """Eq. (4)'s rotation as a matrix exponential, built without a cosine or sine.

    R(p) = expm(G), where G is skew-symmetric with G[i+d/2, i] = angle_i and
    G[i, i+d/2] = -angle_i: a rotation by angle_i in the plane (e_i, e_{i+d/2})
    that turns e_i towards e_{i+d/2}.  scipy's expm evaluates it by scaling and
    squaring a Pade approximant.  The full d x d product also checks that no
    other component mixes in.
    """
    from scipy.linalg import expm
    D = 16
    P = D // 2
    invf, axis = inv_freq(100.0, D), pair_axis(D, sections, interleaved)
    for _ in range(5):
        pos = RNG.uniform(-6, 6, 3)
        G = np.zeros((D, D))
        for i in range(P):
            a = pos[axis[i]] * invf[i]
            G[i + P, i], G[i, i + P] = a, -a
        R = expm(G)
        assert np.allclose(R.T @ R, np.eye(D), atol=1e-12)
        x = RNG.standard_normal((4, D))
        assert np.allclose(rotate_keys(x, np.broadcast_to(pos, (4, 3)), invf, axis), x @ R.T,
                           rtol=0, atol=1e-12)


@pytest.mark.parametrize("interleaved", [False, True])
def test_one_dimensional_sections_are_textbook_rope_at_t(interleaved):
    """Sections [d/2, 0, 0] put every pair on the t axis: plain 1-D RoPE at position
    t, whatever h and w hold (the rotary form of models without M-RoPE, such as the
    InternVL3.5 family the paper also evaluates).  Reference: transformers' Llama
    rotary embedding in float32, so the tolerance is that of float32 angles."""
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding, apply_rotary_pos_emb
    D, S, theta = 128, 64, 1e6
    cfg = LlamaConfig(hidden_size=2 * D, num_attention_heads=2, head_dim=D, rope_theta=theta)
    rot = LlamaRotaryEmbedding(config=cfg)
    x = RNG.standard_normal((1, 1, S, D))
    t = np.arange(S, dtype=np.float64)
    cos, sin = rot(torch.zeros(1, S, D), torch.arange(S)[None])
    _, ref = apply_rotary_pos_emb(torch.from_numpy(x).float(), torch.from_numpy(x).float(), cos, sin)
    hw = RNG.uniform(-5000, 5000, (S, 2))
    pos = np.concatenate([t[:, None], hw], axis=1)
    axis = pair_axis(D, (D // 2, 0, 0), interleaved)
    assert (axis == 0).all()
    ours = rotate_keys(x, pos[None, None], inv_freq(theta, D), axis)
    assert np.allclose(ours, ref.double().numpy(), rtol=0, atol=2e-5)
