"""Pins for the oracle's decode attention (Eq. (14)).

Against torch's scaled_dot_product_attention in float64 (a library routine) on the
same rotated query, plus closed forms: a single key returns its value row, equal
keys return the mean of the value rows, each query head reads KV head qh // G, an
empty cache returns zeros."""
import numpy as np
import torch

import oracle

RNG = np.random.default_rng(31)
ROPE = {"head_dim": 64, "sections": (8, 12, 12), "interleaved": False, "theta": 1e6}


def _contig(B, NL, H, S, D):
    return {"paged": False, "s_max": S,
            "k": RNG.standard_normal((B, NL, H, S, D)).astype(np.float32),
            "v": RNG.standard_normal((B, NL, H, S, D)).astype(np.float32)}


def test_matches_torch_sdpa_with_gqa():
    B, NL, H, S, D, G = 3, 2, 2, 40, 64, 3
    cache = _contig(B, NL, H, S, D)
    q = RNG.standard_normal((B, H * G, D)).astype(np.float32)
    q_pos = np.array([17, 300, 5])
    lens = np.array([40, 1, 23])
    scale = 0.125
    out = oracle.decode_attention(ROPE, cache, 1, q, q_pos, lens, scale, "f32")
    invf = oracle.inv_freq(1e6, D)
    axis = oracle.pair_axis(D, (8, 12, 12), False)
    for b in range(B):
        n = lens[b]
        qr = oracle.rotate_keys(q[b].astype(np.float64), np.full(3, float(q_pos[b])), invf, axis)
        k = torch.from_numpy(cache["k"][b, 1, :, :n].astype(np.float64)).repeat_interleave(G, 0)
        v = torch.from_numpy(cache["v"][b, 1, :, :n].astype(np.float64)).repeat_interleave(G, 0)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(qr)[:, None], k, v, scale=scale)[:, 0]
        assert np.allclose(out[b], ref.numpy(), rtol=0, atol=1e-12)


def test_closed_forms():
    B, NL, H, S, D = 2, 1, 2, 8, 64
    cache = _contig(B, NL, H, S, D)
    q = RNG.standard_normal((B, 4, D)).astype(np.float32)
    # a single key returns its value row, whatever the query
    out = oracle.decode_attention(ROPE, cache, 0, q, np.array([3, 9]), np.array([1, 1]), 0.2, "f32")
    for b in range(B):
        for qh in range(4):
            assert np.allclose(out[b, qh], cache["v"][b, 0, qh // 2, 0], atol=1e-7)
    # equal keys: uniform weights, the mean of the value rows
    cache["k"][:] = cache["k"][:, :, :, :1]
    out = oracle.decode_attention(ROPE, cache, 0, q, np.array([3, 9]), np.array([5, 8]), 0.2, "f32")
    for b, n in enumerate((5, 8)):
        for qh in range(4):
            assert np.allclose(out[b, qh], cache["v"][b, 0, qh // 2, :n].mean(0), atol=1e-7)
    # empty cache
    out = oracle.decode_attention(ROPE, cache, 0, q, np.array([3, 9]), np.array([0, 2]), 0.2, "f32")
    assert not out[0].any() and out[1].any()


def test_paged_rows_follow_the_block_table():
    B, NL, H, D, bs = 2, 2, 1, 64, 4
    table = np.array([[2, 0, 5], [1, 4, 3]])
    k = RNG.standard_normal((NL, 6, bs, H, D)).astype(np.float32)
    v = RNG.standard_normal((NL, 6, bs, H, D)).astype(np.float32)
    paged = {"paged": True, "block_size": bs, "block_table": table, "max_blocks": 3, "n_blocks": 6,
             "k": k, "v": v}
    contig = {"paged": False, "s_max": 12,
              "k": np.stack([np.concatenate([k[:, t] for t in table[b]], 1) for b in range(B)]).transpose(0, 1, 3, 2, 4),
              "v": np.stack([np.concatenate([v[:, t] for t in table[b]], 1) for b in range(B)]).transpose(0, 1, 3, 2, 4)}
    q = RNG.standard_normal((B, 1, D)).astype(np.float32)
    a = oracle.decode_attention(ROPE, paged, 1, q, np.array([4, 6]), np.array([11, 7]), 0.1, "f32")
    c = oracle.decode_attention(ROPE, contig, 1, q, np.array([4, 6]), np.array([11, 7]), 0.1, "f32")
    assert np.array_equal(a, c)
