"""Pins for the oracle's gather / inject plumbing (Eq. (11)-(13)) and the memory store.

The oracle vectorises over layers and heads; these tests rebuild the expected cache
with scalar pure-Python loops on tiny shapes (brute force), check Eq. (13)'s
concatenation through the block table for the paged layout, and exercise the
error paths.
"""
import math
import os

import numpy as np
import pytest

from oracle import (ERR_BLOCK, ERR_CAPACITY, ERR_INDEX, bf16_bits_to_f64, f64_to_bf16_bits,
                    rebind_inject, store_raw)

RNG = np.random.default_rng(11)


def _axis(i, sections):
    return 0 if i < sections[0] else (1 if i < sections[0] + sections[1] else 2)


def _brute_key(x, pos, theta, sections):
    """Scalar RoPE of one row, written out element by element (math.cos/math.sin)."""
    D = len(x)
    P = D // 2
    out = [0.0] * D
    for i in range(P):
        ang = pos[_axis(i, sections)] * theta ** (-(2.0 * i) / D)
        c, s = math.cos(ang), math.sin(ang)
        out[i] = x[i] * c - x[i + P] * s
        out[i + P] = x[i + P] * c + x[i] * s
    return out


def _tiny(paged, dtype="f32"):
    B, M, NL, H, D = 3, 6, 2, 2, 8
    sections = (1, 2, 1)
    if dtype == "f32":
        mk = RNG.standard_normal((B, M, NL, H, D)).astype(np.float32)
        mv = RNG.standard_normal((B, M, NL, H, D)).astype(np.float32)
    else:
        mk = f64_to_bf16_bits(RNG.standard_normal((B, M, NL, H, D)))
        mv = f64_to_bf16_bits(RNG.standard_normal((B, M, NL, H, D)))
    mem = {"k": mk, "v": mv, "n_visual": np.array([6, 5, 6]), "dtype": dtype}
    sel_off = np.array([0, 3, 3, 7])              # sequence 1 selects nothing
    sel_idx = np.array([4, 0, 2, 5, 1, 0, 3])
    new_pos = RNG.uniform(0, 40, (7, 3))
    cache_len = np.array([5, 2, 9])
    rope = {"head_dim": D, "sections": sections, "interleaved": False, "theta": 100.0}
    if paged:
        bs, n_blocks, max_blocks = 4, 12, 4
        table = np.array([[3, 7, 0, -1], [5, -1, -1, -1], [1, 2, 9, 11]])
        cache = {"paged": True, "block_size": bs, "n_blocks": n_blocks, "max_blocks": max_blocks,
                 "block_table": table}
        shape = (NL, n_blocks, bs, H, D)
    else:
        cache = {"paged": False, "s_max": 16}
        shape = (B, NL, H, 16, D)
    if dtype == "f32":
        cache["k"] = RNG.standard_normal(shape).astype(np.float32)
        cache["v"] = RNG.standard_normal(shape).astype(np.float32)
    else:
        cache["k"] = f64_to_bf16_bits(RNG.standard_normal(shape))
        cache["v"] = f64_to_bf16_bits(RNG.standard_normal(shape))
    return rope, mem, sel_off, sel_idx, new_pos, cache, cache_len


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_inject_brute_force(paged, dtype):
    rope, mem, sel_off, sel_idx, new_pos, cache, cache_len = _tiny(paged, dtype)
    out = rebind_inject(rope, mem, sel_off, sel_idx, new_pos, cache, cache_len)
    B, M, NL, H, D = mem["k"].shape
    ek, ev = cache["k"].copy(), cache["v"].copy()
    slots = []
    for b in range(B):
        for j in range(sel_off[b + 1] - sel_off[b]):
            g = sel_off[b] + j
            s = cache_len[b] + j
            if paged:
                blk = cache["block_table"][b][s // cache["block_size"]]
                off = s % cache["block_size"]
                slots.append(blk * cache["block_size"] + off)
            else:
                slots.append(b * cache["s_max"] + s)
            for l in range(NL):
                for h in range(H):
                    row = mem["k"][b, sel_idx[g], l, h]
                    x = [float(v) for v in (row if dtype == "f32" else bf16_bits_to_f64(row))]
                    y = np.array(_brute_key(x, new_pos[g], rope["theta"], rope["sections"]))
                    y = y.astype(np.float32) if dtype == "f32" else f64_to_bf16_bits(y)
                    if paged:
                        ek[l, blk, off, h] = y
                        ev[l, blk, off, h] = mem["v"][b, sel_idx[g], l, h]
                    else:
                        ek[b, l, h, s] = y
                        ev[b, l, h, s] = mem["v"][b, sel_idx[g], l, h]
    if dtype == "f32":
        assert np.allclose(out["k"], ek, rtol=0, atol=2e-6)
    else:
        diff = np.abs(out["k"].astype(np.int64) - ek.astype(np.int64))
        assert diff.max() <= 1                     # brute force uses libm pow; <= 1 bf16 ulp
    assert np.array_equal(out["v"], ev)
    assert out["slot_mapping"].tolist() == slots
    assert out["new_cache_len"].tolist() == [5 + 3, 2, 9 + 4]
    assert out["err"] == 0


def _value_rows_brute(cache, b, slot, NL, H):
    """Value rows [NL][H] of logical slot `slot` of sequence b, by walking the
    block table by hand (paged) or indexing the sequence's rows (contiguous)."""
    rows = []
    for l in range(NL):
        for h in range(H):
            if cache["paged"]:
                blk = cache["block_table"][b][slot // cache["block_size"]]
                rows.append(cache["v"][l, blk, slot % cache["block_size"], h])
            else:
                rows.append(cache["v"][b, l, h, slot])
    return np.array(rows).reshape((NL, H) + rows[0].shape)


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_key_only_memory_takes_values_from_the_cache(paged, dtype):
    """Key-only memory: the value rows injected for token m are those of cache slot
    v_slot[b][m] (a filled slot of the same sequence); keys are as with a full memory."""
    rope, mem, sel_off, sel_idx, new_pos, cache, cache_len = _tiny(paged, dtype)
    B, M, NL, H, D = mem["k"].shape
    v_slot = np.stack([RNG.integers(0, cache_len[b], M) for b in range(B)]).astype(np.int32)
    konly = {"k": mem["k"], "v": None, "v_slot": v_slot, "n_visual": mem["n_visual"],
             "dtype": dtype}
    full = rebind_inject(rope, mem, sel_off, sel_idx, new_pos, cache, cache_len)
    out = rebind_inject(rope, konly, sel_off, sel_idx, new_pos, cache, cache_len)
    assert out["err"] == 0
    assert np.array_equal(out["k"], full["k"])
    assert out["slot_mapping"].tolist() == full["slot_mapping"].tolist()
    ev = cache["v"].copy()
    for b in range(B):
        for j in range(sel_off[b + 1] - sel_off[b]):
            m = sel_idx[sel_off[b] + j]
            want = _value_rows_brute(cache, b, int(v_slot[b, m]), NL, H)
            s = cache_len[b] + j
            for l in range(NL):
                for h in range(H):
                    if paged:
                        blk = cache["block_table"][b][s // cache["block_size"]]
                        ev[l, blk, s % cache["block_size"], h] = want[l, h]
                    else:
                        ev[b, l, h, s] = want[l, h]
    assert np.array_equal(out["v"], ev)


def test_key_only_memory_value_slot_must_be_filled():
    rope, mem, sel_off, sel_idx, new_pos, cache, cache_len = _tiny(False)
    B, M = mem["k"].shape[:2]
    v_slot = np.zeros((B, M), np.int32)
    v_slot[0, 4] = cache_len[0]          # token 4 of sequence 0 (first pick): not yet filled
    v_slot[2, 3] = -1                    # token 3 of sequence 2 (last pick)
    konly = {"k": mem["k"], "v": None, "v_slot": v_slot, "n_visual": mem["n_visual"],
             "dtype": "f32"}
    out = rebind_inject(rope, konly, sel_off, sel_idx, new_pos, cache, cache_len)
    assert out["err"] == ERR_INDEX
    assert out["slot_mapping"][0] == -1 and out["slot_mapping"][6] == -1
    assert (out["slot_mapping"][1:6] >= 0).all()
    assert np.array_equal(out["k"][0, :, :, cache_len[0]], cache["k"][0, :, :, cache_len[0]])
    assert np.array_equal(out["v"][2, :, :, cache_len[2] + 3], cache["v"][2, :, :, cache_len[2] + 3])


def test_paged_concat_through_block_table():
    """Eq. (13): the logical sequence read through the block table is Concat[old, new]."""
    rope, mem, sel_off, sel_idx, new_pos, cache, cache_len = _tiny(True)
    out = rebind_inject(rope, mem, sel_off, sel_idx, new_pos, cache, cache_len)
    bs, table = cache["block_size"], cache["block_table"]

    def logical(k, b, n):
        return np.stack([k[:, table[b][s // bs], s % bs] for s in range(n)], axis=1)

    for b in range(3):
        K = sel_off[b + 1] - sel_off[b]
        old = logical(cache["k"], b, cache_len[b])
        new = logical(out["k"], b, cache_len[b] + K)
        assert np.array_equal(new[:, :cache_len[b]], old)
        newv = logical(out["v"], b, cache_len[b] + K)
        want_v = np.stack([mem["v"][b, sel_idx[sel_off[b] + j]] for j in range(K)], axis=1) \
            if K else np.zeros_like(newv[:, :0])
        assert np.array_equal(newv[:, cache_len[b]:], want_v)


def test_contiguous_rows_outside_new_slots_untouched():
    rope, mem, sel_off, sel_idx, new_pos, cache, cache_len = _tiny(False)
    out = rebind_inject(rope, mem, sel_off, sel_idx, new_pos, cache, cache_len)
    touched = np.zeros((3, 16), bool)
    for b in range(3):
        touched[b, cache_len[b]:cache_len[b] + sel_off[b + 1] - sel_off[b]] = True
    for b in range(3):
        for s in range(16):
            same = np.array_equal(out["k"][b, :, :, s], cache["k"][b, :, :, s])
            assert same != touched[b, s]


def test_error_paths_skip_rows_and_flag():
    rope, mem, sel_off, sel_idx, new_pos, cache, cache_len = _tiny(False)
    bad = sel_idx.copy()
    bad[1] = 6                                   # sequence 0 has n_visual = 6
    out = rebind_inject(rope, mem, sel_off, bad, new_pos, cache, cache_len)
    assert out["err"] == ERR_INDEX and out["slot_mapping"][1] == -1
    out = rebind_inject(rope, mem, sel_off, sel_idx, new_pos, cache, np.array([5, 2, 13]))
    assert out["err"] == ERR_CAPACITY             # slots 13..16 of a 16-slot cache
    assert out["slot_mapping"][3:].tolist()[-1] == -1
    rope, mem, sel_off, sel_idx, new_pos, cache, cache_len = _tiny(True)
    cache["block_table"] = cache["block_table"].copy()
    cache["block_table"][2, 2] = 12              # n_blocks = 12
    out = rebind_inject(rope, mem, sel_off, sel_idx, new_pos, cache, cache_len)
    assert out["err"] == ERR_BLOCK
    cache["block_table"][2, 2] = 9
    out = rebind_inject(rope, mem, sel_off, sel_idx, new_pos, cache, np.array([5, 2, 14]))
    assert out["err"] & ERR_CAPACITY               # slot 16 needs logical block 4 of 4


def test_store_raw_brute_force():
    B, S, M, NL, H, D = 2, 9, 4, 3, 2, 8
    raw_k = RNG.standard_normal((B, S, H, D)).astype(np.float32)
    raw_v = RNG.standard_normal((B, S, H, D)).astype(np.float32)
    vis = np.array([[2, 3, 4, 5], [8, 0, 7, -1]])
    nvis = np.array([4, 3])
    mk = np.zeros((B, M, NL, H, D), np.float32)
    mv = np.zeros_like(mk)
    k2, v2, err = store_raw(mk, mv, 1, raw_k, raw_v, vis, nvis)
    assert err == 0
    for b in range(B):
        for m in range(M):
            for l in range(NL):
                if l == 1 and m < nvis[b]:
                    assert np.array_equal(k2[b, m, l], raw_k[b, vis[b, m]])
                    assert np.array_equal(v2[b, m, l], raw_v[b, vis[b, m]])
                else:
                    assert not k2[b, m, l].any() and not v2[b, m, l].any()
    _, _, err = store_raw(mk, mv, 0, raw_k, raw_v, np.array([[2, 3, 4, 9], [8, 0, 7, -1]]), nvis)
    assert err == ERR_INDEX


def test_table3_flop_accounting():
    """Table 3's PRCR FLOPs equal 3 x hidden x layers x K (three flops per rebound element)."""
    path = os.path.join(os.path.dirname(__file__), "golden", "table3_flops.txt")
    rows = [l.split() for l in open(path) if l.strip() and not l.startswith("#")]
    assert len(rows) == 4
    for _, K, printed, hidden, layers in rows:
        val = 3 * int(hidden) * int(layers) * int(K)
        assert f"{val / 1e6:.2f}M" == printed


def test_table3_extra_memory_is_768_visual_tokens_of_raw_k_and_v():
    """Table 3's extra memory (108 MB, 192 MB) is, for both models, exactly the raw K and
    V memory of 768 visual tokens in bf16 at their cache shapes (Eq. (7), reading R14).
    The small-K workloads at Table 3's operating points take 768 visual tokens for that
    reason: their memory must come out at the printed sizes."""
    import workloads
    path = os.path.join(os.path.dirname(__file__), "golden", "table3_memory.txt")
    rows = [l.split() for l in open(path) if l.strip() and not l.startswith("#")]
    assert len(rows) == 2
    for model, printed in rows:
        w = workloads.paper_k(model.lower(), 32)
        nbytes = int(np.prod(workloads.mem_shape(w))) * 2 * 2      # K and V, bf16
        assert nbytes == int(printed) * 2 ** 20, (model, nbytes)
        assert w.M_max == 768
