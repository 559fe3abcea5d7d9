"""Pins for the oracle's prefill capture (Eq. (4), Eq. (6)-(7)).

The rotated prefill keys are checked against transformers' Qwen2-VL multimodal
rotary routine (a library reference, run in float64 and rounded once); placement
is brute-forced; and the method's consistency property is checked end to end:
rebinding a visual token at its original coordinates (IDENTITY reassignment,
i.e. direct reuse, Eq. (4)) reproduces the key the prefill wrote.
"""
import numpy as np
import torch

import oracle
import workloads

RNG = np.random.default_rng(21)


def _setup(paged=False, NL=3, H=2, D=64, sections=(8, 12, 12)):
    pos, vis_index, n_tokens, n_visual = workloads.prompt()
    B, S = vis_index.shape
    M = int(n_visual.max()) + 2
    rope = {"head_dim": D, "sections": sections, "interleaved": False, "theta": 1e4}
    mem = {"k": np.zeros((B, M, NL, H, D), np.float32), "v": np.zeros((B, M, NL, H, D), np.float32),
           "coords": np.zeros((B, M, 3), np.int32), "n_visual": n_visual, "dtype": "f32"}
    if paged:
        bs = 4
        need = [(int(n) + 16 + bs - 1) // bs for n in n_tokens]
        table = np.full((B, max(need)), -1, np.int32)
        perm = RNG.permutation(sum(need)).astype(np.int32)
        o = 0
        for b, n in enumerate(need):
            table[b, :n] = perm[o:o + n]
            o += n
        cache = {"paged": True, "block_size": bs, "block_table": table, "max_blocks": max(need),
                 "n_blocks": sum(need)}
        shape = (NL, sum(need), bs, H, D)
    else:
        cache = {"paged": False, "s_max": S + 16}
        shape = (B, NL, H, S + 16, D)
    cache["k"] = RNG.standard_normal(shape).astype(np.float32)
    cache["v"] = RNG.standard_normal(shape).astype(np.float32)
    raw = [(RNG.standard_normal((B, S, H, D)).astype(np.float32),
            RNG.standard_normal((B, S, H, D)).astype(np.float32)) for _ in range(NL)]
    return rope, mem, cache, raw, pos, vis_index, n_tokens


def _capture_all(rope, mem, cache, raw, pos, vis_index, n_tokens):
    start = np.zeros(len(n_tokens), np.int64)
    for layer, (rk, rv) in enumerate(raw):
        out = oracle.prefill_capture(rope, mem, layer, rk, rv, pos, n_tokens, vis_index, True, cache,
                                     start)
        assert out["err"] == 0
        mem = dict(mem, k=out["mem_k"], v=out["mem_v"], coords=out["coords"], v_slot=out["v_slot"])
        cache = dict(cache, k=out["k"], v=out["v"])
    return mem, cache


def test_prefill_keys_match_qwen2vl_rotary():
    from transformers.models.qwen2_vl.modeling_qwen2_vl import apply_multimodal_rotary_pos_emb
    rope, mem, cache, raw, pos, vis_index, n_tokens = _setup()
    mem2, cache2 = _capture_all(rope, mem, cache, raw, pos, vis_index, n_tokens)
    invf = 1e4 ** (-(2.0 * np.arange(32)) / 64)          # textbook frequencies, written out
    for b in range(2):
        n = int(n_tokens[b])
        fr = torch.from_numpy(pos[b, :n].T.astype(np.float64)[:, None, :, None] * invf)   # [3,1,n,P]
        emb = torch.cat([fr, fr], dim=-1)
        for layer in range(3):
            x = torch.from_numpy(raw[layer][0][b, :n].astype(np.float64)).transpose(0, 1)[None]
            _, ref = apply_multimodal_rotary_pos_emb(x, x, emb.cos(), emb.sin(), [8, 12, 12])
            ref = ref[0].transpose(0, 1).numpy().astype(np.float32)          # [n, H, D]
            got = cache2["k"][b, layer, :, :n].transpose(1, 0, 2)
            assert np.allclose(got, ref, rtol=0, atol=2e-6)


def test_prefill_placement_brute_force():
    rope, mem, cache, raw, pos, vis_index, n_tokens = _setup(paged=True)
    mem2, cache2 = _capture_all(rope, mem, cache, raw, pos, vis_index, n_tokens)
    bs, table = cache["block_size"], cache["block_table"]
    for layer in range(3):
        for b in range(2):
            for s in range(int(n_tokens[b])):
                blk, off = table[b][s // bs], s % bs
                assert np.array_equal(cache2["v"][layer, blk, off], raw[layer][1][b, s])
                m = vis_index[b, s]
                if m >= 0:
                    assert np.array_equal(mem2["k"][b, m, layer], raw[layer][0][b, s])
                    assert np.array_equal(mem2["v"][b, m, layer], raw[layer][1][b, s])
                    assert mem2["coords"][b, m].tolist() == pos[b, s].tolist()
            # slots beyond the prompt are untouched
            for s in range(int(n_tokens[b]), table.shape[1] * bs):
                if table[b][s // bs] >= 0:
                    blk, off = table[b][s // bs], s % bs
                    assert np.array_equal(cache2["k"][layer, blk, off], cache["k"][layer, blk, off])


def test_identity_rebinding_reproduces_prefill_keys():
    """Eq. (4) vs Eq. (12): rebinding at the original coordinates gives the stored key."""
    for paged in (False, True):
        rope, mem, cache, raw, pos, vis_index, n_tokens = _setup(paged=paged)
        mem2, cache2 = _capture_all(rope, mem, cache, raw, pos, vis_index, n_tokens)
        sel = [np.array([0, 3, 7, 11]), np.array([2, 5, 29])]
        sel_off = np.array([0, 4, 7])
        sel_idx = np.concatenate(sel)
        p_txt = n_tokens - 1
        new_pos, _, err = oracle.reassign_batch(mem2["coords"], mem2["n_visual"], sel_off, sel_idx,
                                                p_txt, "identity")
        assert err == 0
        out = oracle.rebind_inject(rope, mem2, sel_off, sel_idx, new_pos, cache2, n_tokens)
        for b in range(2):
            for j, m in enumerate(sel[b]):
                s_orig = int(np.nonzero(vis_index[b] == m)[0][0])
                s_new = int(n_tokens[b]) + j
                if paged:
                    bs, t = cache["block_size"], cache["block_table"]
                    a = out["k"][:, t[b][s_orig // bs], s_orig % bs]
                    c = out["k"][:, t[b][s_new // bs], s_new % bs]
                else:
                    a, c = out["k"][b, :, :, s_orig], out["k"][b, :, :, s_new]
                assert np.array_equal(a, c)


def test_key_only_memory_prefill_and_identity_round_trip():
    """A key-only memory gets the same keys and, per visual token, the prompt slot
    that holds its value rows; an IDENTITY revisit through it then reproduces the
    prefill's key and value rows at the new slots (values read from the cache)."""
    for paged in (False, True):
        rope, mem, cache, raw, pos, vis_index, n_tokens = _setup(paged=paged)
        full, cache_f = _capture_all(rope, mem, cache, raw, pos, vis_index, n_tokens)
        konly = dict(mem, v=None, v_slot=np.full(mem["coords"].shape[:2], -5, np.int32))
        konly, cache_k = _capture_all(rope, konly, cache, raw, pos, vis_index, n_tokens)
        assert konly["v"] is None
        assert np.array_equal(konly["k"], full["k"]) and np.array_equal(cache_k["k"], cache_f["k"])
        for b in range(2):
            for s_ in range(int(n_tokens[b])):
                m = vis_index[b, s_]
                if m >= 0:
                    assert konly["v_slot"][b, m] == s_
        assert (konly["v_slot"][0, int(full["n_visual"][0]):] == -5).all()
        sel = [np.array([0, 3, 7, 11]), np.array([2, 5, 29])]
        sel_off = np.array([0, 4, 7])
        sel_idx = np.concatenate(sel)
        new_pos, _, err = oracle.reassign_batch(konly["coords"], konly["n_visual"], sel_off, sel_idx,
                                                n_tokens - 1, "identity")
        out = oracle.rebind_inject(rope, konly, sel_off, sel_idx, new_pos, cache_k, n_tokens)
        assert err == 0 and out["err"] == 0
        for b in range(2):
            for j, m in enumerate(sel[b]):
                s_orig = int(np.nonzero(vis_index[b] == m)[0][0])
                s_new = int(n_tokens[b]) + j
                for which in ("k", "v"):
                    if paged:
                        bs, t = cache["block_size"], cache["block_table"]
                        a = out[which][:, t[b][s_orig // bs], s_orig % bs]
                        c = out[which][:, t[b][s_new // bs], s_new % bs]
                    else:
                        a, c = out[which][b, :, :, s_orig], out[which][b, :, :, s_new]
                    assert np.array_equal(a, c)


def test_prefill_errors():
    rope, mem, cache, raw, pos, vis_index, n_tokens = _setup()
    bad = vis_index.copy()
    bad[0, 6] = 99
    out = oracle.prefill_capture(rope, mem, 0, raw[0][0], raw[0][1], pos, n_tokens, bad, True, cache,
                                 np.zeros(2, np.int64))
    assert out["err"] == oracle.ERR_INDEX
    out = oracle.prefill_capture(rope, mem, 0, raw[0][0], raw[0][1], pos, n_tokens, vis_index, True,
                                 cache, np.array([0, 20]))
    assert out["err"] == oracle.ERR_CAPACITY          # 20 + 39 > s_max = 55
