"""GPU parity of decode attention over the active cache (Eq. (14)) against the
float64 oracle, and the whole path end to end: prefill capture -> PCR revisit ->
decode attention.

Tolerance (derived from the arithmetic): scores and the softmax are accumulated in
float32 over at most a chunk of keys per lane group before the float32 merges, so
|out - ref| <= 5e-5 * max |V| over the attended rows (+ 1e-6)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, to_dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _check(out, ref, cache_o, lens, n_kv, G, dtype, layer):
    out = out.cpu().numpy()
    for b in range(len(lens)):
        for kvh in range(n_kv):
            n = int(lens[b])
            vmax = np.abs(oracle.storage_to_f64(oracle.cache_rows(cache_o, layer, b, kvh, n, "v"),
                                                dtype)).max() if n else 0.0
            for g in range(G):
                qh = kvh * G + g
                d = np.abs(out[b, qh] - ref[b, qh]).max()
                assert d <= 5e-5 * vmax + 1e-6, (b, qh, d, vmax)


CASES = [("bf16", 128, 4, False), ("bf16", 128, 7, True), ("bf16", 128, 8, False),
         ("bf16", 64, 2, True), ("f32", 64, 1, False), ("f32", 128, 4, True), ("bf16", 128, 1, True)]


@pytest.mark.parametrize("dtype,D,G,paged", CASES)
def test_decode_attention_parity(dtype, D, G, paged):
    B, NL, H, layer = 4, 2, 2, 1
    lens = np.array([0, 1, 700, 333], np.int32)
    cap = 800
    g = torch.Generator().manual_seed(D + G)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rnd = lambda *s: torch.randn(s, generator=g).to(tdt)
    rng = np.random.default_rng(G)
    if paged:
        bs = 16
        need = (cap + bs - 1) // bs
        table = rng.permutation(B * need).astype(np.int32).reshape(B, need)
        k, v = rnd(NL, B * need, bs, H, D), rnd(NL, B * need, bs, H, D)
        cache_o = {"paged": True, "block_size": bs, "block_table": table, "max_blocks": need,
                   "n_blocks": B * need}
    else:
        k, v = rnd(B, NL, H, cap, D), rnd(B, NL, H, cap, D)
        cache_o = {"paged": False, "s_max": cap}
    cache_o["k"], cache_o["v"] = workloads.as_numpy_storage(k), workloads.as_numpy_storage(v)
    q = rnd(B, H * G, D)
    q_pos = rng.integers(0, 20000, B).astype(np.int32)
    _say(f"decode attention {dtype} D={D} G={G} paged={paged}")
    cache = prcr.Cache(k.to(DEV), v.to(DEV), to_dev(cache_o["block_table"]) if paged else None)
    rope = prcr.Rope(D, (8, 12, 12) if D == 64 else (16, 24, 24), False, 1e6)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q.to(DEV), to_dev(q_pos), to_dev(lens), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = oracle.decode_attention(rope.__dict__ | {"sections": rope.sections}, cache_o, layer,
                                  workloads.as_numpy_storage(q), q_pos, lens, D ** -0.5, dtype)
    _check(out, ref, cache_o, lens, H, G, dtype, layer)
    assert not out[0].any()


# Paged pools whose KV-head count is a multiple of 4 take the head-per-wave
# mapping (a workgroup's waves on the heads of the same slots): every head checked.
HEAD_WAVE_CASES = [("bf16", 128, 4, 4, 16), ("bf16", 128, 2, 8, 16), ("f32", 64, 1, 4, 5),
                   ("bf16", 64, 8, 4, 1), ("bf16", 128, 3, 12, 16), ("f32", 128, 4, 8, 7)]


@pytest.mark.parametrize("dtype,D,G,H,bs", HEAD_WAVE_CASES)
def test_decode_attention_parity_paged_head_waves(dtype, D, G, H, bs):
    B, NL, layer = 4, 2, 1
    lens = np.array([0, 1, 700, 333], np.int32)
    cap = 800
    g = torch.Generator().manual_seed(100 + D + G + H)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rnd = lambda *s: torch.randn(s, generator=g).to(tdt)
    rng = np.random.default_rng(H * 10 + G)
    need = (cap + bs - 1) // bs
    table = rng.permutation(B * need + 3)[:B * need].astype(np.int32).reshape(B, need)
    k, v = rnd(NL, B * need + 3, bs, H, D), rnd(NL, B * need + 3, bs, H, D)
    cache_o = {"paged": True, "block_size": bs, "block_table": table, "max_blocks": need,
               "n_blocks": B * need + 3}
    cache_o["k"], cache_o["v"] = workloads.as_numpy_storage(k), workloads.as_numpy_storage(v)
    q = rnd(B, H * G, D)
    q_pos = rng.integers(0, 20000, B).astype(np.int32)
    _say(f"decode attention paged head-per-wave {dtype} D={D} G={G} H={H} block {bs}")
    cache = prcr.Cache(k.to(DEV), v.to(DEV), to_dev(table))
    rope = prcr.Rope(D, (8, 12, 12) if D == 64 else (16, 24, 24), False, 1e6)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q.to(DEV), to_dev(q_pos), to_dev(lens), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = oracle.decode_attention(rope.__dict__ | {"sections": rope.sections}, cache_o, layer,
                                  workloads.as_numpy_storage(q), q_pos, lens, D ** -0.5, dtype)
    _check(out, ref, cache_o, lens, H, G, dtype, layer)
    assert not out[0].any()


def test_decode_after_prefill_and_revisit():
    """The path end to end on the GPU against the oracle: every layer's prefill
    capture, a PCR revisit of selected visual tokens, then decode attention of the
    next text token (Eq. (4), (6)-(14))."""
    pos, vis, n_tok, n_vis = workloads.prompt()
    B, S = vis.shape
    NL, H, D, G = 3, 2, 128, 4
    M = int(n_vis.max())
    rope_d = {"head_dim": D, "sections": (24, 20, 20), "interleaved": True, "theta": 5e6}
    g = torch.Generator().manual_seed(77)
    raw = [(torch.randn((B, S, H, D), generator=g).to(torch.bfloat16),
            torch.randn((B, S, H, D), generator=g).to(torch.bfloat16)) for _ in range(NL)]
    s_max = S + 40
    ck = torch.zeros((B, NL, H, s_max, D), dtype=torch.bfloat16)
    cv = torch.zeros_like(ck)
    mem = prcr.Memory(torch.zeros((B, M, NL, H, D), dtype=torch.bfloat16, device=DEV),
                      torch.zeros((B, M, NL, H, D), dtype=torch.bfloat16, device=DEV),
                      torch.zeros((B, M, 3), dtype=torch.int32, device=DEV), to_dev(n_vis))
    cache = prcr.Cache(ck.to(DEV), cv.to(DEV))
    rope = prcr.Rope(D, rope_d["sections"], True, rope_d["theta"])
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    zero = torch.zeros(B, dtype=torch.int32, device=DEV)
    for layer, (rk, rv) in enumerate(raw):
        prcr.prefill_capture(rope, mem, layer, rk.to(DEV), rv.to(DEV), to_dev(pos), to_dev(n_tok),
                             to_dev(vis), cache, zero, err=err)
    sel = [np.array([1, 4, 9, 10, 22]), np.array([0, 7, 29])]
    sel_off = np.array([0, 5, 8], np.int32)
    sel_idx = np.concatenate(sel).astype(np.int32)
    p_txt = (pos[np.arange(B), n_tok - 1, 0]).astype(np.int32)        # latest text position
    _, next_pos, new_len, _ = prcr.revisit(rope, mem, to_dev(sel_off), to_dev(sel_idx), to_dev(p_txt),
                                           cache, to_dev(n_tok), "pcr", 2, err=err)
    q = torch.randn((B, H * G, D), generator=g).to(torch.bfloat16)
    outs = [prcr.decode_attention(rope, cache, layer, q.to(DEV), next_pos, new_len, err=err)
            for layer in range(NL)]
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    _say("prefill -> revisit -> decode on the GPU done; running the oracle pipeline")

    npy = workloads.as_numpy_storage
    mem_o = {"k": np.zeros((B, M, NL, H, D), np.uint16), "v": np.zeros((B, M, NL, H, D), np.uint16),
             "coords": np.zeros((B, M, 3), np.int32), "n_visual": n_vis, "dtype": "bf16"}
    cache_o = {"paged": False, "s_max": s_max, "k": npy(ck), "v": npy(cv)}
    for layer, (rk, rv) in enumerate(raw):
        o = oracle.prefill_capture(rope_d, mem_o, layer, npy(rk), npy(rv), pos, n_tok, vis, True,
                                   cache_o, np.zeros(B, np.int64))
        mem_o = dict(mem_o, k=o["mem_k"], v=o["mem_v"], coords=o["coords"])
        cache_o = dict(cache_o, k=o["k"], v=o["v"])
    new_pos_o, next_o, e1 = oracle.reassign_batch(mem_o["coords"], n_vis, sel_off, sel_idx, p_txt)
    res = oracle.rebind_inject(rope_d, mem_o, sel_off, sel_idx, new_pos_o, cache_o, n_tok)
    assert e1 == 0 and res["err"] == 0
    assert np.array_equal(next_pos.cpu().numpy(), next_o)
    assert np.array_equal(new_len.cpu().numpy(), res["new_cache_len"])
    cache_o = dict(cache_o, k=res["k"], v=res["v"])
    for layer in range(NL):
        ref = oracle.decode_attention(rope_d, cache_o, layer, npy(q), next_o, res["new_cache_len"],
                                      D ** -0.5, "bf16")
        _check(outs[layer], ref, cache_o, res["new_cache_len"], H, G, "bf16", layer)


@pytest.mark.parametrize("paged", [False, True])
def test_decode_graph_replays_match_eager(paged):
    """prcr_decode_attention captured in a HIP graph: each replay, after eager work
    that clobbers the output and the workspace, reproduces the eager result bit for
    bit (the kernels clear nothing with memsets, so replays are self-contained)."""
    B, NL, H, D, G, layer = 4, 2, 2, 128, 4, 1
    lens = np.array([0, 1, 700, 333], np.int32)
    cap = 800
    g = torch.Generator().manual_seed(91)
    rnd = lambda *s: torch.randn(s, generator=g).to(torch.bfloat16)
    if paged:
        bs, need = 16, 50
        table = np.random.default_rng(92).permutation(B * need).astype(np.int32).reshape(B, need)
        cache = prcr.Cache(rnd(NL, B * need, bs, H, D).to(DEV), rnd(NL, B * need, bs, H, D).to(DEV),
                           to_dev(table))
    else:
        cache = prcr.Cache(rnd(B, NL, H, cap, D).to(DEV), rnd(B, NL, H, cap, D).to(DEV))
    rope = prcr.Rope(D, (16, 24, 24), False, 1e6)
    q = rnd(B, H * G, D).to(DEV)
    q_pos, cl = to_dev(np.array([5, 900, 3000, 17], np.int32)), to_dev(lens)
    out = torch.empty((B, H * G, D), dtype=torch.float32, device=DEV)
    ws = torch.empty(prcr.decode_workspace_bytes(cache, B, H * G) // 4 + 1, dtype=torch.float32,
                     device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    s = torch.cuda.Stream(device=DEV)
    _say(f"graph capture of decode attention, paged={paged}, 3 replays")

    def call():
        prcr.decode_attention(rope, cache, layer, q, q_pos, cl, None, out, ws, err, s)

    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        call()
    torch.cuda.synchronize()
    eager = out.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        call()
    torch.cuda.synchronize()
    for r in range(3):
        out.fill_(float("nan"))                     # eager work between replays
        ws.fill_(float("nan"))
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {r}"
    assert int(err.item()) == 0


def test_decode_many_sequences():
    """3000 sequences (the batch is a grid dimension of the partial kernel) with
    cache lengths 0-40, paged with block 5, against the oracle."""
    B, NL, H, D, G, layer, bs = 3000, 2, 1, 64, 2, 1, 5
    rng = np.random.default_rng(77)
    lens = rng.integers(0, 41, B).astype(np.int32)
    need = 9
    table = rng.permutation(B * need).astype(np.int32).reshape(B, need)
    g = torch.Generator().manual_seed(78)
    k = torch.randn((NL, B * need, bs, H, D), generator=g)
    v = torch.randn((NL, B * need, bs, H, D), generator=g)
    q = torch.randn((B, H * G, D), generator=g)
    q_pos = rng.integers(0, 5000, B).astype(np.int32)
    _say(f"decode attention over {B} sequences, paged block {bs}")
    cache = prcr.Cache(k.to(DEV), v.to(DEV), to_dev(table))
    rope = prcr.Rope(D, (8, 12, 12), False, 1e6)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q.to(DEV), to_dev(q_pos), to_dev(lens), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    cache_o = {"paged": True, "block_size": bs, "block_table": table, "max_blocks": need,
               "n_blocks": B * need, "k": k.numpy(), "v": v.numpy()}
    ref = oracle.decode_attention(rope.__dict__ | {"sections": rope.sections}, cache_o, layer,
                                  q.numpy(), q_pos, lens, D ** -0.5, "f32")
    _check(out, ref, cache_o, lens, H, G, "f32", layer)


def _reference_over_kept(rope_d, cache_o, layer, q, q_pos, lens_eff, skip, dtype):
    """The oracle's attention over the keys the library keeps: slots below
    lens_eff[b], minus the logical blocks skip[b].  Attention does not depend on
    the order of its keys, so the kept rows of each sequence are packed into a
    contiguous cache and handed to the oracle unchanged."""
    kk, vv = cache_o["k"], cache_o["v"]
    paged = cache_o["paged"]
    NL, H, D = (kk.shape[0], kk.shape[3], kk.shape[4]) if paged else (kk.shape[1], kk.shape[2], kk.shape[4])
    bs = cache_o.get("block_size", 1)
    keep = [[s for s in range(int(n)) if not (paged and s // bs in skip.get(b, ()))]
            for b, n in enumerate(lens_eff)]
    cap = max(1, max(len(x) for x in keep))
    kc = np.zeros((len(keep), NL, H, cap, D), kk.dtype)
    vc = np.zeros_like(kc)
    for b, slots in enumerate(keep):
        for i, s in enumerate(slots):
            if paged:
                blk = cache_o["block_table"][b, s // bs]
                kc[b, layer, :, i], vc[b, layer, :, i] = kk[layer, blk, s % bs], vv[layer, blk, s % bs]
            else:
                kc[b, layer, :, i], vc[b, layer, :, i] = kk[b, layer, :, s], vv[b, layer, :, s]
    packed = {"paged": False, "s_max": cap, "k": kc, "v": vc}
    kept = np.array([len(x) for x in keep], np.int32)
    ref = oracle.decode_attention(rope_d, packed, layer, q, q_pos, kept, D ** -0.5, dtype)
    return ref, packed, kept


@pytest.mark.parametrize("paged", [False, True])
def test_decode_data_errors(paged):
    """Data errors of decode attention, as the header documents them: a cache_len
    below 0 or above the capacity is clamped (PRCR_DERR_CAPACITY), and a block-table
    entry outside the pool skips that block's keys (PRCR_DERR_BLOCK).  The output is
    the oracle's attention over the keys that remain.  Paged: pool block 0 holds NaN
    in every layer and no table entry names it, so a skipped or past-the-end row
    whose value leaked into a sum would show as NaN."""
    B, NL, H, D, G, layer = 4, 2, 2, 128, 4, 1
    g = torch.Generator().manual_seed(501)
    rnd = lambda *s: torch.randn(s, generator=g).to(torch.bfloat16)
    rng = np.random.default_rng(502)
    if paged:
        bs, need = 16, 40
        cap, n_blocks = bs * need, B * need + 1
        table = (1 + rng.permutation(B * need)).astype(np.int32).reshape(B, need)
        table[0, 3] = -1                    # slots 48..63 of sequence 0
        table[1, 0] = n_blocks + 7          # slots 0..15 of sequence 1
        table[3, need - 1] = n_blocks       # the last block of sequence 3
        skip = {0: {3}, 1: {0}, 3: {need - 1}}
        k, v = rnd(NL, n_blocks, bs, H, D), rnd(NL, n_blocks, bs, H, D)
        k[:, 0], v[:, 0] = float("nan"), float("nan")
        lens = np.array([500, 333, cap + 40, cap], np.int32)
        expect = prcr.DERR_BLOCK | prcr.DERR_CAPACITY
        cache_o = {"paged": True, "block_size": bs, "block_table": table, "max_blocks": need,
                   "n_blocks": n_blocks}
        cache = prcr.Cache(k.to(DEV), v.to(DEV), to_dev(table))
    else:
        cap = 600
        skip = {}
        k, v = rnd(B, NL, H, cap, D), rnd(B, NL, H, cap, D)
        lens = np.array([-3, cap + 9, 100, 0], np.int32)
        expect = prcr.DERR_CAPACITY
        cache_o = {"paged": False, "s_max": cap}
        cache = prcr.Cache(k.to(DEV), v.to(DEV))
    cache_o["k"], cache_o["v"] = workloads.as_numpy_storage(k), workloads.as_numpy_storage(v)
    q = rnd(B, H * G, D)
    q_pos = rng.integers(0, 20000, B).astype(np.int32)
    rope = prcr.Rope(D, (16, 24, 24), False, 1e6)
    _say(f"decode attention data errors, paged={paged}, lens {lens.tolist()}")
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q.to(DEV), to_dev(q_pos), to_dev(lens), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == expect
    assert torch.isfinite(out).all()
    ref, packed, kept = _reference_over_kept(rope.__dict__ | {"sections": rope.sections}, cache_o,
                                             layer, workloads.as_numpy_storage(q), q_pos,
                                             np.clip(lens, 0, cap), skip, "bf16")
    _check(out, ref, packed, kept, H, G, "bf16", layer)
