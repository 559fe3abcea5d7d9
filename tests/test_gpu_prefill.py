"""GPU parity of the fused prefill capture (prcr_prefill_capture) against the
oracle, and the end-to-end property that a revisit at the original coordinates
(IDENTITY reassignment) reproduces the keys the prefill wrote, bit for bit.

Also the key-only memory (values left in the standard cache, found through the
memory's value-slot table): prefill capture, then PCR revisits (two launches and
fused) against the oracle, and a value slot that is not yet filled."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, assert_keys_close, to_dev

pytestmark = pytest.mark.gpu

MAPS = [("f32", 64, (8, 12, 12), False), ("bf16", 128, (16, 24, 24), False),
        ("bf16", 128, (24, 20, 20), True), ("f32", 128, (22, 21, 21), True),
        ("bf16", 128, (64, 0, 0), False)]                     # 1-D rotary


def _say(msg):
    print(msg, flush=True)


class Prefill:
    def __init__(self, dtype, D, sections, inter, paged, NL=3, H=3, seed=5, key_only=False,
                 prompt=None, block_size=4):
        self.pos, self.vis_index, self.n_tokens, self.n_visual = workloads.prompt(**(prompt or {}))
        B, S = self.vis_index.shape
        M = int(self.n_visual.max()) + 2
        self.B, self.S, self.M, self.NL, self.H, self.D, self.dtype = B, S, M, NL, H, D, dtype
        self.rope = {"head_dim": D, "sections": sections, "interleaved": inter,
                     "theta": 5e6 if inter else 1e6}
        g = torch.Generator().manual_seed(seed)
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        rnd = lambda *shape: torch.randn(shape, generator=g).to(tdt)
        self.raw = [(rnd(B, S, H, D), rnd(B, S, H, D)) for _ in range(NL)]
        self.mem_k = torch.zeros((B, M, NL, H, D), dtype=tdt)
        self.mem_v = None if key_only else torch.zeros_like(self.mem_k)
        self.key_only = key_only
        self.paged = paged
        if paged:
            bs = block_size
            need = [(int(n) + 16 + bs - 1) // bs for n in self.n_tokens]
            rng = np.random.default_rng(seed)
            table = np.full((B, max(need)), -1, np.int32)
            perm = rng.permutation(sum(need)).astype(np.int32)
            o = 0
            for b, n in enumerate(need):
                table[b, :n] = perm[o:o + n]
                o += n
            self.cache_cfg = {"paged": True, "block_size": bs, "block_table": table,
                              "max_blocks": max(need), "n_blocks": sum(need)}
            shape = (NL, sum(need), bs, H, D)
        else:
            self.cache_cfg = {"paged": False, "s_max": S + 16}
            shape = (B, NL, H, S + 16, D)
        self.cache_k, self.cache_v = rnd(*shape), rnd(*shape)

    def run_gpu(self, vis_index=None, start=None):
        vis = self.vis_index if vis_index is None else vis_index
        st = np.zeros(self.B, np.int32) if start is None else np.asarray(start, np.int32)
        v_slot = (torch.full((self.B, self.M), -5, dtype=torch.int32, device=DEV)
                  if self.key_only else None)
        mem = prcr.Memory(self.mem_k.to(DEV), None if self.key_only else self.mem_v.to(DEV),
                          torch.zeros((self.B, self.M, 3), dtype=torch.int32, device=DEV),
                          to_dev(self.n_visual), v_slot)
        cache = prcr.Cache(self.cache_k.to(DEV), self.cache_v.to(DEV),
                           to_dev(self.cache_cfg["block_table"]) if self.paged else None)
        rope = prcr.Rope(self.D, self.rope["sections"], self.rope["interleaved"], self.rope["theta"])
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        for layer, (rk, rv) in enumerate(self.raw):
            prcr.prefill_capture(rope, mem, layer, rk.to(DEV), rv.to(DEV), to_dev(self.pos),
                                 to_dev(self.n_tokens), to_dev(vis), cache, to_dev(st), err=err)
        torch.cuda.synchronize()
        return mem, cache, rope, int(err.item())

    def run_oracle(self, vis_index=None, start=None):
        vis = self.vis_index if vis_index is None else vis_index
        st = np.zeros(self.B, np.int64) if start is None else np.asarray(start, np.int64)
        npy = workloads.as_numpy_storage
        mem = {"k": npy(self.mem_k), "v": None if self.key_only else npy(self.mem_v),
               "v_slot": np.full((self.B, self.M), -5, np.int32) if self.key_only else None,
               "coords": np.zeros((self.B, self.M, 3), np.int32),
               "n_visual": self.n_visual, "dtype": self.dtype}
        cache = dict(self.cache_cfg, k=npy(self.cache_k), v=npy(self.cache_v))
        err = 0
        for layer, (rk, rv) in enumerate(self.raw):
            out = oracle.prefill_capture(self.rope, mem, layer, npy(rk), npy(rv), self.pos, self.n_tokens,
                                         vis, True, cache, st)
            err |= out["err"]
            mem = dict(mem, k=out["mem_k"], v=out["mem_v"], coords=out["coords"], v_slot=out["v_slot"])
            cache = dict(cache, k=out["k"], v=out["v"])
        return mem, cache, err


def _compare(pf, mem, cache, err, ref_mem, ref_cache, ref_err):
    npy = workloads.as_numpy_storage
    assert err == ref_err
    assert np.array_equal(npy(mem.k), ref_mem["k"])
    if pf.key_only:
        assert np.array_equal(mem.v_slot.cpu().numpy(), ref_mem["v_slot"])
    else:
        assert np.array_equal(npy(mem.v), ref_mem["v"])
    assert np.array_equal(mem.coords.cpu().numpy(), ref_mem["coords"])
    assert np.array_equal(npy(cache.v), ref_cache["v"])
    gk = npy(cache.k)
    same = gk == ref_cache["k"]
    if not same.all():
        rows = ~np.all(same, axis=-1)
        assert_keys_close(gk[rows], ref_cache["k"][rows], pf.dtype)


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("dtype,D,sections,inter", MAPS)
def test_prefill_capture_parity(dtype, D, sections, inter, paged):
    pf = Prefill(dtype, D, sections, inter, paged)
    _say(f"prefill capture {dtype} D={D} {sections} inter={inter} paged={paged}")
    mem, cache, rope, err = pf.run_gpu()
    ref_mem, ref_cache, ref_err = pf.run_oracle()
    _compare(pf, mem, cache, err, ref_mem, ref_cache, ref_err)


@pytest.mark.parametrize("dtype,D,H", [("bf16", 128, 8), ("bf16", 128, 16), ("bf16", 64, 8),
                                        ("bf16", 64, 16), ("f32", 128, 8), ("f32", 64, 12),
                                        ("bf16", 128, 4), ("bf16", 128, 2), ("bf16", 64, 4),
                                        ("f32", 128, 2), ("f32", 64, 4), ("f32", 128, 1),
                                        ("bf16", 128, 3), ("bf16", 128, 1)])
@pytest.mark.parametrize("paged", [False, True])
def test_prefill_head_counts(dtype, D, H, paged):
    """Head counts on every side of the kernel's specialisation.  When n_kv_heads is a
    multiple of a wave iteration's rows (8 at bf16 d 128 and f32 d 64, 16 at bf16 d 64,
    4 at f32 d 128), an iteration is one token.  When it is half of them (bf16 d 128
    with 4, bf16 d 64 with 8, f32 d 128 with 2, f32 d 64 with 4), an iteration is two
    tokens whose angles the wave evaluates once each.  Otherwise (bf16 d 128 with 3, 2
    or 1 heads, bf16 d 64 with 4, f32 d 128 with 1, f32 d 64 with 12) each row
    evaluates its own angles."""
    sections = (16, 24, 24) if D == 128 else (8, 12, 12)
    pf = Prefill(dtype, D, sections, False, paged, NL=2, H=H, seed=11)
    _say(f"prefill capture {dtype} D={D} H={H} paged={paged}")
    mem, cache, rope, err = pf.run_gpu()
    ref_mem, ref_cache, ref_err = pf.run_oracle()
    _compare(pf, mem, cache, err, ref_mem, ref_cache, ref_err)


def test_prefill_capture_errors():
    pf = Prefill("bf16", 128, (16, 24, 24), False, False)
    vis = pf.vis_index.copy()
    vis[0, 6] = pf.M + 5                       # visual index outside the memory
    _say("prefill capture with a bad visual index and a start past capacity")
    mem, cache, rope, err = pf.run_gpu(vis, start=[0, 20])
    ref_mem, ref_cache, ref_err = pf.run_oracle(vis, start=[0, 20])
    assert ref_err == (oracle.ERR_INDEX | oracle.ERR_CAPACITY)
    _compare(pf, mem, cache, err, ref_mem, ref_cache, ref_err)


@pytest.mark.parametrize("paged", [False, True])
def test_identity_revisit_reproduces_prefill_keys(paged):
    """Prefill-capture every layer, then revisit visual tokens at their original
    coordinates: the injected keys and values equal the prefill's rows bit for bit."""
    pf = Prefill("bf16", 128, (16, 24, 24), False, paged, NL=4, H=4)
    _say(f"prefill -> IDENTITY revisit round trip, paged={paged}")
    mem, cache, rope, err = pf.run_gpu()
    assert err == 0
    sel = [np.array([0, 3, 7, 11, 23]), np.array([2, 5, 29])]
    sel_off = np.array([0, 5, 8], np.int32)
    sel_idx = np.concatenate(sel).astype(np.int32)
    p_txt = (pf.n_tokens - 1).astype(np.int32)
    err_t = torch.zeros(1, dtype=torch.int32, device=DEV)
    _, _, _, slots = prcr.revisit(rope, mem, to_dev(sel_off), to_dev(sel_idx), to_dev(p_txt), cache,
                                  to_dev(pf.n_tokens), "identity", 2, err=err_t)
    torch.cuda.synchronize()
    assert int(err_t.item()) == 0
    slots = slots.cpu().numpy()
    for b in range(2):
        for j, m in enumerate(sel[b]):
            s_orig = int(np.nonzero(pf.vis_index[b] == m)[0][0])
            new = int(slots[sel_off[b] + j])
            if paged:
                bs, t = pf.cache_cfg["block_size"], pf.cache_cfg["block_table"]
                a = (slice(None), int(t[b][s_orig // bs]), s_orig % bs)
                c = (slice(None), new // bs, new % bs)
            else:
                a = (b, slice(None), slice(None), s_orig)
                c = (new // pf.cache_cfg["s_max"], slice(None), slice(None), new % pf.cache_cfg["s_max"])
            assert torch.equal(cache.k[a].view(torch.int16), cache.k[c].view(torch.int16))
            assert torch.equal(cache.v[a].view(torch.int16), cache.v[c].view(torch.int16))


# --- key-only memory ---------------------------------------------------------
KEY_ONLY = [("bf16", 128, (24, 20, 20), True), ("f32", 64, (8, 12, 12), False)]


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("dtype,D,sections,inter", KEY_ONLY)
def test_key_only_prefill_parity(dtype, D, sections, inter, paged):
    pf = Prefill(dtype, D, sections, inter, paged, key_only=True)
    _say(f"key-only prefill capture {dtype} D={D} paged={paged}")
    mem, cache, rope, err = pf.run_gpu()
    ref_mem, ref_cache, ref_err = pf.run_oracle()
    _compare(pf, mem, cache, err, ref_mem, ref_cache, ref_err)


def _key_only_revisit(pf, sel_off, sel_idx, fused, v_slot_patch=None):
    """Key-only prefill on both sides, then one PCR revisit on both; returns
    (GPU cache, slots, new lengths, err) and the oracle's result."""
    mem, cache, rope, err = pf.run_gpu()
    ref_mem, ref_cache, _ = pf.run_oracle()
    assert err == 0
    if v_slot_patch is not None:
        b, m, v = v_slot_patch
        mem.v_slot[b, m] = v
        ref_mem["v_slot"][b, m] = v
    p_txt = (pf.n_tokens - 1).astype(np.int32)
    err_t = torch.zeros(1, dtype=torch.int32, device=DEV)
    so, si = to_dev(sel_off), to_dev(sel_idx)
    if fused:
        _, _, new_len, slots = prcr.revisit(rope, mem, so, si, to_dev(p_txt), cache,
                                            to_dev(pf.n_tokens), "pcr", 2, err=err_t)
    else:
        new_pos, _ = prcr.reassign_coords(mem, so, si, to_dev(p_txt), "pcr", 2, err=err_t)
        new_len, slots = prcr.rebind_inject(rope, mem, so, si, new_pos, cache, to_dev(pf.n_tokens),
                                            err=err_t)
    torch.cuda.synchronize()
    pos_o, _, _ = oracle.reassign_batch(ref_mem["coords"], ref_mem["n_visual"], sel_off, sel_idx,
                                        p_txt, "pcr", 2)
    ref = oracle.rebind_inject(pf.rope, ref_mem, sel_off, sel_idx, pos_o, ref_cache, pf.n_tokens)
    return cache, slots.cpu().numpy(), new_len.cpu().numpy(), int(err_t.item()), ref


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("paged", [False, True])
def test_key_only_revisit_parity(paged, fused):
    """Values of the revisited tokens come from the prompt slots the prefill wrote."""
    pf = Prefill("bf16", 128, (16, 24, 24), False, paged, NL=4, H=4, key_only=True)
    sel_off = np.array([0, 5, 8], np.int32)
    sel_idx = np.array([0, 3, 7, 11, 23, 2, 5, 29], np.int32)
    _say(f"key-only revisit paged={paged} fused={fused}")
    cache, slots, new_len, err, ref = _key_only_revisit(pf, sel_off, sel_idx, fused)
    npy = workloads.as_numpy_storage
    assert err == ref["err"] == 0
    assert np.array_equal(slots, ref["slot_mapping"])
    assert np.array_equal(new_len, ref["new_cache_len"])
    assert np.array_equal(npy(cache.v), ref["v"])
    assert_keys_close(npy(cache.k), ref["k"], "bf16")


def test_key_only_value_slot_not_filled():
    """A value slot at or beyond cache_len is rejected: flag, token skipped."""
    pf = Prefill("bf16", 128, (16, 24, 24), False, False, NL=2, H=2, key_only=True)
    sel_off = np.array([0, 3, 5], np.int32)
    sel_idx = np.array([1, 4, 9, 2, 5], np.int32)
    patch = (0, 4, int(pf.n_tokens[0]))          # sequence 0, token 4 -> first free slot
    _say("key-only revisit with a value slot that is not filled")
    cache, slots, new_len, err, ref = _key_only_revisit(pf, sel_off, sel_idx, False, patch)
    npy = workloads.as_numpy_storage
    assert err == ref["err"] == oracle.ERR_INDEX
    assert slots[1] == -1 and np.array_equal(slots, ref["slot_mapping"])
    assert np.array_equal(npy(cache.v), ref["v"])
    assert_keys_close(npy(cache.k), ref["k"], "bf16")


def test_prefill_graph_replays_match_eager():
    """One layer of prcr_prefill_capture captured in a HIP graph: each replay, after
    eager work that restores the cache and the memory to their contents before the
    call, reproduces the eager result."""
    pf = Prefill("bf16", 128, (24, 20, 20), True, True, NL=2, H=4)
    _say("graph capture of prefill capture (paged), 3 replays")
    mem = prcr.Memory(pf.mem_k.to(DEV), pf.mem_v.to(DEV),
                      torch.zeros((pf.B, pf.M, 3), dtype=torch.int32, device=DEV),
                      to_dev(pf.n_visual))
    cache = prcr.Cache(pf.cache_k.to(DEV), pf.cache_v.to(DEV), to_dev(pf.cache_cfg["block_table"]))
    rope = prcr.Rope(pf.D, pf.rope["sections"], pf.rope["interleaved"], pf.rope["theta"])
    rk, rv = pf.raw[1][0].to(DEV), pf.raw[1][1].to(DEV)
    args = (to_dev(pf.pos), to_dev(pf.n_tokens), to_dev(pf.vis_index))
    start = torch.zeros(pf.B, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    s = torch.cuda.Stream(device=DEV)

    def call():
        prcr.prefill_capture(rope, mem, 1, rk, rv, *args, cache, start, True, err, s)

    outs = (cache.k, cache.v, mem.k, mem.v, mem.coords)
    before = [t.clone() for t in outs]
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        call()
    torch.cuda.synchronize()
    eager = [t.clone() for t in outs]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        call()
    torch.cuda.synchronize()
    for r in range(3):
        for t, t0 in zip(outs, before):
            t.copy_(t0)                                 # eager work between replays
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs, eager):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b), f"replay {r}"
    assert int(err.item()) == 0
