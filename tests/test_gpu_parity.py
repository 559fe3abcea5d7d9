"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bit-exact: new positions, next text positions, slot mapping, new cache lengths,
value rows and every cache byte outside the new slots.  Keys: within 1 bf16 ulp
(bfloat16) or 1e-5 relative, element by element (float32).  Each test prints what it
runs before touching the GPU.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, Case, assert_keys_close, assert_parity, run_both, to_dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("cfg", [1, 2, 3, 5])
def test_workload_small(cfg):
    w = workloads.make(cfg, "small")
    _say(f"workload {cfg} small: B={w.B} NL={w.NL} H={w.H} D={w.D} K={w.total_k}")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len)
    exact, n = assert_parity(case, gpu, ref)
    _say(f"  keys bit-exact {exact}/{n}")


def test_workload2_full_size():
    w = workloads.make(2, "full")
    _say(f"workload 2 full: NL={w.NL} K={w.total_k}")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len)
    exact, n = assert_parity(case, gpu, ref)
    _say(f"  keys bit-exact {exact}/{n}")


def test_video_four_revisits():
    """Workload 4: four successive revisits appending to the same cache."""
    w = workloads.make(4, "small")
    _say(f"workload 4 small: B={w.B} NL={w.NL}, 4 revisits of 1024")
    case = Case(w)
    lens = w.cache_len.astype(np.int64).copy()
    p_txt = w.p_txt.astype(np.int64).copy()
    for r, (so, si) in enumerate(w.revisits):
        gpu, ref = run_both(case, so, si, p_txt, lens)
        # the GPU cache tensors are updated in place; keep the oracle's copy in step
        assert_parity(case, gpu, ref)
        lens = ref["new_cache_len"] + w.decode_between
        p_txt = ref["next_pos"] + w.decode_between - 1
        _say(f"  revisit {r} ok, next_pos {ref['next_pos'].tolist()}")
    assert (lens <= w.s_max).all()


@pytest.mark.parametrize("mode", ["pcr", "shift", "identity", "lpa", "uir", "pcr_right"])
@pytest.mark.parametrize("cfg", [1, 3])
def test_modes(cfg, mode):
    w = workloads.make(cfg, "small")
    _say(f"workload {cfg} small, mode {mode}")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, mode=mode)
    assert_parity(case, gpu, ref)


@pytest.mark.parametrize("l_ext", [0, 1, 5])
def test_left_extension(l_ext):
    w = workloads.make(5, "small")
    _say(f"workload 5 small, L={l_ext}")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, l_ext=l_ext)
    assert_parity(case, gpu, ref)


COMPILED = [
    ("f32", 64, (8, 12, 12), False), ("f32", 64, (11, 11, 10), True),
    ("f32", 128, (16, 24, 24), False), ("f32", 128, (22, 21, 21), True),
    ("f32", 128, (24, 20, 20), True),
    ("bf16", 64, (8, 12, 12), False), ("bf16", 64, (11, 11, 10), True),
    ("bf16", 128, (16, 24, 24), False), ("bf16", 128, (22, 21, 21), True),
    ("bf16", 128, (24, 20, 20), True),
    # 1-D rotary: every pair on t (models without M-RoPE)
    ("f32", 64, (32, 0, 0), False), ("bf16", 128, (64, 0, 0), False),
    ("bf16", 128, (64, 0, 0), True),
]


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("dtype,D,sections,inter", COMPILED)
def test_every_instantiation_with_ragged_edges(dtype, D, sections, inter, paged):
    """Empty and one-token selections, 3 KV heads (rows not a multiple of a wave's
    rows), a token count that leaves a partial workgroup, block size 7."""
    w = workloads.custom(B=5, NL=3, H=3, D=D, dtype=dtype, sections=sections, interleaved=inter,
                         theta=5e6 if inter else 1e6, frames=2, gh=9, gw=7,
                         ks=(0, 1, 13, 0, 30), lens=(0, 11, 29, 3, 40), paged=paged, block_size=7)
    _say(f"custom {dtype} D={D} {sections} inter={inter} paged={paged} K={w.total_k}")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len)
    assert_parity(case, gpu, ref)


def test_empty_selection_writes_lengths_only():
    w = workloads.custom(B=4, ks=(0, 0, 0, 0), lens=(5, 0, 9, 2))
    _say("all-empty selection")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len)
    assert_parity(case, gpu, ref)
    assert gpu["new_cache_len"].tolist() == [5, 0, 9, 2]


def test_data_errors_are_flagged_and_skipped():
    w = workloads.custom(B=3, NL=2, H=2, ks=(6, 4, 5), lens=(10, 25, 5), s_max=28)
    sel_idx = w.sel_idx.copy()
    sel_idx[2] = w.M_max + 3           # index outside the memory
    sel_idx[3] = -1
    _say("bad indices + capacity overflow (sequence 1 runs past s_max)")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, sel_idx, w.p_txt, w.cache_len)
    assert ref["err"] == (oracle.ERR_INDEX | oracle.ERR_CAPACITY)
    assert_parity(case, gpu, ref)


def test_paged_block_errors_are_flagged_and_skipped():
    w = workloads.custom(B=3, NL=2, H=4, ks=(6, 4, 9), lens=(10, 20, 5), paged=True,
                         block_size=4)
    w.block_table = w.block_table.copy()
    w.block_table[0, 3] = w.n_blocks + 5            # slot 12..15 of sequence 0
    w.block_table[2, -1] = -1
    _say("paged: block id outside the pool, missing block")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len)
    assert ref["err"] & oracle.ERR_BLOCK
    assert_parity(case, gpu, ref)


def test_malformed_offsets_flagged():
    w = workloads.custom(B=3, ks=(5, 0, 3), lens=(3, 4, 5))
    case = Case(w)
    mem, cache = case.memory(), case.cache()
    bad_off = to_dev(np.array([0, 5, 3, 8], np.int32))     # not non-decreasing
    si = to_dev(w.sel_idx)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    _say("malformed sel_off")
    pos, nxt = prcr.reassign_coords(mem, bad_off, si, to_dev(w.p_txt), err=err)
    _, slots = prcr.rebind_inject(case.rope(), mem, bad_off, si, pos, cache, to_dev(w.cache_len),
                                  err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & prcr.DERR_OFFSETS
    assert (slots.cpu().numpy() >= -1).all()


@pytest.mark.parametrize("bad", [[0, 5, 5, 100], [-4, 5, 5, 8]])
def test_malformed_offsets_fused(bad):
    """The single-launch revisit with offsets outside [0, total_k]: the tokens of
    the malformed sequence are skipped with PRCR_DERR_OFFSETS, and its range
    reduction reads no index beyond the selection."""
    w = workloads.custom(B=3, ks=(5, 0, 3), lens=(3, 4, 5))
    case = Case(w)
    mem, cache = case.memory(), case.cache()
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    _say(f"fused revisit with sel_off {bad}")
    _, _, _, slots = prcr.revisit(case.rope(), mem, to_dev(np.array(bad, np.int32)), to_dev(w.sel_idx),
                                  to_dev(w.p_txt), cache, to_dev(w.cache_len), "pcr", 2, err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & prcr.DERR_OFFSETS
    sl = slots.cpu().numpy()
    skipped = slice(5, 8) if bad[-1] != 8 else slice(0, 5)
    assert (sl[skipped] == -1).all()
    assert (sl >= -1).all()


def test_position_range_flag():
    """A PCR rational too large for exact double division is flagged and stays close."""
    w = workloads.custom(B=1, ks=(40,), lens=(7,), gh=12, gw=10)
    w.coords = w.coords.copy()
    w.coords[0, :, 1] *= 100_000_000                 # h span ~1e9
    p_txt = np.array([2_000_000_000], np.int32)
    case = Case(w)
    mem = case.memory()
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    _say("huge coordinate span")
    pos, nxt = prcr.reassign_coords(mem, to_dev(w.sel_off), to_dev(w.sel_idx), to_dev(p_txt), err=err)
    torch.cuda.synchronize()
    ref, nref, _ = oracle.reassign_batch(w.coords, w.n_visual, w.sel_off, w.sel_idx, p_txt)
    assert int(err.item()) == prcr.DERR_RANGE
    assert np.allclose(pos.cpu().numpy(), ref, rtol=4e-16, atol=0)
    assert np.array_equal(nxt.cpu().numpy(), nref)


def test_nondefault_stream():
    w = workloads.make(3, "small")
    _say("workload 3 small on a side stream")
    case = Case(w)
    torch.cuda.synchronize()
    s = torch.cuda.Stream(device=DEV)
    with torch.cuda.stream(s):
        gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, stream=s)
    assert_parity(case, gpu, ref)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_store_raw(dtype):
    B, S, NL, H, D = 3, 50, 4, 4, 128
    M = 33
    g = torch.Generator().manual_seed(5)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    raw_k = torch.randn((B, S, H, D), generator=g).to(tdt)
    raw_v = torch.randn((B, S, H, D), generator=g).to(tdt)
    rng = np.random.default_rng(5)
    vis = np.stack([rng.choice(S, M, replace=False) for _ in range(B)]).astype(np.int32)
    vis[1, 7] = S + 2                                   # bad source row
    nvis = np.array([33, 20, 0], np.int32)
    mk = torch.zeros((B, M, NL, H, D), dtype=tdt)
    mv = torch.zeros_like(mk)
    _say(f"store_raw {dtype}")
    mem = prcr.Memory(mk.to(DEV), mv.to(DEV), torch.zeros((B, M, 3), dtype=torch.int32, device=DEV),
                      to_dev(nvis))
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    for layer in range(NL):
        prcr.store_raw(mem, layer, raw_k.to(DEV), raw_v.to(DEV), to_dev(vis), err=err)
    torch.cuda.synchronize()
    ek, ev = workloads.as_numpy_storage(mk), workloads.as_numpy_storage(mv)
    hk, hv = workloads.as_numpy_storage(raw_k), workloads.as_numpy_storage(raw_v)
    e_all = 0
    for layer in range(NL):
        ek, ev, e = oracle.store_raw(ek, ev, layer, hk, hv, vis, nvis)
        e_all |= e
    assert int(err.item()) == e_all == oracle.ERR_INDEX
    assert np.array_equal(workloads.as_numpy_storage(mem.k), ek)
    assert np.array_equal(workloads.as_numpy_storage(mem.v), ev)


# ---------------------------------------------------------------------------
# The fused single-launch revisit (prcr_revisit) against the same oracle.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("cfg", [1, 2, 3, 5])
def test_fused_workload_small(cfg):
    w = workloads.make(cfg, "small")
    _say(f"fused: workload {cfg} small")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, fused=True)
    assert_parity(case, gpu, ref)


@pytest.mark.parametrize("mode", ["pcr", "shift", "identity", "lpa", "uir", "pcr_right"])
def test_fused_modes(mode):
    w = workloads.make(3, "small")
    _say(f"fused: workload 3 small, mode {mode}")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, mode=mode, l_ext=3,
                        fused=True)
    assert_parity(case, gpu, ref)


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("dtype,D,sections,inter", [COMPILED[0], COMPILED[4], COMPILED[7],
                                                    COMPILED[9], COMPILED[11]])
def test_fused_ragged_edges(dtype, D, sections, inter, paged):
    w = workloads.custom(B=5, NL=3, H=3, D=D, dtype=dtype, sections=sections, interleaved=inter,
                         theta=5e6 if inter else 1e6, frames=2, gh=9, gw=7,
                         ks=(0, 1, 13, 0, 30), lens=(0, 11, 29, 3, 40), paged=paged, block_size=7)
    _say(f"fused: custom {dtype} D={D} {sections} inter={inter} paged={paged}")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, mode="shift", fused=True)
    assert_parity(case, gpu, ref)


def test_fused_data_errors():
    w = workloads.custom(B=3, NL=2, H=2, ks=(6, 4, 5), lens=(10, 25, 5), s_max=28)
    sel_idx = w.sel_idx.copy()
    sel_idx[0] = w.M_max + 3          # the first token of sequence 0 is invalid
    sel_idx[3] = -1
    _say("fused: bad indices (including a sequence's first token) + capacity overflow")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, sel_idx, w.p_txt, w.cache_len, fused=True)
    assert ref["err"] == (oracle.ERR_INDEX | oracle.ERR_CAPACITY)
    assert_parity(case, gpu, ref)


def test_fused_video_four_revisits():
    w = workloads.make(4, "small")
    _say("fused: workload 4 small, 4 revisits")
    case = Case(w)
    lens = w.cache_len.astype(np.int64).copy()
    p_txt = w.p_txt.astype(np.int64).copy()
    for so, si in w.revisits:
        gpu, ref = run_both(case, so, si, p_txt, lens, fused=True)
        assert_parity(case, gpu, ref)
        lens = ref["new_cache_len"] + w.decode_between
        p_txt = ref["next_pos"] + w.decode_between - 1


def test_graph_replays_match_eager():
    """prcr_revisit captured in a HIP graph: every replay, with eager work that
    clobbers the target rows in between, reproduces the eager result."""
    w = workloads.make(5, "small")
    _say("graph capture of prcr_revisit (workload 5 small), 3 replays")
    case = Case(w)
    mem, cache, rope = case.memory(), case.cache(), case.rope()
    so, si = to_dev(w.sel_off), to_dev(w.sel_idx)
    pt, cl = to_dev(w.p_txt), to_dev(w.cache_len)
    new_pos = torch.empty((w.total_k, 3), dtype=torch.float64, device=DEV)
    next_pos = torch.empty((w.B,), dtype=torch.int32, device=DEV)
    new_len = torch.empty((w.B,), dtype=torch.int32, device=DEV)
    slots = torch.empty((w.total_k,), dtype=torch.int64, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    s = torch.cuda.Stream(device=DEV)
    torch.cuda.synchronize()

    def call():
        prcr.revisit(rope, mem, so, si, pt, cache, cl, "pcr", 2, new_pos, next_pos, new_len,
                     slots, err, s)

    with torch.cuda.stream(s):
        call()
    torch.cuda.synchronize()
    eager = [t.clone() for t in (cache.k, cache.v, new_pos, next_pos, new_len, slots)]
    blk = slots // w.block_size
    off = slots % w.block_size
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        call()
    torch.cuda.synchronize()
    for r in range(3):
        cache.k[:, blk, off] = 0                    # eager work between replays
        cache.v[:, blk, off] = 0
        new_pos.zero_(); next_pos.zero_(); new_len.zero_(); slots.fill_(-7)
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize()
        for a, b in zip((cache.k, cache.v, new_pos, next_pos, new_len, slots), eager):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a,
                               b.view(torch.int16) if b.dtype == torch.bfloat16 else b), f"replay {r}"
    assert int(err.item()) == 0


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("paged", [False, True])
def test_many_sequences(paged, fused):
    """3000 sequences of 0-3 selected tokens each (a token's sequence is found by a
    ballot over all 3001 selection offsets, 47 rounds of 64), against the oracle."""
    rng = np.random.default_rng(300)
    B = 3000
    ks = rng.integers(0, 4, B)
    lens = rng.integers(0, 21, B)
    w = workloads.custom(B=B, NL=2, H=1, D=64, dtype="f32", sections=(8, 12, 12), gh=3, gw=4,
                         ks=tuple(int(k) for k in ks), lens=tuple(int(x) for x in lens),
                         paged=paged, block_size=5, seed=301)
    _say(f"{B} sequences, total_k={w.total_k}, paged={paged}, fused={fused}")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, fused=fused)
    assert_parity(case, gpu, ref)


@pytest.mark.parametrize("ks", [
    (300,) + (1,) * 9,          # mean 31: 64-thread workgroups, the long sequence in 5 rounds
    (700, 1, 0, 3),             # mean 176: 256 threads, 3 rounds
    (900, 100),                 # mean 500: 512 threads, 2 rounds
    (2000, 600),                # mean 1300: 1024 threads, 2 rounds
])
def test_reassign_skewed_selections(ks):
    """The reassignment sizes its workgroup to the mean selection per sequence, so a
    sequence far above the mean loops over its tokens in several rounds: positions,
    next positions and the rebound rows against the oracle."""
    lens = tuple(10 + 3 * i for i in range(len(ks)))
    w = workloads.custom(B=len(ks), NL=1, H=1, D=64, dtype="f32", sections=(8, 12, 12),
                         frames=4, gh=24, gw=24, ks=ks, lens=lens, seed=500 + len(ks))
    _say(f"skewed selections {ks[:4]}..., total_k={w.total_k}")
    case = Case(w)
    for fused in (False, True):
        gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, fused=fused)
        assert_parity(case, gpu, ref)
        case = Case(w)


@pytest.mark.parametrize("dtype,paged", [("bf16", False), ("bf16", True), ("f32", False)])
def test_special_values(dtype, paged):
    """NaN, infinities, the largest finite value (whose rotation overflows), the
    smallest subnormal and signed zeros in the selected tokens' raw rows.  Values
    (NaN payloads included) are copied bit for bit; keys follow the oracle: NaN
    where it has NaN, equal infinities, finite results within the key tolerance."""
    w = workloads.custom(B=3, NL=2, H=2, dtype=dtype, ks=(4, 1, 6), lens=(5, 17, 2), paged=paged,
                         block_size=8)
    vals = workloads.torch_values(w, "cpu")
    big = 3.3895313892515355e38 if dtype == "bf16" else 3.4028234663852886e38
    tiny = 9.183549615799121e-41 if dtype == "bf16" else 1.401298464324817e-45
    k, v = vals["mem_k"], vals["mem_v"]
    for j in range(w.total_k):
        b = int(np.searchsorted(w.sel_off, j, side="right") - 1)
        m = int(w.sel_idx[j])
        row = k[b, m, j % w.NL, j % w.H]
        row[3] = float("nan")
        row[10], row[74] = float("inf"), 1.0
        row[70] = float("-inf")
        row[20], row[84] = big, big
        row[21], row[85] = -big, big
        row[30] = tiny
        row[40], row[104] = -0.0, 0.0
        vrow = v[b, m, (j + 1) % w.NL, (j + 1) % w.H]
        vrow[5] = float("nan")
        vrow[6] = float("-inf")
        vrow[7] = tiny
    if dtype == "bf16":
        vb = v.view(torch.int16)
        vb[0, int(w.sel_idx[0]), 0, 0, 9] = 0x7FC1                     # NaN with a payload
        vb[0, int(w.sel_idx[0]), 0, 0, 11] = -0x0040                     # 0xFFC0: negative NaN
    else:
        vi = v.view(torch.int32)
        vi[0, int(w.sel_idx[0]), 0, 0, 9] = 0x7FC00001
        vi[0, int(w.sel_idx[0]), 0, 0, 11] = -0x00400000                 # 0xFFC00000
    _say(f"special values: {dtype}, paged={paged}, {w.total_k} tokens")
    case = Case(w, vals)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len)
    assert np.isnan(oracle.storage_to_f64(ref["k"], dtype)).any()      # the specials reached the keys
    assert np.isinf(oracle.storage_to_f64(ref["k"], dtype)).any()
    exact, n = assert_parity(case, gpu, ref)
    _say(f"  keys equal to the oracle {exact}/{n}")


INT32_MAX, INT32_MIN = 2**31 - 1, -2**31


@pytest.mark.parametrize("fused", [False, True], ids=["two-call", "fused"])
@pytest.mark.parametrize("mode,p_txt", [("shift", INT32_MAX - 3), ("lpa", INT32_MAX - 9),
                                        ("pcr", INT32_MAX), ("uir", INT32_MAX)])
def test_next_position_beyond_int32(mode, p_txt, fused):
    """The next text position is returned as int32: a value beyond its range is
    saturated and flagged with PRCR_DERR_RANGE, never wrapped.  Positions (double)
    and keys follow the oracle as usual."""
    w = workloads.make(1, "small")
    _say(f"workload 1, mode {mode}, p_txt {p_txt}, {'fused' if fused else 'two-call'}")
    case = Case(w)
    pt = np.full(w.B, p_txt, np.int64)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, pt, w.cache_len, mode=mode, fused=fused)
    nxt = np.asarray(ref["next_pos"], np.int64)
    over = (nxt > INT32_MAX) | (nxt < INT32_MIN)
    assert over.all()                       # the case reaches beyond int32
    ref["next_pos"] = np.clip(nxt, INT32_MIN, INT32_MAX)
    ref["err"] |= prcr.DERR_RANGE
    assert_parity(case, gpu, ref)


def test_revisit_refuses_outputs_over_its_inputs():
    """next_pos over p_txt (an in-place advance) or over cache_len, and new lengths
    over p_txt, race with the other waves of the single launch: refused by the
    binding and, called directly, by the C ABI (PRCR_ERR_ALIAS), before any launch."""
    import ctypes
    w = workloads.make(1, "small")
    _say("alias refusal: workload 1, binding and C ABI")
    case = Case(w)
    mem, cache = case.memory(), case.cache()
    so, si = to_dev(w.sel_off), to_dev(w.sel_idx)
    pt, cl = to_dev(w.p_txt), to_dev(w.cache_len)
    for kw in (dict(next_pos=pt), dict(next_pos=cl), dict(new_cache_len=pt)):
        with pytest.raises(ValueError):
            prcr.revisit(case.rope(), mem, so, si, pt, cache, cl, "pcr", 2, **kw)
    L = prcr.lib()
    slots = torch.empty(w.total_k, dtype=torch.int64, device=DEV)
    new_len = torch.empty(w.B, dtype=torch.int32, device=DEV)
    st = L.prcr_revisit(ctypes.byref(case.rope().to_c()), ctypes.byref(mem.to_c()),
                        so.data_ptr(), si.data_ptr(), w.total_k, pt.data_ptr(), 0, 2,
                        ctypes.byref(cache.to_c()), cl.data_ptr(), None, pt.data_ptr(),
                        new_len.data_ptr(), slots.data_ptr(), None, None)
    assert st == 7
    torch.cuda.synchronize()
    assert np.array_equal(pt.cpu().numpy(), w.p_txt)           # nothing was launched
