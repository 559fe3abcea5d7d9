"""Randomized GPU parity: many small configurations drawn from a fixed seed.

Each draws:
* the storage type, head dimension and axis map (every compiled map, 1-D included);
* a contiguous or paged cache, with block sizes from 1 to 32;
* the sequence, layer and head counts;
* the visual grid (with frames), the per-sequence selection sizes (empty included) and
  the cache lengths;
* the reassignment rule, the left extension, and the two-call or fused path.

Each configuration is checked against the oracle to the parity bar: bit-exact
positions, slots, lengths and values, keys within the key tolerance.  Decode
attention gets random configurations of its own (grouped-query ratio, lengths,
capacity, layout), checked to the decode tolerance, and so does the prefill capture
(prompt mixes of text and images or video frames, cache offsets, key-only memory).  The
raw-memory store gets random storage types, head dims, counts, source rows and layer
orders, with every byte of the memory compared."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, Case, assert_parity, run_both, to_dev
from test_gpu_prefill import Prefill, _compare

pytestmark = pytest.mark.gpu

MAPS = {64: [((8, 12, 12), False), ((11, 11, 10), True), ((32, 0, 0), False)],
        128: [((16, 24, 24), False), ((22, 21, 21), True), ((24, 20, 20), True),
              ((64, 0, 0), False), ((64, 0, 0), True)]}
MODES = ["pcr", "shift", "identity", "lpa", "uir", "pcr_right"]


def _draw(seed):
    r = np.random.default_rng(seed)
    D = int(r.choice([64, 128]))
    sections, inter = MAPS[D][int(r.integers(len(MAPS[D])))]
    B = int(r.integers(1, 7))
    frames, gh, gw = int(r.integers(1, 4)), int(r.integers(1, 10)), int(r.integers(1, 10))
    M = frames * gh * gw
    ks = tuple(int(r.integers(0, min(M, 40) + 1)) for _ in range(B))
    lens = tuple(int(r.integers(0, 61)) for _ in range(B))
    paged = bool(r.integers(2))
    w = workloads.custom(B=B, NL=int(r.integers(1, 5)), H=int(r.integers(1, 6)), D=D,
                         dtype=str(r.choice(["f32", "bf16"])), sections=sections, interleaved=inter,
                         theta=float(r.choice([1e4, 1e6, 5e6])), frames=frames, gh=gh, gw=gw,
                         ks=ks, lens=lens, paged=paged, block_size=int(r.choice([1, 3, 16, 32])),
                         seed=seed)
    return w, str(r.choice(MODES)), int(r.integers(0, 5)), bool(r.integers(2))


@pytest.mark.parametrize("seed", range(9000, 9200))
def test_random_configuration(seed):
    w, mode, l_ext, fused = _draw(seed)
    print(f"seed {seed}: {w.dtype} D={w.D} {w.sections} inter={w.interleaved} B={w.B} NL={w.NL} "
          f"H={w.H} M={w.M_max} K={list(np.diff(w.sel_off))} paged={w.paged} "
          f"bs={w.block_size} mode={mode} L={l_ext} fused={fused}", flush=True)
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, mode=mode, l_ext=l_ext,
                        fused=fused)
    assert_parity(case, gpu, ref)


@pytest.mark.parametrize("seed", range(9500, 9540))
def test_random_decode_configuration(seed):
    r = np.random.default_rng(seed)
    D = int(r.choice([64, 128]))
    sections, inter = MAPS[D][int(r.integers(len(MAPS[D])))]
    dtype = str(r.choice(["f32", "bf16"]))
    B, H, G, NL = int(r.integers(1, 6)), int(r.choice([1, 2, 3, 4, 8])), int(r.choice([1, 2, 3, 4, 7, 8])), 2
    layer = int(r.integers(NL))
    cap = int(r.integers(1, 400))
    lens = r.integers(0, cap + 1, B).astype(np.int32)
    paged = bool(r.integers(2))
    print(f"seed {seed}: decode {dtype} D={D} {sections} B={B} H={H} G={G} cap={cap} "
          f"lens={lens.tolist()} paged={paged}", flush=True)
    g = torch.Generator().manual_seed(seed)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rnd = lambda *shape: (torch.randn(shape, generator=g) * float(r.choice([0.1, 1.0, 2.0]))).to(tdt)
    if paged:
        bs = int(r.choice([1, 5, 16]))
        need = (cap + bs - 1) // bs
        n_blocks = B * need + int(r.integers(0, 4))
        table = r.permutation(n_blocks)[:B * need].astype(np.int32).reshape(B, need)
        k, v = rnd(NL, n_blocks, bs, H, D), rnd(NL, n_blocks, bs, H, D)
        cache_o = {"paged": True, "block_size": bs, "block_table": table, "max_blocks": need,
                   "n_blocks": n_blocks}
    else:
        k, v = rnd(B, NL, H, cap, D), rnd(B, NL, H, cap, D)
        cache_o = {"paged": False, "s_max": cap}
    cache_o["k"], cache_o["v"] = workloads.as_numpy_storage(k), workloads.as_numpy_storage(v)
    q = rnd(B, H * G, D)
    q_pos = r.integers(0, 100000, B).astype(np.int32)
    cache = prcr.Cache(k.to(DEV), v.to(DEV), to_dev(cache_o["block_table"]) if paged else None)
    rope = prcr.Rope(D, sections, inter, 1e6)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q.to(DEV), to_dev(q_pos), to_dev(lens), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = oracle.decode_attention(rope.__dict__ | {"sections": rope.sections}, cache_o, layer,
                                  workloads.as_numpy_storage(q), q_pos, lens, D ** -0.5, dtype)
    out = out.cpu().numpy()
    for b in range(B):
        n = int(lens[b])
        for kvh in range(H):
            vmax = np.abs(oracle.storage_to_f64(oracle.cache_rows(cache_o, layer, b, kvh, n, "v"),
                                                dtype)).max() if n else 0.0
            for gg in range(G):
                qh = kvh * G + gg
                d = np.abs(out[b, qh] - ref[b, qh]).max()
                assert d <= 5e-5 * vmax + 1e-6, (b, qh, d, vmax)


@pytest.mark.parametrize("seed", range(9700, 9730))
def test_random_prefill_configuration(seed):
    r = np.random.default_rng(seed)
    D = int(r.choice([64, 128]))
    sections, inter = MAPS[D][int(r.integers(len(MAPS[D])))]
    B = int(r.integers(1, 4))
    prompt = {"B": B, "n_before": tuple(int(x) for x in r.integers(0, 12, B)),
              "grid": tuple((int(r.integers(1, 7)), int(r.integers(1, 7))) for _ in range(B)),
              "n_after": tuple(int(x) for x in r.integers(0, 9, B)),
              "frames": tuple(int(x) for x in r.integers(1, 4, B))}
    dtype = str(r.choice(["f32", "bf16"]))
    paged, key_only = bool(r.integers(2)), bool(r.integers(2))
    pf = Prefill(dtype, D, sections, inter, paged, NL=int(r.integers(1, 4)), H=int(r.integers(1, 5)),
                 seed=seed, key_only=key_only, prompt=prompt, block_size=int(r.choice([1, 4, 16])))
    start = r.integers(0, 17, pf.B).astype(np.int32)
    print(f"seed {seed}: prefill {dtype} D={D} {sections} inter={inter} prompt={prompt} "
          f"NL={pf.NL} H={pf.H} paged={paged} key_only={key_only} start={start.tolist()}", flush=True)
    mem, cache, rope, err = pf.run_gpu(start=start)
    ref_mem, ref_cache, ref_err = pf.run_oracle(start=start)
    _compare(pf, mem, cache, err, ref_mem, ref_cache, ref_err)


def _bits(t):
    a = workloads.as_numpy_storage(t)
    return a.view(np.uint32) if a.dtype == np.float32 else a


@pytest.mark.parametrize("seed", range(9800, 9830))
def test_random_store_configuration(seed):
    """prcr_store_raw on a random configuration: storage type, head dim (any whose half
    row is whole 16-byte chunks), head, sequence, visual-token and layer counts, ragged
    counts (zero and full included), repeated and out-of-range source rows, a key-only
    memory, several layers in a random order.  Every byte of the memory against the
    oracle."""
    r = np.random.default_rng(seed)
    dtype = "f32" if r.integers(2) else "bf16"
    D = int(r.choice([8, 16, 24, 32, 64, 96, 128] if dtype == "f32" else [16, 32, 64, 96, 128]))
    H, B, M, NL = int(r.integers(1, 17)), int(r.integers(1, 41)), int(r.integers(1, 81)), int(r.integers(1, 6))
    S = int(r.integers(1, 2 * M + 2))
    key_only = bool(r.integers(4) == 0)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    print(f"seed {seed}: store_raw {dtype} D={D} H={H} B={B} M={M} S={S} NL={NL} key_only={key_only}",
          flush=True)
    g = torch.Generator().manual_seed(seed)
    raw_k = torch.randn((B, S, H, D), generator=g).to(tdt)
    raw_v = torch.randn((B, S, H, D), generator=g).to(tdt)
    mk = torch.randn((B, M, NL, H, D), generator=g).to(tdt)
    mv = None if key_only else torch.randn((B, M, NL, H, D), generator=g).to(tdt)
    vis = r.integers(0, S, (B, M)).astype(np.int32)             # repeats allowed
    bad = r.random((B, M)) < 0.03
    vis[bad] = np.where(r.integers(2, size=int(bad.sum())) == 0, -1 - r.integers(0, 5, int(bad.sum())),
                        S + r.integers(0, 5, int(bad.sum())))
    nvis = r.integers(0, M + 1, B).astype(np.int32)
    nvis[r.random(B) < 0.2] = M
    nvis[r.random(B) < 0.1] = 0
    layers = [int(x) for x in r.integers(0, NL, int(r.integers(1, 2 * NL + 1)))]
    mem = prcr.Memory(mk.to(DEV), None if key_only else mv.to(DEV),
                      torch.zeros((B, M, 3), dtype=torch.int32, device=DEV), to_dev(nvis),
                      to_dev(np.zeros((B, M), np.int32)) if key_only else None)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    rk, rv, vd = raw_k.to(DEV), raw_v.to(DEV), to_dev(vis)
    for layer in layers:
        prcr.store_raw(mem, layer, rk, None if key_only else rv, vd, err=err)
    torch.cuda.synchronize()
    ek, ev = _bits(mk), None if key_only else _bits(mv)
    e_all = 0
    for layer in layers:
        ek, ev, e = oracle.store_raw(ek, ev, layer, _bits(raw_k), _bits(raw_v), vis, nvis)
        e_all |= e
    assert int(err.item()) == e_all
    assert np.array_equal(_bits(mem.k), ek)
    if not key_only:
        assert np.array_equal(_bits(mem.v), ev)
