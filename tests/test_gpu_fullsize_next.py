"""Full-size parity of prefill capture and decode attention, in the shapes and
launch configuration that bench.py times.

Prefill capture (Eq. (4), (6)-(7)): 32 prompts x 2560 tokens (2048 visual, a
64 x 32 grid), 36 layers x 8 KV heads, d 128, bf16, interleaved M-RoPE
[22, 21, 21], one layer per call.
* every (token, head) key row against the oracle's rotation of the raw row at the
  token's position ids (within 1 bf16 ulp; the oracle in worker processes);
* every cache value row equals its raw row bit for bit, every memory row of a
  visual token equals the raw rows, the coordinates equal the prompt's position ids;
* every other byte of the cache and of the memory is unchanged (compared on the
  GPU against copies taken before the call).

Decode attention (Eq. (14)): the active cache of the 32-sequence workload after
its revisit (lengths 2801-4246), 8 KV heads, 32 query heads, d 128, bf16, on the
first and the last layer, and of the paged 64-sequence workload (4 KV heads, 16
query heads, block 16) on its last layer; every (sequence, query head) output
against the oracle, with the tolerance of the small-size tests.  The paged rows
are gathered through the block table with torch indexing, independently of the
kernel.
"""
import multiprocessing as mp
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, bf16_key, to_dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _i16(t):
    return t.view(torch.int16)


def test_prefill_capture_full_size():
    B, NL, H, D, layer = 32, 36, 8, 128, 17
    pos, vis, n_tok, n_vis = workloads.prompt(B, n_before=(256,) * B, grid=((64, 32),) * B,
                                              n_after=(256,) * B, frames=(1,) * B)
    S, M = pos.shape[1], int(n_vis.max())
    _say(f"prefill capture full size: {B} x {S} tokens, layer {layer}")
    g = torch.Generator(device=DEV)
    g.manual_seed(3000)
    raw_k = torch.randn((B, S, H, D), generator=g, device=DEV).to(torch.bfloat16)
    raw_v = torch.randn((B, S, H, D), generator=g, device=DEV).to(torch.bfloat16)
    mem = prcr.Memory(torch.randn((B, M, NL, H, D), generator=g, device=DEV).to(torch.bfloat16),
                      torch.randn((B, M, NL, H, D), generator=g, device=DEV).to(torch.bfloat16),
                      torch.full((B, M, 3), -7, dtype=torch.int32, device=DEV), to_dev(n_vis))
    s_max = S + 256
    cache = prcr.Cache(torch.randn((B, NL, H, s_max, D), generator=g, device=DEV).to(torch.bfloat16),
                       torch.randn((B, NL, H, s_max, D), generator=g, device=DEV).to(torch.bfloat16))
    rope = prcr.Rope(D, (22, 21, 21), True, 5e6)
    before = [t.clone() for t in (cache.k, cache.v, mem.k, mem.v, mem.coords)]

    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    start = torch.zeros(B, dtype=torch.int32, device=DEV)
    prcr.prefill_capture(rope, mem, layer, raw_k, raw_v, to_dev(pos), to_dev(n_tok), to_dev(vis),
                         cache, start, True, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert (n_tok == S).all()

    # every row: values, memory rows, coordinates, key norms
    ck, cv = cache.k[:, layer].transpose(1, 2), cache.v[:, layer].transpose(1, 2)   # [B][s][H][D]
    assert torch.equal(_i16(cv[:, :S]), _i16(raw_v)), "a cache value row differs from its raw row"
    vis_t = to_dev(vis).long()
    bb, ss = torch.nonzero(vis_t >= 0, as_tuple=True)
    mm = vis_t[bb, ss]
    assert torch.equal(_i16(mem.k[bb, mm, layer]), _i16(raw_k[bb, ss])), "a memory key row differs"
    assert torch.equal(_i16(mem.v[bb, mm, layer]), _i16(raw_v[bb, ss])), "a memory value row differs"
    assert torch.equal(mem.coords[bb, mm], to_dev(pos)[bb, ss]), "memory coordinates differ"
    P = D // 2
    for b0 in range(0, B, 4):
        x = raw_k[b0:b0 + 4].float()
        y = ck[b0:b0 + 4, :S].float()
        nx = x[..., :P] ** 2 + x[..., P:] ** 2
        ny = y[..., :P] ** 2 + y[..., P:] ** 2
        assert bool(((ny - nx).abs() <= 2.0 ** -6 * nx + 1e-30).all()), "a key pair changed norm"

    # every other byte: the cache outside this layer's prompt slots, the memory
    # outside this layer's rows of visual tokens, coordinates of non-visual entries
    written = torch.zeros(cache.k.shape[:-1], dtype=torch.bool, device=DEV)
    written[:, layer, :, :S] = True
    for now, old, name in ((cache.k, before[0], "cache key"), (cache.v, before[1], "cache value")):
        changed = (_i16(now) != _i16(old)).any(-1)
        assert not bool((changed & ~written).any()), f"a {name} row outside the prompt changed"
    mwritten = torch.zeros(mem.k.shape[:-2], dtype=torch.bool, device=DEV)     # [B][M][NL]
    mwritten[bb, mm, layer] = True
    for now, old, name in ((mem.k, before[2], "memory key"), (mem.v, before[3], "memory value")):
        changed = (_i16(now) != _i16(old)).any(-1).any(-1)
        assert not bool((changed & ~mwritten).any()), f"a {name} row outside the visual rows changed"
    cwritten = torch.zeros((B, M), dtype=torch.bool, device=DEV)
    cwritten[bb, mm] = True
    assert not bool(((mem.coords != before[4]).any(-1) & ~cwritten).any()), "coordinates changed"
    del before, written, mwritten

    # every key row against the oracle's rotation at the token's position ids
    got = workloads.as_numpy_storage(ck[:, :S])                     # [B][S][H][D]
    raw = workloads.as_numpy_storage(raw_k)
    rope_d = {"head_dim": D, "sections": (22, 21, 21), "interleaved": True, "theta": 5e6}
    tasks = [(rope_d, raw[b], "bf16", pos[b].astype(np.float64)[:, None, :]) for b in range(B)]
    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    _say(f"  oracle over {len(tasks)} prompts, {workers} worker processes")
    with mp.get_context("spawn").Pool(workers) as pool:
        refs = pool.starmap(oracle.rebind_row, tasks)
    exact = 0
    for b, ref in enumerate(refs):
        d = np.abs(bf16_key(got[b]) - bf16_key(ref))
        assert d.max() <= 1, f"prompt {b}: {int((d > 1).sum())} key elements beyond 1 bf16 ulp"
        exact += int((d == 0).sum())
    _say(f"keys: {exact}/{got.size} elements bit-exact, the rest within 1 bf16 ulp")


@pytest.mark.parametrize("cfg,layer", [(3, 0), (3, 35), (5, 27)])
def test_decode_attention_full_size(cfg, layer):
    w = workloads.make(cfg, "full")
    Hq = 4 * w.H
    _say(f"decode attention full size: workload {cfg}, {w.B} sequences, {w.H} KV heads, "
         f"{Hq} query heads, layer {layer}, paged={w.paged}")
    g = torch.Generator(device=DEV)
    g.manual_seed(4000 + layer)
    shape = workloads.cache_shape(w)
    cache = prcr.Cache(torch.randn(shape, generator=g, device=DEV).to(torch.bfloat16),
                       torch.randn(shape, generator=g, device=DEV).to(torch.bfloat16),
                       to_dev(w.block_table) if w.paged else None)
    rope = prcr.Rope(w.D, w.sections, w.interleaved, w.theta)
    lens = (w.cache_len + np.diff(w.sel_off)).astype(np.int32)
    q = torch.randn((w.B, Hq, w.D), generator=g, device=DEV).to(torch.bfloat16)
    q_pos = (w.p_txt + 1).astype(np.int32)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q, to_dev(q_pos), to_dev(lens), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    out = out.cpu().numpy()
    q_np = workloads.as_numpy_storage(q)
    rope_d = {"head_dim": w.D, "sections": w.sections, "interleaved": w.interleaved,
              "theta": w.theta}
    G = Hq // w.H
    worst = 0.0
    for b in range(w.B):
        n = int(lens[b])
        for kvh in range(w.H):
            if w.paged:
                slots = np.arange(n)
                blk = torch.from_numpy(w.block_table[b, slots // w.block_size].astype(np.int64)).to(DEV)
                off = torch.from_numpy((slots % w.block_size).astype(np.int64)).to(DEV)
                k = workloads.as_numpy_storage(cache.k[layer, blk, off, kvh])
                v = workloads.as_numpy_storage(cache.v[layer, blk, off, kvh])
            else:
                k = workloads.as_numpy_storage(cache.k[b, layer, kvh, :n])
                v = workloads.as_numpy_storage(cache.v[b, layer, kvh, :n])
            worst = max(worst, _check_group(rope_d, w, k, v, n, q_np, q_pos, out, b, kvh, G))
    _say(f"decode attention: every output, worst |out - ref| / max|V| = {worst:.2e}")


def _check_group(rope_d, w, k, v, n, q_np, q_pos, out, b, kvh, G):
    """The G query heads of KV head kvh of sequence b against the oracle; returns the
    largest |out - ref| / max|V|."""
    one = {"paged": False, "s_max": n, "k": k[None, None, None], "v": v[None, None, None]}
    vmax = np.abs(oracle.storage_to_f64(v, "bf16")).max()
    worst = 0.0
    for qh in range(kvh * G, (kvh + 1) * G):
        ref = oracle.decode_attention(rope_d, one, 0, q_np[b:b + 1, qh:qh + 1], q_pos[b:b + 1],
                                      np.array([n]), w.D ** -0.5, "bf16")[0, 0]
        dmax = np.abs(out[b, qh] - ref).max()
        worst = max(worst, dmax / vmax)
        assert dmax <= 5e-5 * vmax + 1e-6, (int(b), int(qh), dmax, vmax)
    return worst


@pytest.mark.parametrize("paged", [False, True])
def test_decode_attention_long_context(paged):
    """One sequence of 262,144 keys (the whole capacity), 8 KV heads, 32 query heads,
    bf16: the split-K path with all of its splits on one sequence, against the
    oracle on sampled query heads."""
    n, H, Hq, D, NL, layer = 262144, 8, 32, 128, 1, 0
    _say(f"decode attention long context: {n} keys, paged={paged}")
    g = torch.Generator(device=DEV)
    g.manual_seed(4200 + int(paged))
    rng = np.random.default_rng(4200 + int(paged))
    if paged:
        bs = 16
        n_blocks = n // bs
        table = rng.permutation(n_blocks).astype(np.int32)[None]
        shape = (NL, n_blocks, bs, H, D)
    else:
        shape = (1, NL, H, n, D)
    cache = prcr.Cache(torch.randn(shape, generator=g, device=DEV).to(torch.bfloat16),
                       torch.randn(shape, generator=g, device=DEV).to(torch.bfloat16),
                       to_dev(table) if paged else None)
    rope = prcr.Rope(D, (16, 24, 24), False, 1e6)
    q = torch.randn((1, Hq, D), generator=g, device=DEV).to(torch.bfloat16)
    q_pos = np.array([n + 40], np.int32)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q, to_dev(q_pos), to_dev(np.array([n], np.int32)),
                                err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    out = out.cpu().numpy()
    q_np = workloads.as_numpy_storage(q)
    rope_d = {"head_dim": D, "sections": (16, 24, 24), "interleaved": False, "theta": 1e6}
    for qh in rng.choice(Hq, 4, replace=False):
        kvh = int(qh) // (Hq // H)
        if paged:
            slots = np.arange(n)
            blk = torch.from_numpy(table[0, slots // bs].astype(np.int64)).to(DEV)
            off = torch.from_numpy((slots % bs).astype(np.int64)).to(DEV)
            k = workloads.as_numpy_storage(cache.k[layer, blk, off, kvh])
            v = workloads.as_numpy_storage(cache.v[layer, blk, off, kvh])
        else:
            k = workloads.as_numpy_storage(cache.k[0, layer, kvh])
            v = workloads.as_numpy_storage(cache.v[0, layer, kvh])
        one = {"paged": False, "s_max": n, "k": k[None, None, None], "v": v[None, None, None]}
        ref = oracle.decode_attention(rope_d, one, 0, q_np[:, qh:qh + 1], q_pos, np.array([n]),
                                      D ** -0.5, "bf16")[0, 0]
        vmax = np.abs(oracle.storage_to_f64(v, "bf16")).max()
        dmax = np.abs(out[0, qh] - ref).max()
        _say(f"  query head {int(qh)}: max |out - ref| = {dmax:.3g} (max |V| {vmax:.3g})")
        assert dmax <= 5e-5 * vmax + 1e-6, (int(qh), dmax, vmax)
    del cache
    torch.cuda.empty_cache()
