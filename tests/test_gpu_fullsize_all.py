"""Every entry of the full-size rebinding calls against the oracle.

Workloads 3 (32 sequences, contiguous) and 5 (64 sequences, paged) at their full
sizes, in the launch configuration bench.py times, through the C-ABI entry points:

* positions, next text positions, slot mapping and new cache lengths: bit-exact;
* every rebound key element (Eq. (12)): within 1 bf16 ulp of the oracle's rebinding
  of the raw memory row at the oracle's positions, computed in float64 by the oracle
  itself, chunk by chunk in a pool of worker processes;
* every value row (Eq. (12)): bit-exact against its memory row;
* every cache byte outside the new slots (Eq. (13)): unchanged, compared on the GPU
  against a copy of the whole cache taken before the call.
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
CHUNK = 256          # tokens per oracle task


def _say(msg):
    print(msg, flush=True)


def _rows_at(w, cache_t, slot_ids):
    """Cache rows [T, NL, H, D] at global slot ids (device tensor of int64)."""
    if w.paged:
        return cache_t[:, slot_ids // w.block_size, slot_ids % w.block_size].permute(1, 0, 2, 3)
    return cache_t[slot_ids // w.s_max, :, :, slot_ids % w.s_max]


@pytest.mark.parametrize("cfg", [3, 5])
def test_full_size_every_entry(cfg):
    w = workloads.make(cfg, "full")
    _say(f"workload {cfg} full, every entry: B={w.B} NL={w.NL} H={w.H} K={w.total_k} "
         f"entries={w.entries()}")
    vals = workloads.torch_values(w, DEV)
    mem = prcr.Memory(vals["mem_k"], vals["mem_v"], to_dev(w.coords), to_dev(w.n_visual))
    cache = prcr.Cache(vals["cache_k"], vals["cache_v"], to_dev(w.block_table) if w.paged else None)
    rope = prcr.Rope(w.D, w.sections, w.interleaved, w.theta)
    k0, v0 = cache.k.clone(), cache.v.clone()

    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    so, si = to_dev(w.sel_off), to_dev(w.sel_idx)
    new_pos, next_pos = prcr.reassign_coords(mem, so, si, to_dev(w.p_txt), "pcr", 2, err=err)
    new_len, slots = prcr.rebind_inject(rope, mem, so, si, new_pos, cache, to_dev(w.cache_len),
                                        err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0

    pos_o, next_o, err_o = oracle.reassign_batch(w.coords, w.n_visual, w.sel_off, w.sel_idx,
                                                 w.p_txt)
    assert err_o == 0
    assert np.array_equal(new_pos.cpu().numpy(), pos_o), "positions differ"
    assert np.array_equal(next_pos.cpu().numpy(), next_o), "next positions differ"
    oc = {"paged": w.paged, "s_max": w.s_max, "block_table": w.block_table,
          "block_size": w.block_size, "max_blocks": w.max_blocks, "n_blocks": w.n_blocks}
    tok_b_np = np.repeat(np.arange(w.B), np.diff(w.sel_off))
    j_np = np.arange(w.total_k) - w.sel_off[tok_b_np]
    exp_slots = np.array([oracle.slot_of(oc, int(b), int(w.cache_len[b]) + int(j))[0]
                          for b, j in zip(tok_b_np, j_np)], np.int64)
    assert np.array_equal(slots.cpu().numpy(), exp_slots), "slot mapping differs"
    assert np.array_equal(new_len.cpu().numpy(), w.cache_len + np.diff(w.sel_off)), \
        "cache lengths differ"

    # every byte outside the new slots: rows that changed must all be new rows
    sl = torch.from_numpy(exp_slots).to(DEV)
    expected = torch.zeros(cache.k.shape[:-1], dtype=torch.bool, device=DEV)
    if w.paged:
        expected[:, sl // w.block_size, sl % w.block_size] = True
    else:
        expected[sl // w.s_max, :, :, sl % w.s_max] = True
    for now, before, name in ((cache.k, k0, "key"), (cache.v, v0, "value")):
        changed = (now.view(torch.int16) != before.view(torch.int16)).any(-1)
        assert not bool((changed & ~expected).any()), f"a {name} row outside the new slots changed"
        del changed
    del k0, v0, expected
    torch.cuda.empty_cache()

    # every value row, bit-exact against its memory row
    tok_b = torch.from_numpy(tok_b_np).to(DEV)
    tok_m = si.long()
    assert torch.equal(_rows_at(w, cache.v, sl).view(torch.int16),
                       mem.v[tok_b, tok_m].view(torch.int16)), "a value row differs"

    # every key element against the oracle's rebinding, 1 bf16 ulp
    raw = workloads.as_numpy_storage(mem.k[tok_b, tok_m])
    got = workloads.as_numpy_storage(_rows_at(w, cache.k, sl))
    tasks = [(w.rope(), raw[t0:t0 + CHUNK], w.dtype, pos_o[t0:t0 + CHUNK, None, None, :])
             for t0 in range(0, w.total_k, CHUNK)]
    workers = max(1, min(8, len(os.sched_getaffinity(0))))
    _say(f"  oracle over {len(tasks)} chunks of {CHUNK} tokens, {workers} worker processes")
    with mp.get_context("spawn").Pool(workers) as pool:
        refs = pool.starmap(oracle.rebind_row, tasks)
    exact = worst = 0
    for i, ref in enumerate(refs):
        t0 = i * CHUNK
        d = np.abs(bf16_key(got[t0:t0 + CHUNK]) - bf16_key(ref))
        worst = max(worst, int(d.max()))
        exact += int((d == 0).sum())
    assert worst <= 1, f"a key element is {worst} bf16 ulp from the oracle"
    _say(f"  keys: {exact}/{got.size} bit-exact, the rest within 1 bf16 ulp")
    del mem, cache, vals
    torch.cuda.empty_cache()
