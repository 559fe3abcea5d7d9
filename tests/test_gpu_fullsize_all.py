"""Every entry of the full-size rebinding calls against the oracle.

Workloads 3 (32 sequences, contiguous) and 5 (64 sequences, paged) at their full
sizes, in the launch configuration bench.py times, and the bench's other sections
(workload 3's TP-8 shard, 8,192 slots per sequence, 1-D rotary positions, key-only
memories, workload 4's four successive video revisits), through the C-ABI entry
points:

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


def _every_entry(w, mem, cache, rope, sel_off, sel_idx, p_txt, cache_len, v_slot=None):
    """One reassign + rebind call, every output checked as described above; with
    v_slot (a key-only memory) the values come from those slots of the same cache.
    Returns (next positions, new lengths) from the oracle."""
    p_txt = np.asarray(p_txt, np.int64)
    cache_len = np.asarray(cache_len, np.int64)
    k0, v0 = cache.k.clone(), cache.v.clone()
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    so, si = to_dev(np.asarray(sel_off, np.int32)), to_dev(np.asarray(sel_idx, np.int32))
    new_pos, next_pos = prcr.reassign_coords(mem, so, si, to_dev(p_txt.astype(np.int32)), "pcr", 2,
                                             err=err)
    new_len, slots = prcr.rebind_inject(rope, mem, so, si, new_pos, cache,
                                        to_dev(cache_len.astype(np.int32)), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0

    pos_o, next_o, err_o = oracle.reassign_batch(w.coords, w.n_visual, sel_off, sel_idx, p_txt)
    assert err_o == 0
    assert np.array_equal(new_pos.cpu().numpy(), pos_o), "positions differ"
    assert np.array_equal(next_pos.cpu().numpy(), next_o), "next positions differ"
    oc = {"paged": w.paged, "s_max": w.s_max, "block_table": w.block_table,
          "block_size": w.block_size, "max_blocks": w.max_blocks, "n_blocks": w.n_blocks}
    total_k = len(sel_idx)
    tok_b_np = np.repeat(np.arange(w.B), np.diff(sel_off))
    j_np = np.arange(total_k) - np.asarray(sel_off)[tok_b_np]
    exp_slots = np.array([oracle.slot_of(oc, int(b), int(cache_len[b]) + int(j))[0]
                          for b, j in zip(tok_b_np, j_np)], np.int64)
    assert np.array_equal(slots.cpu().numpy(), exp_slots), "slot mapping differs"
    exp_len = cache_len + np.diff(sel_off)
    assert np.array_equal(new_len.cpu().numpy(), exp_len), "cache lengths differ"

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

    # every value row, bit-exact against its source row (the memory, or for a key-only
    # memory the value slot's rows as they were before the call)
    tok_b = torch.from_numpy(tok_b_np).to(DEV)
    tok_m = si.long()
    if v_slot is None:
        want_v = mem.v[tok_b, tok_m]
    else:
        src = np.array([oracle.slot_of(oc, int(b), int(v_slot[b, m]))[0]
                        for b, m in zip(tok_b_np, sel_idx)], np.int64)
        want_v = _rows_at(w, v0, torch.from_numpy(src).to(DEV))
    assert torch.equal(_rows_at(w, cache.v, sl).view(torch.int16), want_v.view(torch.int16)), \
        "a value row differs"
    del k0, v0, expected, want_v
    torch.cuda.empty_cache()

    # every key element against the oracle's rebinding, 1 bf16 ulp
    raw = workloads.as_numpy_storage(mem.k[tok_b, tok_m])
    got = workloads.as_numpy_storage(_rows_at(w, cache.k, sl))
    tasks = [(w.rope(), raw[t0:t0 + CHUNK], w.dtype, pos_o[t0:t0 + CHUNK, None, None, :])
             for t0 in range(0, total_k, CHUNK)]
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
    return next_o, exp_len


def _prepare(w, key_only=False):
    vals = workloads.torch_values(w, DEV)
    v_slot = None
    if key_only:
        del vals["mem_v"]
        v_slot = workloads.value_slots(w)
        mem = prcr.Memory(vals["mem_k"], None, to_dev(w.coords), to_dev(w.n_visual), to_dev(v_slot))
    else:
        mem = prcr.Memory(vals["mem_k"], vals["mem_v"], to_dev(w.coords), to_dev(w.n_visual))
    cache = prcr.Cache(vals["cache_k"], vals["cache_v"], to_dev(w.block_table) if w.paged else None)
    rope = prcr.Rope(w.D, w.sections, w.interleaved, w.theta)
    return mem, cache, rope, v_slot


def _variant(name):
    if name == "workload3":
        return workloads.make(3, "full")
    if name == "workload5":
        return workloads.make(5, "full")
    if name == "workload3-tp8-shard":
        return workloads.tp_shard(workloads.make(3, "full"), 8)
    if name == "workload3-8192-slots":
        return workloads.with_capacity(workloads.make(3, "full"), 8192)
    if name == "workload3-1d-rotary":
        return workloads.one_d(workloads.make(3, "full"))
    raise ValueError(name)


@pytest.mark.parametrize("name", ["workload3", "workload5", "workload3-tp8-shard",
                                  "workload3-8192-slots", "workload3-1d-rotary"])
def test_full_size_every_entry(name):
    w = _variant(name)
    _say(f"{name} full, every entry: B={w.B} NL={w.NL} H={w.H} K={w.total_k} "
         f"entries={w.entries()}")
    mem, cache, rope, _ = _prepare(w)
    _every_entry(w, mem, cache, rope, w.sel_off, w.sel_idx, w.p_txt, w.cache_len)
    del mem, cache
    torch.cuda.empty_cache()


@pytest.mark.parametrize("cfg", [3, 5])
def test_full_size_every_entry_key_only_memory(cfg):
    w = workloads.make(cfg, "full")
    _say(f"workload {cfg} full, key-only memory, every entry")
    mem, cache, rope, v_slot = _prepare(w, key_only=True)
    _every_entry(w, mem, cache, rope, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, v_slot)
    del mem, cache
    torch.cuda.empty_cache()


def test_full_size_every_entry_video_four_revisits():
    """Workload 4: four successive revisits of 1024 tokens into the same caches, 32
    text tokens decoded in between; each revisit checked in full."""
    w = workloads.make(4, "full")
    _say(f"workload 4 full: B={w.B} NL={w.NL}, 4 revisits of 1024 tokens, every entry")
    mem, cache, rope, _ = _prepare(w)
    lens = w.cache_len.astype(np.int64)
    p_txt = w.p_txt.astype(np.int64)
    for r, (so, si) in enumerate(w.revisits):
        nxt, new_len = _every_entry(w, mem, cache, rope, so, si, p_txt, lens)
        lens = new_len + w.decode_between
        p_txt = nxt + w.decode_between - 1
    assert (lens <= w.s_max).all()
    del mem, cache
    torch.cuda.empty_cache()
