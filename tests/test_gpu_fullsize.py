"""Full-size parity in the launch configuration that bench.py times.

Workloads 3 (32 sequences, contiguous), 4 (video, four successive revisits) and 5
(64 sequences, paged) at their full sizes, through the same C-ABI entry points:

* positions, next text positions, slot mapping and new cache lengths: every token,
  bit-exact against the oracle;
* keys and values: a random sample of (token, layer, head) entries against the
  oracle's row-by-row rebinding (1 bf16 ulp for keys, bit-exact values);
* properties that hold at any size, over every entry on the device: each value row
  equals its memory row bit for bit, and each rotated key pair keeps its norm within
  bf16 rounding;
* a random sample of cache rows outside the new slots is unchanged.

The key-only memory runs at workloads 3 and 5 too: every injected value row equals
the cache row at the token's value slot, keys as above.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, bf16_key, to_dev

pytestmark = pytest.mark.gpu
N_SAMPLE = 3000


def _say(msg):
    print(msg, flush=True)


def _oracle_cache(w):
    return {"paged": w.paged, "s_max": w.s_max, "block_table": w.block_table,
            "block_size": w.block_size, "max_blocks": w.max_blocks, "n_blocks": w.n_blocks}


def _rows_at(w, cache_t, slot_ids):
    """Cache rows [T, NL, H, D] at global slot ids (device tensor of int64)."""
    if w.paged:
        return cache_t[:, slot_ids // w.block_size, slot_ids % w.block_size].permute(1, 0, 2, 3)
    return cache_t[slot_ids // w.s_max, :, :, slot_ids % w.s_max]


def _untouched_sample(w, new_slots, rng, n=N_SAMPLE):
    """Random cache rows (index tuples) that are not new slots."""
    new = set(int(s) for s in new_slots)
    cap = w.n_blocks * w.block_size if w.paged else w.B * w.s_max
    picks = []
    while len(picks) < n:
        sid = int(rng.integers(0, cap))
        if sid in new:
            continue
        l, h = int(rng.integers(0, w.NL)), int(rng.integers(0, w.H))
        if w.paged:
            picks.append((l, sid // w.block_size, sid % w.block_size, h))
        else:
            picks.append((sid // w.s_max, l, h, sid % w.s_max))
    return tuple(torch.tensor(np.array(c), device=DEV) for c in zip(*picks))


def _check_call(w, mem, cache, rope, sel_off, sel_idx, p_txt, cache_len, rng, v_slot=None):
    """One reassign + rebind call at full size, checked as described above.  With
    v_slot (a key-only memory) the values come from those cache slots."""
    B = w.B
    oc = _oracle_cache(w)
    exp_slots = np.full(len(sel_idx), -1, np.int64)
    for b in range(B):
        for j in range(int(sel_off[b + 1] - sel_off[b])):
            exp_slots[sel_off[b] + j] = oracle.slot_of(oc, b, int(cache_len[b]) + j)[0]
    untouched = _untouched_sample(w, exp_slots, rng)
    before_k, before_v = cache.k[untouched].clone(), cache.v[untouched].clone()

    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    so, si = to_dev(sel_off), to_dev(sel_idx)
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
    assert np.array_equal(slots.cpu().numpy(), exp_slots), "slot mapping differs"
    exp_len = cache_len + np.diff(sel_off)
    assert np.array_equal(new_len.cpu().numpy(), exp_len), "cache lengths differ"

    # every entry: values bit-exact, key pair norms kept
    tok_b = torch.from_numpy(np.repeat(np.arange(B), np.diff(sel_off))).to(DEV)
    tok_m = si.long()
    sl = slots
    got_v = _rows_at(w, cache.v, sl)
    if v_slot is None:
        want_v = mem.v[tok_b, tok_m]
    else:
        tb = np.repeat(np.arange(B), np.diff(sel_off))
        src = np.array([oracle.slot_of(oc, int(b), int(v_slot[b, m]))[0]
                        for b, m in zip(tb, sel_idx)], np.int64)
        want_v = _rows_at(w, cache.v, torch.from_numpy(src).to(DEV))
    assert torch.equal(got_v.view(torch.int16), want_v.view(torch.int16)), \
        "a value row differs from its source row"
    del got_v, want_v
    P = w.D // 2
    for t0 in range(0, len(sel_idx), 2048):
        t1 = min(len(sel_idx), t0 + 2048)
        x = mem.k[tok_b[t0:t1], tok_m[t0:t1]].float()
        y = _rows_at(w, cache.k, sl[t0:t1]).float()
        nx = x[..., :P] ** 2 + x[..., P:] ** 2
        ny = y[..., :P] ** 2 + y[..., P:] ** 2
        assert bool(((ny - nx).abs() <= 2.0 ** -6 * nx + 1e-30).all()), "a key pair changed norm"

    # sampled entries against the oracle's row-by-row rebinding
    g = rng.integers(0, len(sel_idx), N_SAMPLE)
    l = rng.integers(0, w.NL, N_SAMPLE)
    h = rng.integers(0, w.H, N_SAMPLE)
    b = np.repeat(np.arange(B), np.diff(sel_off))[g]
    m = sel_idx[g]
    gt = lambda a: torch.from_numpy(np.asarray(a, np.int64)).to(DEV)
    raw_k = workloads.as_numpy_storage(mem.k[gt(b), gt(m), gt(l), gt(h)])
    sid = exp_slots[g]
    if w.paged:
        idx = (gt(l), gt(sid // w.block_size), gt(sid % w.block_size), gt(h))
    else:
        idx = (gt(sid // w.s_max), gt(l), gt(h), gt(sid % w.s_max))
    got_k = workloads.as_numpy_storage(cache.k[idx])
    got_v = workloads.as_numpy_storage(cache.v[idx])
    ref_k = oracle.rebind_row(w.rope(), raw_k, w.dtype, pos_o[g])
    d = np.abs(bf16_key(got_k) - bf16_key(ref_k))
    assert d.max() <= 1, f"{int((d > 1).sum())} sampled key elements beyond 1 bf16 ulp"
    if v_slot is None:
        assert np.array_equal(got_v, workloads.as_numpy_storage(mem.v[gt(b), gt(m), gt(l), gt(h)]))

    # rows outside the new slots are unchanged
    assert torch.equal(cache.k[untouched].view(torch.int16), before_k.view(torch.int16)), \
        "a key row outside the new slots changed"
    assert torch.equal(cache.v[untouched].view(torch.int16), before_v.view(torch.int16)), \
        "a value row outside the new slots changed"
    return int((d == 0).sum()), d.size, next_o, exp_len


def _prepare(w):
    vals = workloads.torch_values(w, DEV)
    mem = prcr.Memory(vals["mem_k"], vals["mem_v"], to_dev(w.coords), to_dev(w.n_visual))
    cache = prcr.Cache(vals["cache_k"], vals["cache_v"], to_dev(w.block_table) if w.paged else None)
    rope = prcr.Rope(w.D, w.sections, w.interleaved, w.theta)
    return mem, cache, rope


@pytest.mark.parametrize("cfg", [3, 5])
def test_full_size_workload(cfg):
    w = workloads.make(cfg, "full")
    _say(f"workload {cfg} full: B={w.B} NL={w.NL} H={w.H} K={w.total_k} entries={w.entries()}")
    mem, cache, rope = _prepare(w)
    rng = np.random.default_rng(cfg)
    exact, n, _, _ = _check_call(w, mem, cache, rope, w.sel_off, w.sel_idx, w.p_txt.astype(np.int64),
                                 w.cache_len.astype(np.int64), rng)
    _say(f"  sampled keys bit-exact {exact}/{n}")
    del mem, cache
    torch.cuda.empty_cache()


def test_full_size_video_four_revisits():
    w = workloads.make(4, "full")
    _say(f"workload 4 full: B={w.B} NL={w.NL}, 4 revisits of 1024 tokens")
    mem, cache, rope = _prepare(w)
    rng = np.random.default_rng(4)
    lens = w.cache_len.astype(np.int64)
    p_txt = w.p_txt.astype(np.int64)
    for r, (so, si) in enumerate(w.revisits):
        exact, n, nxt, new_len = _check_call(w, mem, cache, rope, so, si, p_txt, lens, rng)
        _say(f"  revisit {r}: sampled keys bit-exact {exact}/{n}")
        lens = new_len + w.decode_between
        p_txt = nxt + w.decode_between - 1
    assert (lens <= w.s_max).all()
    del mem, cache
    torch.cuda.empty_cache()


@pytest.mark.parametrize("cfg", [3, 5])
def test_full_size_key_only_memory(cfg):
    w = workloads.make(cfg, "full")
    _say(f"workload {cfg} full, key-only memory")
    vals = workloads.torch_values(w, DEV)
    del vals["mem_v"]
    v_slot = workloads.value_slots(w)
    mem = prcr.Memory(vals["mem_k"], None, to_dev(w.coords), to_dev(w.n_visual), to_dev(v_slot))
    cache = prcr.Cache(vals["cache_k"], vals["cache_v"], to_dev(w.block_table) if w.paged else None)
    rope = prcr.Rope(w.D, w.sections, w.interleaved, w.theta)
    rng = np.random.default_rng(cfg + 50)
    exact, n, _, _ = _check_call(w, mem, cache, rope, w.sel_off, w.sel_idx, w.p_txt.astype(np.int64),
                                 w.cache_len.astype(np.int64), rng, v_slot=v_slot)
    _say(f"  sampled keys bit-exact {exact}/{n}")
    del mem, cache, vals
    torch.cuda.empty_cache()


def test_full_size_tp8_shard():
    """One GPU's share of workload 3 at 8-way KV-head parallelism: 1 KV head, so each
    (token, layer) row is a single 256-byte row (the small-row regime)."""
    w = workloads.tp_shard(workloads.make(3, "full"), 8)
    _say(f"workload 3 full, TP-8 shard: H={w.H} entries={w.entries()}")
    mem, cache, rope = _prepare(w)
    rng = np.random.default_rng(38)
    exact, n, _, _ = _check_call(w, mem, cache, rope, w.sel_off, w.sel_idx, w.p_txt.astype(np.int64),
                                 w.cache_len.astype(np.int64), rng)
    _say(f"  sampled keys bit-exact {exact}/{n}")
    del mem, cache
    torch.cuda.empty_cache()


def test_full_size_power_of_two_capacity():
    """Workload 3 with 8192 slots per sequence (2 MiB rows per layer and head), the
    cache shape that bench.py times beside the tight one."""
    w = workloads.with_capacity(workloads.make(3, "full"), 8192)
    _say(f"workload 3 full, s_max {w.s_max}")
    mem, cache, rope = _prepare(w)
    rng = np.random.default_rng(39)
    exact, n, _, _ = _check_call(w, mem, cache, rope, w.sel_off, w.sel_idx, w.p_txt.astype(np.int64),
                                 w.cache_len.astype(np.int64), rng)
    _say(f"  sampled keys bit-exact {exact}/{n}")
    del mem, cache
    torch.cuda.empty_cache()


def test_full_size_one_d_rotary():
    """Workload 3's shapes with 1-D rotary positions (every pair on t, each visual
    token's position in t): the form of InternVL3.5's language model."""
    w = workloads.one_d(workloads.make(3, "full"))
    _say(f"workload 3 full, 1-D rotary {w.sections}")
    mem, cache, rope = _prepare(w)
    rng = np.random.default_rng(40)
    exact, n, _, _ = _check_call(w, mem, cache, rope, w.sel_off, w.sel_idx, w.p_txt.astype(np.int64),
                                 w.cache_len.astype(np.int64), rng)
    _say(f"  sampled keys bit-exact {exact}/{n}")
    del mem, cache
    torch.cuda.empty_cache()
