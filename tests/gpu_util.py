"""Shared helpers for the GPU parity tests: run the HIP path through the Python
binding (C ABI) and the CPU oracle on the same seeded inputs, then compare."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads

DEV = torch.device("cuda:0")


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def bf16_key(bits):
    """Monotone integer key of bf16 bit patterns (adjacent values differ by 1)."""
    b = np.asarray(bits).astype(np.uint16)
    return np.where(b & 0x8000, -(b & 0x7FFF).astype(np.int64), b.astype(np.int64))


def assert_keys_close(gpu, ref, dtype, what="keys"):
    """bf16: within 1 ulp of the oracle; f32: within 1e-5 relative, element by element."""
    gpu, ref = np.asarray(gpu), np.asarray(ref)
    if dtype == "bf16":
        d = np.abs(bf16_key(gpu) - bf16_key(ref))
        assert d.max(initial=0) <= 1, f"{what}: {int((d > 1).sum())} elements beyond 1 bf16 ulp"
        return int((d == 0).sum()), d.size
    r = ref.astype(np.float64)
    g = gpu.astype(np.float64)
    # NaN where the oracle has NaN; elsewhere |gpu - ref| <= 1e-5 |ref|, which asks
    # for equality where the oracle has a zero or an infinity.
    assert np.array_equal(np.isnan(g), np.isnan(r)), f"{what}: NaN positions differ"
    num = ~np.isnan(r)
    with np.errstate(invalid="ignore"):
        bad = num & ~((g == r) | (np.abs(g - r) <= 1e-5 * np.abs(r)))
    assert not bad.any(), f"{what}: {int(bad.sum())} elements beyond 1e-5 relative"
    return int(((gpu == ref) | (np.isnan(g) & np.isnan(r))).sum()), gpu.size


class Case:
    """One set of inputs in both forms (host numpy for the oracle, device tensors)."""

    def __init__(self, w: workloads.Workload, vals=None, seed_values=True):
        self.w = w
        if vals is None:
            vals = workloads.torch_values(w, "cpu")
        self.host = {k: workloads.as_numpy_storage(v) for k, v in vals.items()}
        self.dev_vals = {k: v.to(DEV) for k, v in vals.items()}

    def memory(self):
        w = self.w
        return prcr.Memory(self.dev_vals["mem_k"], self.dev_vals["mem_v"], to_dev(w.coords),
                           to_dev(w.n_visual))

    def cache(self):
        w = self.w
        return prcr.Cache(self.dev_vals["cache_k"], self.dev_vals["cache_v"],
                          to_dev(w.block_table) if w.paged else None)

    def rope(self):
        w = self.w
        return prcr.Rope(w.D, w.sections, w.interleaved, w.theta)

    def oracle_cache(self, k=None, v=None):
        w = self.w
        return {"paged": w.paged, "k": self.host["cache_k"] if k is None else k,
                "v": self.host["cache_v"] if v is None else v, "s_max": w.s_max,
                "block_table": w.block_table, "block_size": w.block_size,
                "max_blocks": w.max_blocks, "n_blocks": w.n_blocks}

    def oracle_mem(self):
        w = self.w
        return {"k": self.host["mem_k"], "v": self.host["mem_v"], "n_visual": w.n_visual,
                "dtype": w.dtype}


def run_both(case: Case, sel_off, sel_idx, p_txt, cache_len, mode="pcr", l_ext=2,
             stream=None, fused=False):
    """Reassign + rebind/inject on the GPU (two calls, or the single fused
    prcr_revisit launch) and in the oracle; returns (gpu, ref) dicts."""
    w = case.w
    mem, cache = case.memory(), case.cache()
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    so, si = to_dev(np.asarray(sel_off, np.int32)), to_dev(np.asarray(sel_idx, np.int32))
    pt, cl = to_dev(np.asarray(p_txt, np.int32)), to_dev(np.asarray(cache_len, np.int32))
    if fused:
        new_pos, next_pos, new_len, slots = prcr.revisit(case.rope(), mem, so, si, pt, cache, cl,
                                                         mode, l_ext, err=err, stream=stream)
    else:
        new_pos, next_pos = prcr.reassign_coords(mem, so, si, pt, mode, l_ext, err=err,
                                                 stream=stream)
        new_len, slots = prcr.rebind_inject(case.rope(), mem, so, si, new_pos, cache, cl, err=err,
                                            stream=stream)
    torch.cuda.synchronize()
    gpu = {"new_pos": new_pos.cpu().numpy(), "next_pos": next_pos.cpu().numpy(),
           "slot_mapping": slots.cpu().numpy(), "new_cache_len": new_len.cpu().numpy(),
           "k": workloads.as_numpy_storage(cache.k), "v": workloads.as_numpy_storage(cache.v),
           "err": int(err.item())}
    pos, nxt, err_r = oracle.reassign_batch(w.coords, w.n_visual, sel_off, sel_idx, p_txt, mode,
                                            l_ext)
    out = oracle.rebind_inject(w.rope(), case.oracle_mem(), sel_off, sel_idx, pos,
                               case.oracle_cache(), cache_len)
    ref = {"new_pos": pos, "next_pos": nxt, "slot_mapping": out["slot_mapping"],
           "new_cache_len": out["new_cache_len"], "k": out["k"], "v": out["v"],
           "err": err_r | out["err"]}
    # carry the updated oracle cache forward (multi-revisit workloads)
    case.host["cache_k"], case.host["cache_v"] = out["k"], out["v"]
    return gpu, ref


def new_row_mask(w, slot_mapping):
    """Boolean mask over the cache of the rows written at the given slots."""
    shape = workloads.cache_shape(w)[:-1]
    mask = np.zeros(shape, dtype=bool)
    for sid in np.asarray(slot_mapping):
        if sid < 0:
            continue
        if w.paged:
            mask[:, sid // w.block_size, sid % w.block_size] = True
        else:
            mask[sid // w.s_max, :, :, sid % w.s_max] = True
    return mask


def assert_parity(case, gpu, ref):
    """Bit-exact positions, slots, lengths, values and untouched keys; rebound keys
    within the key tolerance."""
    w = case.w
    assert gpu["err"] == ref["err"], (gpu["err"], ref["err"])
    assert np.array_equal(gpu["new_pos"], ref["new_pos"], equal_nan=True), "new_pos differs"
    assert np.array_equal(gpu["next_pos"], ref["next_pos"]), "next_pos differs"
    assert np.array_equal(gpu["slot_mapping"], ref["slot_mapping"]), "slot_mapping differs"
    assert np.array_equal(gpu["new_cache_len"], ref["new_cache_len"]), "cache_len differs"
    bits = lambda a: np.ascontiguousarray(a).view(np.uint8)   # NaN payloads compare too
    assert np.array_equal(bits(gpu["v"]), bits(ref["v"])), "value cache differs"
    mask = new_row_mask(w, ref["slot_mapping"])
    assert np.array_equal(bits(gpu["k"][~mask]), bits(ref["k"][~mask])), \
        "key cache changed outside new slots"
    return assert_keys_close(gpu["k"][mask], ref["k"][mask], w.dtype)
