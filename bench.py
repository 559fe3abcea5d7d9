"""Throughput of the PRCR rebinding hot path on one MI355X.

A step is one pass of the whole path over one batch: position reassignment
(prcr_reassign_coords) followed by the fused gather -> M-RoPE rebinding -> inject
kernel (prcr_rebind_inject), both launched through the C ABI on one stream, with
every input already resident in HBM.  Each step re-injects into the same slots,
so every step does identical work.

Default workload: 32 sequences x 256 selected tokens, 36 layers x 8 KV heads,
head_dim 128, bf16, interleaved M-RoPE (theta 5e6), contiguous caches of 4256
slots per sequence.  The paged workload (64 sequences x 512 tokens, 28 layers x 4
heads, block size 16) is measured in the same run and reported under "secondary".
Further sections time the same path under SHIFT reassignment, with 8192 cache
slots per sequence (power_of_two_capacity: 2 MiB cache rows, which the memory
channels absorb faster), with a key-only memory, with 1-D rotary positions (the
rotary form of InternVL3.5, the paper's other model family), at one GPU's share of 8-way
KV-head parallelism, over four video revisits and at small selections, and time
the prefill capture (at 36 x 8 and 28 x 4 KV heads), raw-memory store and decode
attention kernels.

Prints one JSON line.  `value` = rebound (sequence, token, layer, KV-head)
entries per second over the timed steps.  `roofline` is for the dominant kernel
(prcr_rebind_inject): algorithmic bytes per launch (4 * head_dim * 2 bytes per
entry: read K, read V, write K, write V) divided by its mean launch time from HIP
events recorded around each launch on its own stream.  `cpu_baseline` is the
CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
_CSRC = "paper_2606_26631_amd/csrc/"
_COMMON = [_CSRC + f for f in ("rotary.h", "prcr_internal.h")]
# Sources each measured kernel and its launch are built from (the host argument
# checks are not among them); a committed counter summary applies only while
# their hash is the one it was taken on.
KERNEL_SOURCES = {
    "rebind": [_CSRC + "rebind.hip", _CSRC + "reassign.hip", _CSRC + "positions.h"] + _COMMON,
    "prefill": [_CSRC + "prefill.hip"] + _COMMON,
    "decode": [_CSRC + "decode.hip"] + _COMMON,
    "store": [_CSRC + "store_raw.hip"] + _COMMON,
}


def kernel_source_hash(kind: str = "rebind") -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kind]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def describe(w) -> dict:
    cfg = {"workload": f"workload {w.cfg} ({w.name})", "sequences": w.B,
           "selected_tokens": w.total_k, "layers": w.NL, "kv_heads": w.H, "head_dim": w.D,
           "storage": w.dtype, "rope": ("interleaved" if w.interleaved else "sectioned")
           + f" {list(w.sections)} theta {w.theta:g}", "mode": "pcr", "l_ext": 2,
           "cache": (f"paged, block {w.block_size}, {w.n_blocks} blocks" if w.paged
                     else f"contiguous, s_max {w.s_max}"),
           "entries_per_step": w.entries(), "algorithmic_bytes_per_step": w.algorithmic_bytes()}
    return cfg


def load_traffic(name: str, kind: str):
    """HBM bytes per launch from a committed rocprofv3 counter summary
    (profiles/counters_<name>.json), if it was taken on the current sources of
    that kernel; else None."""
    path = os.path.join(ROOT, "profiles", f"counters_{name}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        c = json.load(f)
    if c.get("kernel_source_hash") != kernel_source_hash(kind):
        return None
    return c.get("traffic_bytes_per_launch")


class Prepared:
    def __init__(self, w, dev, key_only=False, mode="pcr"):
        import numpy as np
        import torch

        import paper_2606_26631_amd as prcr
        import workloads
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        self.w = w
        vals = workloads.torch_values(w, dev)
        if key_only:
            del vals["mem_v"]
            self.mem = prcr.Memory(vals["mem_k"], None, t(w.coords), t(w.n_visual),
                                   t(workloads.value_slots(w)))
        else:
            self.mem = prcr.Memory(vals["mem_k"], vals["mem_v"], t(w.coords), t(w.n_visual))
        self.cache = prcr.Cache(vals["cache_k"], vals["cache_v"], t(w.block_table) if w.paged else None)
        self.rope = prcr.Rope(w.D, w.sections, w.interleaved, w.theta)
        self.sel_off, self.sel_idx = t(w.sel_off), t(w.sel_idx)
        self.p_txt, self.cache_len = t(w.p_txt), t(w.cache_len)
        self.new_pos = torch.empty((w.total_k, 3), dtype=torch.float64, device=dev)
        self.next_pos = torch.empty((w.B,), dtype=torch.int32, device=dev)
        self.new_len = torch.empty((w.B,), dtype=torch.int32, device=dev)
        self.slots = torch.empty((w.total_k,), dtype=torch.int64, device=dev)
        self.err = torch.zeros(1, dtype=torch.int32, device=dev)
        self.mode = mode

    def reassign(self, stream):
        import paper_2606_26631_amd as prcr
        prcr.reassign_coords(self.mem, self.sel_off, self.sel_idx, self.p_txt, self.mode, 2,
                             self.new_pos, self.next_pos, self.err, stream)

    def rebind(self, stream):
        import paper_2606_26631_amd as prcr
        prcr.rebind_inject(self.rope, self.mem, self.sel_off, self.sel_idx, self.new_pos,
                           self.cache, self.cache_len, self.new_len, self.slots, self.err, stream)


def measure(w, steps, warmup, dev, key_only=False, mode="pcr", with_pattern=False):
    import torch
    p = Prepared(w, dev, key_only, mode)
    s = torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        for _ in range(warmup):
            p.reassign(s)
            p.rebind(s)
        s.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
                torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(s)
        for a, b, c in evs:
            a.record(s)
            p.reassign(s)
            b.record(s)
            p.rebind(s)
            c.record(s)
        t1.record(s)
        torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    rebind_ms = [b.elapsed_time(c) for a, b, c in evs]
    reassign_ms = [a.elapsed_time(b) for a, b, c in evs]
    err = int(p.err.item())
    if err != 0:
        raise RuntimeError(f"device reported data error bits {err}")
    # The same addresses copied with no arithmetic, on the same arrays (where the
    # arrays land in memory moves both alike), after the timed steps.
    pattern_ms = pattern_copy(p, steps, warmup)[1] if with_pattern else None
    del p
    torch.cuda.empty_cache()
    if with_pattern:
        return total_ms, rebind_ms, reassign_ms, pattern_ms
    return total_ms, rebind_ms, reassign_ms


_COPYREF = None


def copyref_lib():
    """The reference copy kernels (libprcr_copyref.so, built next to libprcr.so)."""
    global _COPYREF
    if _COPYREF is None:
        import ctypes
        path = os.path.join(ROOT, "paper_2606_26631_amd", "libprcr_copyref.so")
        if not os.path.exists(path):
            raise ImportError(f"{path} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(path)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.prcr_copyref_stream.restype = ctypes.c_int
        L.prcr_copyref_stream.argtypes = [vp, vp, i64, i64, vp]
        L.prcr_copyref_decode_read.restype = ctypes.c_int
        L.prcr_copyref_decode_read.argtypes = [vp, vp, vp, vp, vp] + [i32] * 10 + [vp]
        L.prcr_copyref_prefill.restype = ctypes.c_int
        L.prcr_copyref_prefill.argtypes = [vp] * 8 + [i32] * 7 + [vp]
        L.prcr_copyref_pattern.restype = ctypes.c_int
        L.prcr_copyref_pattern.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i64, vp]
        _COPYREF = L
    return _COPYREF


def _timed(fn, stream, steps, warmup):
    """Mean and per-launch times (ms) of fn() from HIP events on `stream`."""
    import torch
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for _ in range(warmup):
            fn()
        evs = []
        for _ in range(steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            evs.append((a, b))
        torch.cuda.synchronize()
    ms = [a.elapsed_time(b) for a, b in evs]
    return sum(ms) / len(ms), ms


def copy_reference(dev, nbytes=1 << 31, steps=20, warmup=3):
    """A plain streaming copy of nbytes (each workgroup owns one contiguous 16 KB
    chunk, 16-byte non-temporal accesses): the attainable read + write rate of this
    GPU.  Mean of `steps` launches, as for the rebind."""
    import torch
    L = copyref_lib()
    src = torch.ones(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    s = torch.cuda.Stream(device=dev)

    def run():
        if L.prcr_copyref_stream(src.data_ptr(), dst.data_ptr(), nbytes, 16384, s.cuda_stream) != 0:
            raise RuntimeError("prcr_copyref_stream failed")

    mean_ms, ms = _timed(run, s, steps, warmup)
    ok = bool(torch.equal(dst[:: 1 << 20], src[:: 1 << 20]))
    del src, dst
    torch.cuda.empty_cache()
    if not ok:
        raise RuntimeError("the reference copy did not copy")
    return {"kernel": "copyref stream_kernel (16 KB per workgroup)", "bytes_read": nbytes,
            "bytes_written": nbytes, "mean_launch_us": round(mean_ms * 1e3, 2),
            "achieved": round(2 * nbytes / (mean_ms / 1e3) / 1e9, 1), "unit": "GB/s",
            "frac": round(2 * nbytes / (mean_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}


def rebind_rows_per_wave(total_k, rows_total, k_step=16, rows_target=72, min_waves=4096):
    """(layer, head) rows of one token per wave in the rebinding kernel's launch for
    bf16 / head_dim 128 (16-row load batches): about 72, in whole batches, fewer on
    small problems so that at least 4096 waves run per array."""
    rows_all = total_k * rows_total
    target = rows_target
    if rows_all < target * min_waves:
        target = rows_all // min_waves
    target = max(k_step, (target + k_step - 1) // k_step * k_step)
    groups = (rows_total + target - 1) // target
    per = (rows_total + groups - 1) // groups
    return (per + k_step - 1) // k_step * k_step


def pattern_offsets(w):
    """Per-token byte offsets of the rebind's reads and writes for workload w
    (bf16, head_dim 128): token g's first row in the memory, its row 0 in the cache,
    and the cache's row-group rule.  Returns (src_tok, dst_tok, group_log2,
    group_stride, rows_total, rows_per_wave)."""
    import numpy as np
    if w.dtype != "bf16" or w.D != 128:
        raise ValueError("the pattern copy is built for bf16 rows of head_dim 128")
    row = w.D * 2
    rows_total = w.NL * w.H
    so = np.asarray(w.sel_off, np.int64)
    b = np.repeat(np.arange(w.B, dtype=np.int64), np.diff(so))
    j = np.arange(w.total_k, dtype=np.int64) - so[b]
    m = np.asarray(w.sel_idx, np.int64)
    slot = np.asarray(w.cache_len, np.int64)[b] + j
    src_tok = (b * w.M_max + m) * rows_total * row
    if w.paged:
        if w.H & (w.H - 1):
            raise ValueError("paged pattern copy needs a power-of-two KV-head count")
        blk = np.asarray(w.block_table, np.int64)[b, slot // w.block_size]
        dst_tok = (blk * w.block_size + slot % w.block_size) * w.H * row
        group_log2 = int(w.H).bit_length() - 1
        group_stride = w.n_blocks * w.block_size * w.H * row
    else:
        dst_tok = (b * rows_total * w.s_max + slot) * row
        group_log2, group_stride = 0, w.s_max * row
    # every access stays inside the arrays
    mem_bytes = w.B * w.M_max * rows_total * row
    r_last = rows_total - 1
    last_dst = (r_last >> group_log2) * group_stride + (r_last & ((1 << group_log2) - 1)) * row
    cache_bytes = int(np.prod(workloads_cache_shape(w))) * 2
    assert src_tok.min() >= 0 and int(src_tok.max()) + rows_total * row <= mem_bytes
    assert dst_tok.min() >= 0 and int(dst_tok.max()) + last_dst + row <= cache_bytes
    return (src_tok, dst_tok, group_log2, group_stride, rows_total,
            rebind_rows_per_wave(w.total_k, rows_total))


def workloads_cache_shape(w):
    import workloads
    return workloads.cache_shape(w)


def pattern_copy(p, steps, warmup):
    """The rebind's access pattern on the prepared arrays (memory -> cache, keys then
    values) with no arithmetic: mean and per-launch times (ms)."""
    import torch
    L = copyref_lib()
    src_tok, dst_tok, lg, gstride, rows_total, rpw = pattern_offsets(p.w)
    dev = p.cache.k.device
    st, dt = torch.from_numpy(src_tok).to(dev), torch.from_numpy(dst_tok).to(dev)
    s = torch.cuda.Stream(device=dev)

    def run():
        rc = L.prcr_copyref_pattern(p.mem.k.data_ptr(), p.mem.v.data_ptr(), p.cache.k.data_ptr(),
                                    p.cache.v.data_ptr(), st.data_ptr(), dt.data_ptr(),
                                    p.w.total_k, rows_total, rpw, lg, gstride, s.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"prcr_copyref_pattern failed ({rc})")

    return _timed(run, s, steps, warmup)


def small_k_latency(dev, reps=200):
    """Per-revisit latency at Table 3's operating points (one sequence, K = 32 and
    128 of 768 visual tokens, Qwen3-VL-8B and -32B cache shapes), for the two-call
    path (prcr_reassign_coords + prcr_rebind_inject) and the single fused launch
    (prcr_revisit): once as a host loop through the Python binding, once as device
    time per revisit with 50 revisits captured in one HIP graph."""
    import torch

    import paper_2606_26631_amd as prcr
    import workloads
    out = []
    for model in ("qwen3-vl-8b", "qwen3-vl-32b"):
        for K in (32, 128):
            w = workloads.paper_k(model, K)
            p = Prepared(w, dev)
            s = torch.cuda.Stream(device=dev)

            def two():
                p.reassign(s)
                p.rebind(s)

            def fused():
                prcr.revisit(p.rope, p.mem, p.sel_off, p.sel_idx, p.p_txt, p.cache, p.cache_len,
                             "pcr", 2, p.new_pos, p.next_pos, p.new_len, p.slots, p.err, s)

            res = {"model": model, "K": K, "entries": w.entries(), "bytes": w.algorithmic_bytes()}
            for name, fn in (("two_launches", two), ("fused", fused)):
                # host loop through the Python binding (bounded by host call overhead)
                torch.cuda.synchronize()
                with torch.cuda.stream(s):
                    for _ in range(5):
                        fn()
                    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    a.record(s)
                    for _ in range(reps):
                        fn()
                    b.record(s)
                    torch.cuda.synchronize()
                res[name + "_host_loop_us"] = round(a.elapsed_time(b) / reps * 1e3, 2)
                # device time per revisit: n_graph revisits captured in one HIP graph
                n_graph = 50
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=s):
                    for _ in range(n_graph):
                        fn()
                torch.cuda.synchronize()
                with torch.cuda.stream(s):
                    g.replay()
                    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    a.record(s)
                    for _ in range(4):
                        g.replay()
                    b.record(s)
                    torch.cuda.synchronize()
                res[name + "_graph_us"] = round(a.elapsed_time(b) / (4 * n_graph) * 1e3, 2)
                del g
            if int(p.err.item()) != 0:
                raise RuntimeError("device reported a data error in the small-K runs")
            res["fused_graph_GBs"] = round(w.algorithmic_bytes() / (res["fused_graph_us"] / 1e6) / 1e9, 1)
            out.append(res)
            del p
            torch.cuda.empty_cache()
    return out


def prefill_capture_bw(dev, steps=20, NL=36, H=8):
    """Bandwidth of the fused prefill capture (one layer per call) at the 32-sequence
    shape: 32 prompts of 256 text + 64x32 visual + 256 text tokens, NL layers x H KV
    heads (36 x 8 by default; 28 x 4 is the paged workload's model shape), d 128,
    bf16, interleaved M-RoPE.  Algorithmic bytes per call: read raw K+V of every
    prompt row, write K+V into the cache, and K+V into the memory for the visual
    rows (2 * d * 2 bytes each)."""
    import numpy as np
    import torch

    import paper_2606_26631_amd as prcr
    import workloads
    B, D = 32, 128
    pos, vis, n_tok, n_vis = workloads.prompt(B, n_before=(256,) * B, grid=((64, 32),) * B,
                                              n_after=(256,) * B, frames=(1,) * B)
    S = pos.shape[1]
    M = int(n_vis.max())
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    g = torch.Generator(device=dev)
    g.manual_seed(3000)
    raw_k = torch.randn((B, S, H, D), generator=g, device=dev).to(torch.bfloat16)
    raw_v = torch.randn((B, S, H, D), generator=g, device=dev).to(torch.bfloat16)
    mem = prcr.Memory(torch.empty((B, M, NL, H, D), dtype=torch.bfloat16, device=dev),
                      torch.empty((B, M, NL, H, D), dtype=torch.bfloat16, device=dev),
                      torch.zeros((B, M, 3), dtype=torch.int32, device=dev), t(n_vis))
    s_max = S + 256
    cache = prcr.Cache(torch.empty((B, NL, H, s_max, D), dtype=torch.bfloat16, device=dev),
                       torch.empty((B, NL, H, s_max, D), dtype=torch.bfloat16, device=dev))
    rope = prcr.Rope(D, (22, 21, 21), True, 5e6)
    args = (t(pos), t(n_tok), t(vis))
    start = torch.zeros(B, dtype=torch.int32, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    s = torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        for layer in range(3):
            prcr.prefill_capture(rope, mem, layer, raw_k, raw_v, *args, cache, start, True, err, s)
        evs = []
        for i in range(steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s)
            prcr.prefill_capture(rope, mem, i % NL, raw_k, raw_v, *args, cache, start, True, err, s)
            b.record(s)
            evs.append((a, b))
        torch.cuda.synchronize()
    if int(err.item()) != 0:
        raise RuntimeError("device reported a data error in the prefill capture runs")
    ms = [a.elapsed_time(b) for a, b in evs]
    mean_s = sum(ms) / len(ms) / 1e3
    rows = int(n_tok.sum()) * H
    vrows = int(n_vis.sum()) * H
    nbytes = (rows * 2 * 2 + vrows * 2) * D * 2
    # The same reads and writes with no arithmetic (copyref prefill_pattern_kernel),
    # on the same arrays, with the prefill kernel's wave mapping.
    L = copyref_lib()
    state = {"i": 0}

    def pattern():
        rc = L.prcr_copyref_prefill(raw_k.data_ptr(), raw_v.data_ptr(), args[2].data_ptr(),
                                    args[1].data_ptr(), cache.k.data_ptr(), cache.v.data_ptr(),
                                    mem.k.data_ptr(), mem.v.data_ptr(), B, S, H, NL,
                                    state["i"] % NL, s_max, M, s.cuda_stream)
        state["i"] += 1
        if rc != 0:
            raise RuntimeError(f"prcr_copyref_prefill failed ({rc})")

    pat_ms, _ = _timed(pattern, s, steps, 3)
    del mem, cache, raw_k, raw_v
    torch.cuda.empty_cache()
    return {"kernel": "prcr_prefill_capture", "workload": f"{B} prompts x {S} tokens "
            f"({int(n_vis[0])} visual), {NL} layers x {H} KV heads, d {D}, bf16, one layer per call",
            "mean_launch_us": round(mean_s * 1e6, 2), "algorithmic_bytes_per_call": nbytes,
            "achieved": round(nbytes / mean_s / 1e9, 1), "unit": "GB/s",
            "frac": round(nbytes / mean_s / 1e9 / HBM_PEAK_GBS, 4),
            "pattern_copy": {"kernel": "copyref prefill_pattern_kernel (the same reads and writes, no "
                                       "arithmetic)", "mean_launch_us": round(pat_ms * 1e3, 2),
                             "achieved": round(nbytes / (pat_ms / 1e3) / 1e9, 1), "unit": "GB/s",
                             "frac": round(nbytes / (pat_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4)},
            "frac_of_pattern": round(pat_ms / 1e3 / mean_s, 4),
            "traffic": load_traffic("prefill_capture" if H == 8 else f"prefill_capture_{H}kv", "prefill")}


def store_raw_bw(dev, steps=20):
    """Bandwidth of prcr_store_raw (one layer per call) at the 32-sequence shape: 32
    prompts of 2560 rows with 2048 visual tokens, 36 layers x 8 KV heads, d 128,
    bf16.  Algorithmic bytes per call: read and write the K and V rows of every
    visual token (4 * H * d * 2 bytes each)."""
    import numpy as np
    import torch

    import paper_2606_26631_amd as prcr
    B, M, S, NL, H, D = 32, 2048, 2560, 36, 8, 128
    g = torch.Generator(device=dev)
    g.manual_seed(3500)
    # Successive calls read different projections (three sets, 1 GB), as successive
    # layers do: the 268 MB of rows one call reads would otherwise be partly served
    # from the device's last-level cache on the next call.
    raws = [(torch.randn((B, S, H, D), generator=g, device=dev).to(torch.bfloat16),
             torch.randn((B, S, H, D), generator=g, device=dev).to(torch.bfloat16))
            for _ in range(3)]
    mem = prcr.Memory(torch.empty((B, M, NL, H, D), dtype=torch.bfloat16, device=dev),
                      torch.empty((B, M, NL, H, D), dtype=torch.bfloat16, device=dev),
                      torch.zeros((B, M, 3), dtype=torch.int32, device=dev),
                      torch.full((B,), M, dtype=torch.int32, device=dev))
    vis = torch.from_numpy(np.broadcast_to(256 + np.arange(M, dtype=np.int32), (B, M)).copy()).to(dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    s = torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        for layer in range(3):
            prcr.store_raw(mem, layer, *raws[layer % 3], vis, err, s)
        evs = []
        for i in range(steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s)
            prcr.store_raw(mem, i % NL, *raws[i % 3], vis, err, s)
            b.record(s)
            evs.append((a, b))
        torch.cuda.synchronize()
    if int(err.item()) != 0:
        raise RuntimeError("device reported a data error in the store_raw runs")
    mean_s = sum(a.elapsed_time(b) for a, b in evs) / len(evs) / 1e3
    nbytes = B * M * H * D * 2 * 4
    del mem, raws
    torch.cuda.empty_cache()
    return {"kernel": "prcr_store_raw", "workload": f"{B} prompts x {S} rows ({M} visual), {NL} "
            f"layers x {H} KV heads, d {D}, bf16, one layer per call",
            "mean_launch_us": round(mean_s * 1e6, 2), "algorithmic_bytes_per_call": nbytes,
            "achieved": round(nbytes / mean_s / 1e9, 1), "unit": "GB/s",
            "frac": round(nbytes / mean_s / 1e9 / HBM_PEAK_GBS, 4),
            "traffic": load_traffic("store_raw", "store")}


def video_revisits(dev, reps=5):
    """Workload 4 (8 video sequences, 28 layers x 4 KV heads, d 128, bf16): four
    successive revisits of 1024 tokens each, 32 text tokens decoded in between
    (cache lengths and p_txt advance on the device between revisits, untimed).
    Each revisit is one reassign + one rebind launch, timed with HIP events on the
    launch stream; reported per revisit and as the 4-revisit total, median over
    reps repetitions of the whole sequence of revisits.  Every repetition is
    enqueued behind the previous one with no host synchronisation in between: the
    first launch after the queue has drained starts ~25 us late, which an event
    recorded just before it would charge to the first revisit."""
    import statistics

    import numpy as np
    import torch

    import paper_2606_26631_amd as prcr
    import workloads
    w = workloads.make(4, "full")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    vals = workloads.torch_values(w, dev)
    mem = prcr.Memory(vals["mem_k"], vals["mem_v"], t(w.coords), t(w.n_visual))
    cache = prcr.Cache(vals["cache_k"], vals["cache_v"])
    rope = prcr.Rope(w.D, w.sections, w.interleaved, w.theta)
    sels = [(t(so), t(si), int(si.shape[0])) for so, si in w.revisits]
    bufs = [(torch.empty((k, 3), dtype=torch.float64, device=dev),
             torch.empty((w.B,), dtype=torch.int32, device=dev),
             torch.empty((w.B,), dtype=torch.int32, device=dev),
             torch.empty((k,), dtype=torch.int64, device=dev)) for _, _, k in sels]
    lens0, p_txt0 = t(w.cache_len), t(w.p_txt)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    s = torch.cuda.Stream(device=dev)
    all_evs = []
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        for rep in range(reps + 1):                      # the first pass is a warm-up
            lens, p_txt = lens0, p_txt0
            evs = []
            for (so, si, k), (new_pos, next_pos, new_len, slots) in zip(sels, bufs):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(s)
                prcr.reassign_coords(mem, so, si, p_txt, "pcr", 2, new_pos, next_pos, err, s)
                prcr.rebind_inject(rope, mem, so, si, new_pos, cache, lens, new_len, slots, err, s)
                b.record(s)
                evs.append((a, b))
                lens = new_len + w.decode_between
                p_txt = next_pos + (w.decode_between - 1)
            if rep:
                all_evs.append(evs)
        torch.cuda.synchronize()
    times = [[evs[r][0].elapsed_time(evs[r][1]) for evs in all_evs] for r in range(len(sels))]
    if int(err.item()) != 0:
        raise RuntimeError("device reported a data error in the video revisits")
    entries = [k * w.NL * w.H for _, _, k in sels]
    nbytes = [e * 4 * w.D * 2 for e in entries]
    med = [statistics.median(x) for x in times]
    del mem, cache, vals
    torch.cuda.empty_cache()
    return {"workload": f"workload 4 (video): {w.B} sequences, {w.NL} layers x {w.H} KV heads, "
            f"d {w.D}, bf16, 4 revisits of 1024 tokens, {w.decode_between} tokens decoded between",
            "per_revisit_us": [round(m * 1e3, 2) for m in med],
            "per_revisit_GBs": [round(n / (m * 1e6), 1) for n, m in zip(nbytes, med)],
            "total_us": round(sum(med) * 1e3, 2),
            "total_entries": sum(entries), "algorithmic_bytes_total": sum(nbytes),
            "total_GBs": round(sum(nbytes) / (sum(med) * 1e6), 1)}


def small_workloads(dev, reps=20):
    """Workloads 1 (tiny, fp32) and 2 (one Qwen2.5-VL-7B-shaped sequence, bf16): one
    reassign + rebind per launch pair, the median of reps timed pairs, each after a
    512 MB buffer is written so that the 256 MB last-level cache holds none of the
    working set (these calls move at most 22 MB)."""
    import statistics

    import torch

    import workloads
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    res = []
    for cfg in (1, 2):
        w = workloads.make(cfg, "full")
        p = Prepared(w, dev)
        s = torch.cuda.Stream(device=dev)
        pairs, rebinds = [], []
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            for i in range(reps + 3):
                flush.fill_(i & 0xFF)
                a, b, c = (torch.cuda.Event(enable_timing=True) for _ in range(3))
                a.record(s)
                p.reassign(s)
                b.record(s)
                p.rebind(s)
                c.record(s)
                if i >= 3:
                    pairs.append((a, b, c))
            torch.cuda.synchronize()
        if int(p.err.item()) != 0:
            raise RuntimeError(f"device reported a data error in workload {cfg}")
        rb = statistics.median(b.elapsed_time(c) for a, b, c in pairs)
        both = statistics.median(a.elapsed_time(c) for a, b, c in pairs)
        res.append({"workload": f"workload {w.cfg} ({w.name})", "entries": w.entries(),
                    "algorithmic_bytes": w.algorithmic_bytes(), "median_rebind_us": round(rb * 1e3, 2),
                    "median_reassign_plus_rebind_us": round(both * 1e3, 2),
                    "rebind_GBs": round(w.algorithmic_bytes() / (rb * 1e6), 1)})
        del p
    del flush
    torch.cuda.empty_cache()
    return res


def decode_attention_bw(dev, steps=20, cfg=3):
    """Bandwidth of decode attention over a workload's active cache after its revisit
    (lengths + K_b), 4 query heads per KV head, bf16, one layer per call: workload 3
    (32 sequences, 36 layers x 8 KV heads, contiguous) or workload 5 (64 sequences,
    28 layers x 4 KV heads, paged, block 16).  Algorithmic bytes: every attended K
    and V row once, plus the queries and outputs."""
    import numpy as np
    import torch

    import paper_2606_26631_amd as prcr
    import workloads
    w = workloads.make(cfg, "full")
    Hq = 4 * w.H
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    g = torch.Generator(device=dev)
    g.manual_seed(4000 + cfg)
    shape = workloads.cache_shape(w)
    cache = prcr.Cache(torch.randn(shape, generator=g, device=dev).to(torch.bfloat16),
                       torch.randn(shape, generator=g, device=dev).to(torch.bfloat16),
                       t(w.block_table) if w.paged else None)
    rope = prcr.Rope(w.D, w.sections, w.interleaved, w.theta)
    lens = (w.cache_len + np.diff(w.sel_off)).astype(np.int32)
    q = torch.randn((w.B, Hq, w.D), generator=g, device=dev).to(torch.bfloat16)
    q_pos, cl = t(w.p_txt + 1), t(lens)
    out = torch.empty((w.B, Hq, w.D), dtype=torch.float32, device=dev)
    ws = torch.empty(prcr.decode_workspace_bytes(cache, w.B, Hq) // 4 + 1, dtype=torch.float32,
                     device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    s = torch.cuda.Stream(device=dev)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        for layer in range(3):
            prcr.decode_attention(rope, cache, layer, q, q_pos, cl, None, out, ws, err, s)
        evs = []
        for i in range(steps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(s)
            prcr.decode_attention(rope, cache, i % w.NL, q, q_pos, cl, None, out, ws, err, s)
            b.record(s)
            evs.append((a, b))
        torch.cuda.synchronize()
    if int(err.item()) != 0:
        raise RuntimeError("device reported a data error in the decode attention runs")
    ms = [a.elapsed_time(b) for a, b in evs]
    mean_s = sum(ms) / len(ms) / 1e3
    nbytes = int(lens.sum()) * w.H * w.D * 2 * 2 + w.B * Hq * w.D * (2 + 4)
    # The same K and V reads with no arithmetic (copyref decode_read_kernel), on the
    # same cache, with the decode kernel's split and lane layout, one layer per call
    # in the same order as above.
    L = copyref_lib()
    per_split = w.B * Hq * (w.D + 2) * 4
    n_split = prcr.decode_workspace_bytes(cache, w.B, Hq) // per_split
    sink = torch.empty(w.B * w.H * n_split, dtype=torch.int32, device=dev)
    cc = cache.to_c()

    calls = [0]

    def read_pattern():
        layer = calls[0] % w.NL
        calls[0] += 1
        rc = L.prcr_copyref_decode_read(cache.k.data_ptr(), cache.v.data_ptr(),
                                        cache.block_table.data_ptr() if w.paged else None,
                                        cl.data_ptr(), sink.data_ptr(), w.B, w.NL, w.H, layer,
                                        cc.s_max, cc.block_size, cc.max_blocks, cc.n_blocks,
                                        n_split, int(w.paged), s.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"prcr_copyref_decode_read failed ({rc})")

    read_ms, _ = _timed(read_pattern, s, steps, 3)
    read_bytes = int(lens.sum()) * w.H * w.D * 2 * 2
    del cache, ws, sink
    torch.cuda.empty_cache()
    layout = f"paged, block {w.block_size}" if w.paged else "contiguous"
    res = {"kernel": "prcr_decode_attention", "workload": f"workload {cfg}: {w.B} sequences, cache "
           f"lengths {int(lens.min())}-{int(lens.max())}, {w.H} KV heads, {Hq} query heads, d {w.D}, "
           f"bf16, {layout}, one layer per call", "mean_call_us": round(mean_s * 1e6, 2),
           "algorithmic_bytes_per_call": nbytes, "achieved": round(nbytes / mean_s / 1e9, 1),
           "unit": "GB/s", "frac": round(nbytes / mean_s / 1e9 / HBM_PEAK_GBS, 4)}
    read_gbs = read_bytes / (read_ms / 1e3) / 1e9
    res["pattern_read"] = {"kernel": "copyref decode_read_kernel (the same K/V reads, no "
                                     "arithmetic)", "mean_launch_us": round(read_ms * 1e3, 2),
                           "bytes": read_bytes, "achieved": round(read_gbs, 1), "unit": "GB/s",
                           "frac": round(read_gbs / HBM_PEAK_GBS, 4)}
    res["frac_of_pattern"] = round(res["achieved"] / read_gbs, 4)
    res["traffic"] = load_traffic("decode_attention" if cfg == 3 else "decode_attention_paged",
                                  "decode")
    return res


def add_references(roof, w, pattern_ms, copy):
    """The rebind's rate against the streaming copy and against the copy of its own
    access pattern on the same arrays (means of the same number of launches)."""
    mean_s = sum(pattern_ms) / len(pattern_ms) / 1e3
    gbs = w.algorithmic_bytes() / mean_s / 1e9
    roof["pattern_copy"] = {"kernel": "copyref pattern_kernel (the rebind's addresses, no "
                                      "arithmetic)", "mean_launch_us": round(mean_s * 1e6, 2),
                            "achieved": round(gbs, 1), "unit": "GB/s",
                            "frac": round(gbs / HBM_PEAK_GBS, 4)}
    roof["frac_of_pattern"] = round(roof["achieved"] / gbs, 4)
    roof["frac_of_copy"] = round(roof["achieved"] / copy["achieved"], 4)


def roofline(w, rebind_ms, traffic):
    mean_s = sum(rebind_ms) / len(rebind_ms) / 1e3
    gbs = w.algorithmic_bytes() / mean_s / 1e9
    return {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
            "kernel": "prcr_rebind_inject", "mean_launch_us": round(mean_s * 1e6, 2),
            "median_launch_us": round(statistics.median(rebind_ms) * 1e3, 2),
            "min_launch_us": round(min(rebind_ms) * 1e3, 2)}


_CPU_INPUTS = []      # per-sequence oracle inputs, shared with forked workers


def _cpu_inputs(w, max_bytes=3 << 30):
    """Per-sequence oracle inputs of workload w on the host (sequence b's memory
    rows and cache), with seeded N(0, 1) contents rounded to the storage type by
    torch on the CPU; at most max_bytes in all."""
    import numpy as np
    import torch

    import workloads
    g = torch.Generator().manual_seed(5000 + w.cfg)
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16

    def rnd(*shape):
        return workloads.as_numpy_storage(torch.randn(shape, generator=g).to(tdt))

    inputs, held = [], 0
    for b in range(w.B):
        s0, s1 = int(w.sel_off[b]), int(w.sel_off[b + 1])
        M = w.coords.shape[1]
        mem = {"k": rnd(1, M, w.NL, w.H, w.D), "v": rnd(1, M, w.NL, w.H, w.D),
               "n_visual": w.n_visual[b:b + 1], "dtype": w.dtype}
        if w.paged:
            n = int((w.block_table[b] >= 0).sum())
            cache = {"paged": True, "k": rnd(w.NL, n, w.block_size, w.H, w.D),
                     "v": rnd(w.NL, n, w.block_size, w.H, w.D),
                     "block_table": np.arange(n, dtype=np.int32)[None],
                     "block_size": w.block_size, "max_blocks": n, "n_blocks": n}
        else:
            cache = {"paged": False, "k": rnd(1, w.NL, w.H, w.s_max, w.D),
                     "v": rnd(1, w.NL, w.H, w.s_max, w.D), "s_max": w.s_max}
        inputs.append((b, np.array([0, s1 - s0]), w.sel_idx[s0:s1], mem, cache))
        held += sum(x.nbytes for x in (mem["k"], mem["v"], cache["k"], cache["v"]))
        if held >= max_bytes:
            break
    return inputs


def _oracle_loop(w, first, budget_s):
    """Oracle calls over the shared inputs (starting at index first, round robin)
    until budget_s seconds have been spent in them: (entries, seconds, calls)."""
    import oracle
    done, spent, calls, i = 0, 0.0, 0, first
    while spent < budget_s:
        b, sel_off, sel_idx, mem, cache = _CPU_INPUTS[i % len(_CPU_INPUTS)]
        t = time.perf_counter()
        pos, _, _ = oracle.reassign_batch(w.coords[b:b + 1], w.n_visual[b:b + 1], sel_off, sel_idx,
                                          w.p_txt[b:b + 1])
        oracle.rebind_inject(w.rope(), mem, sel_off, sel_idx, pos, cache, w.cache_len[b:b + 1])
        spent += time.perf_counter() - t
        done += len(sel_idx) * w.NL * w.H
        calls += 1
        i += 1
    return done, spent, calls


def _oracle_worker(args):
    w, first, budget_s = args
    return _oracle_loop(w, first, budget_s)


def cpu_model() -> str:
    """The host CPU's model name, from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, budget_s=10.0):
    """The oracle, as it stands, on whole sequences of workload w (one sequence per
    call: reassignment + rebind/inject into that sequence's cache), timed on the
    host before any GPU work: in a pool of worker processes, one per core available
    to this process (at most 16, the host CPU share of one GPU on these machines),
    each for about budget_s seconds and each starting at a different sequence;
    then in this process alone (1 thread).  Inputs (up to 8 sequences, about 7.5
    GB) are built on the host, untimed."""
    import multiprocessing as mp
    _CPU_INPUTS[:] = _cpu_inputs(w, max_bytes=7 << 30)
    n_seq = len(_CPU_INPUTS)
    avail = len(os.sched_getaffinity(0))
    workers = max(1, min(16, avail))
    t = time.perf_counter()
    with mp.get_context("fork").Pool(workers) as pool:
        res = pool.map(_oracle_worker, [(w, i, budget_s) for i in range(workers)])
    wall = time.perf_counter() - t
    done_all = sum(r[0] for r in res)
    out = {"value": round(done_all / wall, 1), "unit": "entries/s", "cores": workers,
           "kind": "oracle", "cpu_model": cpu_model(), "cores_available": avail,
           "sample": f"workload {w.cfg}: {workers} worker processes (one per core), each "
                     f"running whole-sequence oracle calls (reassignment + rebind/inject) over "
                     f"sequences 0..{n_seq - 1} round robin from its own start for about "
                     f"{budget_s:.0f} s: {done_all} entries in {wall:.1f} s wall time, numpy "
                     "float64, one thread per process"}
    done, spent, calls = _oracle_loop(w, 0, budget_s)
    out["one_core"] = {"value": round(done / spent, 1), "unit": "entries/s", "cores": 1,
                       "sample": f"{calls} oracle calls in this process, sequences "
                                 f"0..{n_seq - 1} in turn: {done} entries in {spent:.1f} s"}
    _CPU_INPUTS.clear()
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--secondary", type=int, default=5, help="second workload (0: none)")
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-small-k", action="store_true", help="skip the small-K latency section")
    ap.add_argument("--no-prefill", action="store_true", help="skip the prefill-capture section")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode-attention section")
    ap.add_argument("--no-video", action="store_true", help="skip the four-revisit video section")
    ap.add_argument("--no-key-only", action="store_true", help="skip the key-only memory section")
    ap.add_argument("--no-capacity", action="store_true",
                    help="skip the run with 8192 cache slots per sequence")
    ap.add_argument("--no-one-d", action="store_true",
                    help="skip the run with 1-D rotary positions (InternVL3.5-style)")
    ap.add_argument("--no-shift", action="store_true", help="skip the SHIFT reassignment run")
    ap.add_argument("--no-tp-shard", action="store_true",
                    help="skip the one-GPU share of the workload at 8-way KV-head parallelism")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the rebinding path shards by sequence, KV head or "
              "layer with no exchange, and only N=1 is run and reported.", file=sys.stderr)
        sys.exit(2)

    import workloads
    w = workloads.make(args.workload, "full")
    # The oracle runs first, before this process touches the GPU, so that its
    # worker processes are forked from a process without GPU state.
    cpu = None if args.no_cpu_baseline else cpu_baseline(w, args.cpu_budget)

    import torch
    dev = torch.device("cuda:0")
    khash = kernel_source_hash()
    total_ms, rebind_ms, reassign_ms, pattern_ms = measure(w, args.steps, args.warmup, dev,
                                                           with_pattern=True)
    ms_step = total_ms / args.steps
    out = {
        "metric": "rebound KV entries/sec (layers\u00d7heads\u00d7tokens) and achieved HBM GB/s vs peak",
        "value": round(w.entries() * args.steps / (total_ms / 1e3), 1),
        "unit": "entries/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": describe(w),
        "roofline": roofline(w, rebind_ms, load_traffic(f"rebind_workload{w.cfg}", "rebind")),
        "reassign_mean_us": round(sum(reassign_ms) / len(reassign_ms) * 1e3, 2),
        "kernel_source_hash": khash,
    }
    copy = copy_reference(dev)
    out["attainable_copy"] = copy
    add_references(out["roofline"], w, pattern_ms, copy)
    if args.secondary:
        w2 = workloads.make(args.secondary, "full")
        t2, r2, a2, p2 = measure(w2, args.steps, args.warmup, dev, with_pattern=True)
        out["secondary"] = {"config": describe(w2),
                            "value": round(w2.entries() * args.steps / (t2 / 1e3), 1),
                            "unit": "entries/s", "ms_per_step": round(t2 / args.steps, 4),
                            "roofline": roofline(w2, r2, load_traffic(f"rebind_workload{w2.cfg}", "rebind"))}
        add_references(out["secondary"]["roofline"], w2, p2, copy)
    def key_only():
        wk = workloads.make(args.workload, "full")
        _, rk, _ = measure(wk, args.steps, args.warmup, dev, key_only=True)
        return {"workload": f"workload {wk.cfg} ({wk.name}), key-only memory: values copied from "
                            "the prompt slots of the same cache",
                "roofline": roofline(wk, rk, None)}

    def shift_mode():
        ws_ = workloads.make(args.workload, "full")
        ts, rs, as_ = measure(ws_, args.steps, args.warmup, dev, mode="shift")
        return {"workload": f"workload {ws_.cfg} ({ws_.name}), SHIFT reassignment (the region "
                            "translated to start at the next position, layout kept)",
                "value": round(ws_.entries() * args.steps / (ts / 1e3), 1), "unit": "entries/s",
                "reassign_mean_us": round(sum(as_) / len(as_) * 1e3, 2),
                "roofline": roofline(ws_, rs, None)}

    def capacity_8192():
        wc = workloads.with_capacity(workloads.make(args.workload, "full"), 8192)
        tc, rc, _ = measure(wc, args.steps, args.warmup, dev)
        return {"config": describe(wc), "value": round(wc.entries() * args.steps / (tc / 1e3), 1),
                "unit": "entries/s", "roofline": roofline(wc, rc, None)}

    def one_d_rotary():
        w1 = workloads.one_d(workloads.make(args.workload, "full"))
        t1, r1, _ = measure(w1, args.steps, args.warmup, dev)
        return {"config": describe(w1), "value": round(w1.entries() * args.steps / (t1 / 1e3), 1),
                "unit": "entries/s", "roofline": roofline(w1, r1, None)}

    def tp8_shard():
        wt = workloads.tp_shard(workloads.make(args.workload, "full"), 8)
        tt, rt, _ = measure(wt, args.steps, args.warmup, dev)
        return {"config": describe(wt), "value": round(wt.entries() * args.steps / (tt / 1e3), 1),
                "unit": "entries/s", "roofline": roofline(wt, rt, None)}

    # Further sections: a Python-level failure in one of them is reported in its
    # place (traceback on stderr) and does not cost the measurement above.
    sections = [] if args.no_shift else [("shift_mode", shift_mode)]
    if args.workload == 3 and not args.no_capacity:
        sections.append(("power_of_two_capacity", capacity_8192))
    if not args.no_key_only:
        sections.append(("key_only_memory", key_only))
    if not args.no_one_d:
        sections.append(("one_d_rotary", one_d_rotary))
    if not args.no_tp_shard:
        sections.append(("tp8_shard", tp8_shard))
    if not args.no_video:
        sections.append(("video_revisits", lambda: video_revisits(dev)))
    if not args.no_small_k:
        sections.append(("small_k_latency", lambda: small_k_latency(dev)))
        sections.append(("small_workloads", lambda: small_workloads(dev)))
    if not args.no_prefill:
        sections.append(("prefill_capture", lambda: prefill_capture_bw(dev)))
        sections.append(("prefill_capture_4kv_heads", lambda: prefill_capture_bw(dev, NL=28, H=4)))
        sections.append(("store_raw", lambda: store_raw_bw(dev)))
    if not args.no_decode:
        sections.append(("decode_attention", lambda: decode_attention_bw(dev)))
        sections.append(("decode_attention_paged", lambda: decode_attention_bw(dev, cfg=5)))
    for name, fn in sections:
        try:
            out[name] = fn()
        except Exception as e:              # noqa: BLE001 - reported, not hidden
            import traceback
            traceback.print_exc()
            out[name] = {"error": f"{type(e).__name__}: {e}"}
            try:
                torch.cuda.synchronize()
                torch.cuda.empty_cache()
            except Exception:               # noqa: BLE001 - the error above is the report
                pass
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
