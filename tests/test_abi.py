"""C-ABI checks that need no GPU: the library loads, exports every function that
include/prcr.h declares, and rejects malformed calls on the host before any HIP
call (so no device work is started).  No compute call is made here."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2606_26631_amd as prcr
from paper_2606_26631_amd.binding import CCache, CMem, CRope

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "prcr.h")
FAKE = 0x10000          # 64 KiB-aligned placeholder address; never dereferenced


def _gpu_visible() -> bool:
    import torch
    return torch.cuda.device_count() > 0          # counts devices without initialising them


# The validation tests below pass placeholder pointers and rely on every call being
# rejected on the host.  They are host-side checks: where a GPU is visible they are
# skipped, so that a validation mistake can never turn into a launch on bad memory.
host_only = pytest.mark.skipif(_gpu_visible(), reason="placeholder-pointer checks run on hosts "
                                                      "without a GPU")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(prcr_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    L = prcr.lib()
    names = declared_functions()
    assert {"prcr_store_raw", "prcr_reassign_coords", "prcr_rebind_inject"} <= set(names)
    for n in names:
        assert hasattr(L, n), f"{n} declared in prcr.h but not exported"
    assert L.prcr_version() == 10400


def test_status_strings():
    L = prcr.lib()
    for code in range(10):
        assert len(L.prcr_status_str(code)) > 0
    assert L.prcr_status_str(99) == b"unknown status"


ROPES = [(64, (8, 12, 12), False, 1e6), (64, (11, 11, 10), True, 1e6),
         (128, (16, 24, 24), False, 1e6), (128, (22, 21, 21), True, 5e6),
         (128, (24, 20, 20), True, 5e6),
         # 1-D rotary (every pair on t), under both readings of the sections
         (64, (32, 0, 0), False, 1e4), (128, (64, 0, 0), False, 1e6), (128, (64, 0, 0), True, 1e6)]


@pytest.mark.parametrize("D,sections,inter,theta", ROPES)
def test_host_tables_match_oracle(D, sections, inter, theta):
    r = prcr.Rope(D, sections, inter, theta)
    assert np.array_equal(np.array(r.inv_freq()), oracle.inv_freq(theta, D))
    assert np.array_equal(np.array(r.pair_axis()), oracle.pair_axis(D, sections, inter))


def test_unsupported_axis_map():
    with pytest.raises(prcr.PrcrError) as e:
        prcr.Rope(128, (32, 16, 16), False, 1e6).pair_axis()
    assert e.value.status == 6


# --- structural validation -------------------------------------------------
def good():
    rope = CRope(128, (ctypes.c_int32 * 3)(16, 24, 24), 0, 1e6)
    mem = CMem(FAKE, FAKE, FAKE, FAKE, 2, 100, 28, 4, 128, 1)
    cache = CCache(0, FAKE, FAKE, 512, None, 0, 0, 0)
    return rope, mem, cache


def call_rebind(rope, mem, cache, total_k=10, sel_off=FAKE, sel_idx=FAKE, new_pos=FAKE,
                cache_len=FAKE, new_len=FAKE + 0x100, slots=FAKE, err=None):
    L = prcr.lib()
    return L.prcr_rebind_inject(ctypes.byref(rope) if rope is not None else None,
                                ctypes.byref(mem) if mem is not None else None,
                                sel_off, sel_idx, total_k, new_pos,
                                ctypes.byref(cache) if cache is not None else None,
                                cache_len, new_len, slots, err, None)


FAR = 1 << 40          # a placeholder output address far from every input above


def call_reassign(mem, mode=0, l_ext=2, total_k=10, new_pos=FAKE, p_txt=FAKE, next_pos=FAR,
                  sel_off=FAKE):
    L = prcr.lib()
    return L.prcr_reassign_coords(ctypes.byref(mem) if mem is not None else None, sel_off, FAKE,
                                  total_k, p_txt, mode, l_ext, new_pos, next_pos, None, None)


def call_store(mem, layer=0, raw_k=FAKE, s_src=10):
    L = prcr.lib()
    return L.prcr_store_raw(ctypes.byref(mem) if mem is not None else None, layer, raw_k, FAKE,
                            s_src, FAKE, None, None)


@host_only
def test_rebind_validation_errors():
    rope, mem, cache = good()
    assert call_rebind(None, mem, cache) == 1
    assert call_rebind(rope, None, cache) == 1
    assert call_rebind(rope, mem, None) == 1
    assert call_rebind(rope, mem, cache, sel_off=None) == 1
    assert call_rebind(rope, mem, cache, sel_idx=None) == 1
    assert call_rebind(rope, mem, cache, new_pos=None) == 1
    assert call_rebind(rope, mem, cache, cache_len=None) == 1
    assert call_rebind(rope, mem, cache, total_k=-1) == 2
    # misaligned pointers
    assert call_rebind(rope, mem, cache, new_pos=FAKE + 4) == 4
    assert call_rebind(rope, mem, cache, slots=FAKE + 4) == 4
    assert call_rebind(rope, mem, cache, sel_idx=FAKE + 2) == 4
    # new_cache_len aliasing cache_len
    assert call_rebind(rope, mem, cache, new_len=FAKE) == 7
    # shapes
    r2, m2, c2 = good(); m2.head_dim = 64
    assert call_rebind(r2, m2, c2) == 2                # rope/mem head_dim mismatch
    r2, m2, c2 = good(); r2.section[0] = 15
    assert call_rebind(r2, m2, c2) == 2                # sections do not sum to d/2
    r2, m2, c2 = good(); r2.theta = -1.0
    assert call_rebind(r2, m2, c2) == 2
    r2, m2, c2 = good(); r2.section[0], r2.section[1] = 32, 8
    assert call_rebind(r2, m2, c2) == 6                # valid rope, no compiled map
    r2, m2, c2 = good(); m2.dtype = 7
    assert call_rebind(r2, m2, c2) == 3
    r2, m2, c2 = good(); m2.k = FAKE + 8
    assert call_rebind(r2, m2, c2) == 4
    r2, m2, c2 = good(); c2.v = FAKE + 8
    assert call_rebind(r2, m2, c2) == 4
    r2, m2, c2 = good(); c2.s_max = 0
    assert call_rebind(r2, m2, c2) == 2
    r2, m2, c2 = good(); c2.paged = 1
    assert call_rebind(r2, m2, c2) == 1                # paged without block table
    r2, m2, c2 = good(); c2.paged, c2.block_table = 1, FAKE
    assert call_rebind(r2, m2, c2) == 2                # paged with zero sizes
    r2, m2, c2 = good(); c2.paged = 2
    assert call_rebind(r2, m2, c2) == 2
    r2, m2, c2 = good(); m2.batch = 0
    assert call_rebind(r2, m2, c2) == 2
    # key-only memory: no values needs the value-slot table, aligned
    r2, m2, c2 = good(); m2.v = None
    assert call_rebind(r2, m2, c2) == 1
    r2, m2, c2 = good(); m2.v, m2.v_slot = None, FAKE + 2
    assert call_rebind(r2, m2, c2) == 4


@host_only
def test_reassign_validation_errors():
    _, mem, _ = good()
    assert call_reassign(None) == 1
    assert call_reassign(mem, mode=9) == 5
    assert call_reassign(mem, l_ext=-1) == 5
    assert call_reassign(mem, new_pos=None) == 1
    assert call_reassign(mem, new_pos=FAKE + 4) == 4
    assert call_reassign(mem, p_txt=None) == 1
    m2 = good()[1]; m2.coords = None
    assert call_reassign(m2) == 1


@host_only
def test_store_validation_errors():
    _, mem, _ = good()
    assert call_store(None) == 1
    assert call_store(mem, layer=28) == 2
    assert call_store(mem, layer=-1) == 2
    assert call_store(mem, s_src=0) == 2
    assert call_store(mem, raw_k=None) == 1
    assert call_store(mem, raw_k=FAKE + 8) == 4
    m2 = good()[1]; m2.v = None
    assert call_store(m2) == 1                         # key-only memory without v_slot


def call_revisit(rope, mem, cache, mode=0, l_ext=2, p_txt=FAKE, next_pos=FAKE + 0x200,
                 new_pos=None, cache_len=FAKE, new_len=FAKE + 0x100, sel_off=FAKE):
    L = prcr.lib()
    return L.prcr_revisit(ctypes.byref(rope), ctypes.byref(mem) if mem is not None else None,
                          sel_off, FAKE, 10, p_txt, mode, l_ext, ctypes.byref(cache), cache_len,
                          new_pos, next_pos, new_len, FAKE, None, None)


@host_only
def test_revisit_validation_errors():
    rope, mem, cache = good()
    assert call_revisit(rope, None, cache) == 1
    assert call_revisit(rope, mem, cache, p_txt=None) == 1
    assert call_revisit(rope, mem, cache, next_pos=None) == 1
    assert call_revisit(rope, mem, cache, mode=7) == 5
    assert call_revisit(rope, mem, cache, l_ext=-2) == 5
    assert call_revisit(rope, mem, cache, new_pos=FAKE + 4) == 4
    assert call_revisit(rope, mem, cache, new_len=FAKE) == 7
    r2, m2, c2 = good(); m2.coords = None
    assert call_revisit(r2, m2, c2) == 1
    r2, m2, c2 = good(); r2.section[0], r2.section[1] = 32, 8
    assert call_revisit(r2, m2, c2) == 6


@host_only
def test_output_aliasing_refused():
    # The single-launch revisit: one wave per sequence writes next_pos[b] (and the
    # first workgroup the new lengths) while every other wave still reads p_txt,
    # cache_len, the offsets and the visual counts.  Outputs sharing any byte with
    # those inputs, or with each other, are refused before any HIP call.  The
    # inputs here sit at FAKE (batch 2: 8 bytes each, 12 for the offsets).
    rope, mem, cache = good()
    P = FAKE + 0x400
    assert call_revisit(rope, mem, cache, p_txt=P, next_pos=P) == 7          # in-place p_txt
    assert call_revisit(rope, mem, cache, p_txt=P, next_pos=P + 4) == 7      # partial overlap
    assert call_revisit(rope, mem, cache, p_txt=P, next_pos=P - 4) == 7
    assert call_revisit(rope, mem, cache, next_pos=FAKE + 4) == 7            # cache_len, offsets
    assert call_revisit(rope, mem, cache, p_txt=P, new_len=P) == 7           # lengths over p_txt
    assert call_revisit(rope, mem, cache, next_pos=FAKE + 0x300, new_len=FAKE + 0x304) == 7
    assert call_revisit(rope, mem, cache, sel_off=FAKE + 0x300, cache_len=FAKE + 0x300,
                        p_txt=FAKE + 0x300, new_len=FAKE + 0x308) == 7      # offsets [0x300, 0x30C)
    _, m2, _ = good(); m2.n_visual = FAKE + 0x200                           # visual counts
    assert call_revisit(rope, m2, cache) == 7
    # The two-call path: the lengths must not overlap the old lengths or the
    # offsets; next_pos must not overlap the offsets or the visual counts (a
    # workgroup reads its own p_txt[b] before writing next_pos[b], so next_pos may
    # be p_txt there).
    assert call_rebind(rope, mem, cache, new_len=FAKE + 4) == 7
    assert call_rebind(rope, mem, cache, cache_len=FAKE + 0x300, new_len=FAKE + 8) == 7
    assert call_reassign(mem, next_pos=FAKE) == 7
    assert call_reassign(mem, sel_off=FAKE + 0x300, next_pos=FAKE + 0x308) == 7


@host_only
def test_grid_limits():
    # A launch carries each grid extent as a 32-bit count of work-items.  Problems
    # beyond it are size errors, refused before any HIP call, so these placeholder
    # pointers are never used.
    rope, mem, cache = good()
    assert call_rebind(rope, mem, cache, total_k=1 << 25) == 2
    # reassignment: one workgroup per sequence, 64 threads when at most 64 tokens
    # per sequence are selected, 256 up to 256
    r2, m2, c2 = good(); m2.batch = 1 << 26
    assert call_reassign(m2) == 2
    r2, m2, c2 = good(); m2.batch = 1 << 24
    assert call_reassign(m2, total_k=65 << 24) == 2
    r2, m2, c2 = good(); m2.max_visual = 1 << 26           # four tokens per workgroup
    assert call_store(m2) == 2
    assert call_prefill(rope, mem, cache, s_src=1 << 27) == 2


def call_prefill(rope, mem, cache, layer=0, raw_k=FAKE, raw_v=FAKE, s_src=10, pos=FAKE,
                 n_tokens=FAKE, vis_index=FAKE, write_coords=1, cache_start=FAKE, err=None):
    L = prcr.lib()
    return L.prcr_prefill_capture(ctypes.byref(rope) if rope is not None else None,
                                  ctypes.byref(mem) if mem is not None else None, layer, raw_k,
                                  raw_v, s_src, pos, n_tokens, vis_index, write_coords,
                                  ctypes.byref(cache) if cache is not None else None, cache_start,
                                  err, None)


@host_only
def test_prefill_validation_errors():
    rope, mem, cache = good()
    assert call_prefill(None, mem, cache) == 1
    assert call_prefill(rope, None, cache) == 1
    assert call_prefill(rope, mem, None) == 1
    for arg in ("raw_k", "raw_v", "pos", "n_tokens", "vis_index", "cache_start"):
        assert call_prefill(rope, mem, cache, **{arg: None}) == 1, arg
    assert call_prefill(rope, mem, cache, layer=28) == 2
    assert call_prefill(rope, mem, cache, layer=-1) == 2
    assert call_prefill(rope, mem, cache, s_src=0) == 2
    assert call_prefill(rope, mem, cache, raw_k=FAKE + 8) == 4
    assert call_prefill(rope, mem, cache, pos=FAKE + 2) == 4
    assert call_prefill(rope, mem, cache, err=FAKE + 2) == 4
    r2, m2, c2 = good(); m2.coords = None
    assert call_prefill(r2, m2, c2) == 1                 # coordinates requested, none given
    r2, m2, c2 = good(); m2.v = None
    assert call_prefill(r2, m2, c2) == 1                 # key-only memory without v_slot
    r2, m2, c2 = good(); c2.paged = 1
    assert call_prefill(r2, m2, c2) == 1
    r2, m2, c2 = good(); m2.head_dim = 64
    assert call_prefill(r2, m2, c2) == 2
    r2, m2, c2 = good(); r2.section[0], r2.section[1] = 32, 8
    assert call_prefill(r2, m2, c2) == 6


def call_decode(rope, cache, dtype=1, batch=2, n_layers=28, n_kv=4, layer=0, q=FAKE, n_q=16,
                q_pos=FAKE, cache_len=FAKE, scale=0.088, out=FAKE, ws=FAKE, ws_bytes=1 << 30,
                err=None):
    L = prcr.lib()
    return L.prcr_decode_attention(ctypes.byref(rope) if rope is not None else None,
                                   ctypes.byref(cache) if cache is not None else None, dtype,
                                   batch, n_layers, n_kv, layer, q, n_q, q_pos, cache_len, scale,
                                   out, ws, ws_bytes, err, None)


@host_only
def test_decode_validation_errors():
    rope, _, cache = good()
    assert call_decode(None, cache) == 1
    assert call_decode(rope, None) == 1
    for arg in ("q", "q_pos", "cache_len", "out", "ws"):
        assert call_decode(rope, cache, **{arg: None}) == 1, arg
    assert call_decode(rope, cache, dtype=5) == 3
    assert call_decode(rope, cache, batch=0) == 2
    assert call_decode(rope, cache, n_q=6) == 2             # not a multiple of the KV heads
    assert call_decode(rope, cache, n_q=36) == 2            # 9 query heads per KV head
    assert call_decode(rope, cache, layer=28) == 2
    assert call_decode(rope, cache, scale=float("nan")) == 2
    assert call_decode(rope, cache, ws_bytes=16) == 2       # workspace too small
    assert call_decode(rope, cache, q=FAKE + 8) == 4
    assert call_decode(rope, cache, out=FAKE + 2) == 4
    r2, _, c2 = good(); r2.head_dim = 96; r2.section[0], r2.section[1], r2.section[2] = 16, 16, 16
    assert call_decode(r2, c2) == 6                         # head_dim without a kernel
    r2, _, c2 = good(); c2.paged = 1
    assert call_decode(r2, c2) == 2                         # paged with zero sizes
    r2, _, c2 = good(); c2.paged, c2.block_size, c2.max_blocks, c2.n_blocks = 1, 16, 4, 8
    assert call_decode(r2, c2) == 1                         # paged without a block table
    r2, _, c2 = good(); c2.s_max = (1 << 30) + 1
    assert call_decode(r2, c2) == 2                         # capacity above 2^30 slots
    r2, _, c2 = good(); c2.paged, c2.block_table = 1, FAKE
    c2.block_size, c2.max_blocks, c2.n_blocks = 1 << 16, (1 << 14) + 1, 8
    assert call_decode(r2, c2) == 2


def call_decode_static(rope, cache, dtype=1, batch=2, n_layers=28, n_kv=4, layer=0, q=FAKE,
                       n_q=16, q_pos=FAKE, cache_len=FAKE, scale=0.088, out=FAKE, err=None):
    L = prcr.lib()
    return L.prcr_decode_attention_static(ctypes.byref(rope) if rope is not None else None,
                                          ctypes.byref(cache) if cache is not None else None,
                                          dtype, batch, n_layers, n_kv, layer, q, n_q, q_pos,
                                          cache_len, scale, out, err, None)


@host_only
def test_decode_static_validation_errors():
    # The same host checks as prcr_decode_attention, all before any HIP call; a
    # shape whose split-K partials exceed the static buffer is PRCR_ERR_SCRATCH.
    rope, _, cache = good()
    assert call_decode_static(None, cache) == 1
    assert call_decode_static(rope, None) == 1
    for arg in ("q", "q_pos", "cache_len", "out"):
        assert call_decode_static(rope, cache, **{arg: None}) == 1, arg
    assert call_decode_static(rope, cache, dtype=5) == 3
    assert call_decode_static(rope, cache, batch=0) == 2
    assert call_decode_static(rope, cache, n_q=36) == 2
    assert call_decode_static(rope, cache, layer=28) == 2
    assert call_decode_static(rope, cache, q=FAKE + 8) == 4
    # 65535 sequences x 32 query heads x (128 + 2) floats: about 1 GB of partials
    n = ctypes.c_size_t(0)
    assert prcr.lib().prcr_decode_workspace_size(ctypes.byref(cache), 65535, 32, 4, 128,
                                                 ctypes.byref(n)) == 0
    assert n.value > prcr.binding.STATIC_SCRATCH_BYTES
    assert call_decode_static(rope, cache, batch=65535, n_q=32) == 9


def test_decode_workspace_size():
    L = prcr.lib()
    _, _, cache = good()
    n = ctypes.c_size_t(0)
    assert L.prcr_decode_workspace_size(ctypes.byref(cache), 2, 16, 4, 128, ctypes.byref(n)) == 0
    # [batch][query heads][splits][head_dim + 2] floats, whole splits
    per_split = 2 * 16 * (128 + 2) * 4
    assert n.value > 0 and n.value % per_split == 0
    assert L.prcr_decode_workspace_size(ctypes.byref(cache), 2, 16, 4, 128, None) == 1
    assert L.prcr_decode_workspace_size(ctypes.byref(cache), 2, 16, 4, 100, ctypes.byref(n)) == 6
    assert L.prcr_decode_workspace_size(None, 2, 16, 4, 128, ctypes.byref(n)) == 1
