"""ctypes binding of libprcr.so (argument marshalling only).

Every step of the rebinding path runs in the HIP library; this module checks
tensor devices/dtypes/shapes, passes raw device pointers and the current HIP
stream, and turns non-OK status codes into exceptions.  Output tensors that the
caller does not provide are allocated here with torch (the library itself never
allocates).
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_int, c_int32, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libprcr.so")

PRCR_F32, PRCR_BF16 = 0, 1
MODES = {"pcr": 0, "shift": 1, "identity": 2, "lpa": 3, "uir": 4, "pcr_right": 5}
DERR_INDEX, DERR_CAPACITY, DERR_BLOCK, DERR_OFFSETS, DERR_RANGE = 1, 2, 4, 8, 16
STATUS = {0: "PRCR_OK", 1: "PRCR_ERR_NULL", 2: "PRCR_ERR_SHAPE", 3: "PRCR_ERR_DTYPE",
          4: "PRCR_ERR_ALIGN", 5: "PRCR_ERR_MODE", 6: "PRCR_ERR_UNSUPPORTED",
          7: "PRCR_ERR_ALIAS", 8: "PRCR_ERR_HIP", 9: "PRCR_ERR_SCRATCH"}
STATIC_SCRATCH_BYTES = 16 << 20     # PRCR_STATIC_SCRATCH_BYTES


class PrcrError(RuntimeError):
    def __init__(self, fn: str, status: int, text: str):
        super().__init__(f"{fn}: {STATUS.get(status, status)} ({text})")
        self.status = status


class CRope(ctypes.Structure):
    _fields_ = [("head_dim", c_int32), ("section", c_int32 * 3), ("interleaved", c_int32),
                ("theta", c_double)]


class CMem(ctypes.Structure):
    _fields_ = [("k", c_void_p), ("v", c_void_p), ("coords", c_void_p), ("n_visual", c_void_p),
                ("batch", c_int32), ("max_visual", c_int32), ("n_layers", c_int32),
                ("n_kv_heads", c_int32), ("head_dim", c_int32), ("dtype", c_int),
                ("v_slot", c_void_p)]


class CCache(ctypes.Structure):
    _fields_ = [("paged", c_int32), ("k", c_void_p), ("v", c_void_p), ("s_max", c_int32),
                ("block_table", c_void_p), ("block_size", c_int32), ("max_blocks", c_int32),
                ("n_blocks", c_int32)]


_LIB = None


def lib() -> ctypes.CDLL:
    """Load libprcr.so from the package directory; raise if it was not built."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(or python paper_2606_26631_amd/build.py); there is no fallback path")
    L = ctypes.CDLL(LIB_PATH)
    L.prcr_status_str.restype = ctypes.c_char_p
    L.prcr_status_str.argtypes = [c_int]
    L.prcr_version.restype = c_int32
    L.prcr_version.argtypes = []
    L.prcr_inv_freq.restype = c_int
    L.prcr_inv_freq.argtypes = [POINTER(CRope), POINTER(c_double)]
    L.prcr_pair_axis.restype = c_int
    L.prcr_pair_axis.argtypes = [POINTER(CRope), POINTER(c_int32)]
    L.prcr_store_raw.restype = c_int
    L.prcr_store_raw.argtypes = [POINTER(CMem), c_int32, c_void_p, c_void_p, c_int32, c_void_p,
                                 c_void_p, c_void_p]
    L.prcr_reassign_coords.restype = c_int
    L.prcr_reassign_coords.argtypes = [POINTER(CMem), c_void_p, c_void_p, c_int32, c_void_p, c_int,
                                       c_int32, c_void_p, c_void_p, c_void_p, c_void_p]
    L.prcr_rebind_inject.restype = c_int
    L.prcr_rebind_inject.argtypes = [POINTER(CRope), POINTER(CMem), c_void_p, c_void_p, c_int32,
                                     c_void_p, POINTER(CCache), c_void_p, c_void_p, c_void_p,
                                     c_void_p, c_void_p]
    L.prcr_prefill_capture.restype = c_int
    L.prcr_prefill_capture.argtypes = [POINTER(CRope), POINTER(CMem), c_int32, c_void_p, c_void_p,
                                       c_int32, c_void_p, c_void_p, c_void_p, c_int32,
                                       POINTER(CCache), c_void_p, c_void_p, c_void_p]
    L.prcr_decode_workspace_size.restype = c_int
    L.prcr_decode_workspace_size.argtypes = [POINTER(CCache), c_int32, c_int32, c_int32, c_int32,
                                             POINTER(ctypes.c_size_t)]
    L.prcr_decode_attention.restype = c_int
    L.prcr_decode_attention.argtypes = [POINTER(CRope), POINTER(CCache), c_int, c_int32, c_int32,
                                        c_int32, c_int32, c_void_p, c_int32, c_void_p, c_void_p,
                                        ctypes.c_float, c_void_p, c_void_p, ctypes.c_size_t, c_void_p,
                                        c_void_p]
    L.prcr_decode_attention_static.restype = c_int
    L.prcr_decode_attention_static.argtypes = [POINTER(CRope), POINTER(CCache), c_int, c_int32,
                                               c_int32, c_int32, c_int32, c_void_p, c_int32,
                                               c_void_p, c_void_p, ctypes.c_float, c_void_p,
                                               c_void_p, c_void_p]
    L.prcr_revisit.restype = c_int
    L.prcr_revisit.argtypes = [POINTER(CRope), POINTER(CMem), c_void_p, c_void_p, c_int32, c_void_p,
                               c_int, c_int32, POINTER(CCache), c_void_p, c_void_p, c_void_p,
                               c_void_p, c_void_p, c_void_p, c_void_p]
    _LIB = L
    return L


def _check(fn: str, status: int):
    if status != 0:
        raise PrcrError(fn, status, lib().prcr_status_str(status).decode())


# ---------------------------------------------------------------------------
# Tensor-level API
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else c_void_p(t.data_ptr())


def _stream(stream, device):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream(device)
    return c_void_p(s.cuda_stream)


def _need(t, name, dtype=None, ndim=None, device=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims (got {t.dim()})")


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.float32:
        return PRCR_F32
    if t.dtype == torch.bfloat16:
        return PRCR_BF16
    raise ValueError(f"unsupported element type {t.dtype} (float32 or bfloat16)")


class Rope:
    """M-RoPE definition: head_dim, (t, h, w) pair sections, interleaving, theta."""

    def __init__(self, head_dim: int, sections, interleaved: bool = False, theta: float = 1e6):
        self.head_dim, self.sections = int(head_dim), tuple(int(s) for s in sections)
        self.interleaved, self.theta = bool(interleaved), float(theta)

    def to_c(self) -> CRope:
        return CRope(self.head_dim, (c_int32 * 3)(*self.sections), int(self.interleaved), self.theta)

    def inv_freq(self):
        out = (c_double * (self.head_dim // 2))()
        _check("prcr_inv_freq", lib().prcr_inv_freq(ctypes.byref(self.to_c()), out))
        return list(out)

    def pair_axis(self):
        out = (c_int32 * (self.head_dim // 2))()
        _check("prcr_pair_axis", lib().prcr_pair_axis(ctypes.byref(self.to_c()), out))
        return list(out)


class Memory:
    """Raw Visual Evidence Memory: k, v [B, M_max, NL, H, D]; coords [B, M_max, 3] int32;
    n_visual [B] int32, all on one GPU.  A key-only memory has v None and v_slot
    [B, M_max] int32: the standard-cache slot holding visual token m's value rows."""

    def __init__(self, k, v, coords, n_visual, v_slot=None):
        torch = _torch()
        _need(k, "mem.k", ndim=5)
        if v is None:
            if v_slot is None:
                raise ValueError("a key-only memory (v None) needs v_slot")
        else:
            _need(v, "mem.v", dtype=k.dtype, ndim=5, device=k.device)
            if v.shape != k.shape:
                raise ValueError("mem.k and mem.v shapes differ")
        _need(coords, "mem.coords", torch.int32, 3, k.device)
        _need(n_visual, "mem.n_visual", torch.int32, 1, k.device)
        B, M = k.shape[0], k.shape[1]
        if tuple(coords.shape) != (B, M, 3) or n_visual.shape[0] != B:
            raise ValueError("coords must be [B, M_max, 3] and n_visual [B]")
        if v_slot is not None:
            _need(v_slot, "mem.v_slot", torch.int32, 2, k.device)
            if tuple(v_slot.shape) != (B, M):
                raise ValueError("v_slot must be [B, M_max]")
        self.k, self.v, self.coords, self.n_visual = k, v, coords, n_visual
        self.v_slot = v_slot
        self.device = k.device

    def to_c(self) -> CMem:
        B, M, NL, H, D = self.k.shape
        return CMem(self.k.data_ptr(), None if self.v is None else self.v.data_ptr(),
                    self.coords.data_ptr(), self.n_visual.data_ptr(), B, M, NL, H, D,
                    _dtype_code(self.k), None if self.v_slot is None else self.v_slot.data_ptr())


class Cache:
    """Active decoder cache, contiguous [B, NL, H, S_max, D] or paged
    [NL, n_blocks, block_size, H, D] with block_table [B, max_blocks] int32."""

    def __init__(self, k, v, block_table=None):
        torch = _torch()
        _need(k, "cache.k", ndim=5)
        _need(v, "cache.v", dtype=k.dtype, ndim=5, device=k.device)
        if v.shape != k.shape:
            raise ValueError("cache.k and cache.v shapes differ")
        if block_table is not None:
            _need(block_table, "cache.block_table", torch.int32, 2, k.device)
        self.k, self.v, self.block_table = k, v, block_table
        self.paged = block_table is not None
        self.device = k.device

    def to_c(self) -> CCache:
        if self.paged:
            NL, nb, bs, H, D = self.k.shape
            return CCache(1, self.k.data_ptr(), self.v.data_ptr(), 0, self.block_table.data_ptr(),
                          bs, self.block_table.shape[1], nb)
        return CCache(0, self.k.data_ptr(), self.v.data_ptr(), self.k.shape[3], None, 0, 0, 0)

    def check_matches(self, mem: Memory):
        B, M, NL, H, D = mem.k.shape
        if self.k.dtype != mem.k.dtype:
            raise ValueError("cache and memory element types differ")
        if self.paged:
            if (self.k.shape[0], self.k.shape[3], self.k.shape[4]) != (NL, H, D):
                raise ValueError("paged cache must be [NL, n_blocks, block_size, H, D]")
            if self.block_table.shape[0] != B:
                raise ValueError("block_table must have one row per sequence")
        elif (self.k.shape[0], self.k.shape[1], self.k.shape[2], self.k.shape[4]) != (B, NL, H, D):
            raise ValueError("contiguous cache must be [B, NL, H, S_max, D]")


def _selection(mem: Memory, sel_off, sel_idx):
    torch = _torch()
    _need(sel_off, "sel_off", torch.int32, 1, mem.device)
    _need(sel_idx, "sel_idx", torch.int32, 1, mem.device)
    if sel_off.shape[0] != mem.k.shape[0] + 1:
        raise ValueError("sel_off must have batch + 1 entries")
    return int(sel_idx.shape[0])


def _overlap(a, b) -> bool:
    """Whether two tensors share any byte of device memory."""
    if a is None or b is None or a.numel() == 0 or b.numel() == 0:
        return False
    x, y = a.data_ptr(), b.data_ptr()
    return x < y + b.numel() * b.element_size() and y < x + a.numel() * a.element_size()


def _no_alias(pairs):
    for (oname, o), (iname, i) in pairs:
        if _overlap(o, i):
            raise ValueError(f"{oname} must not share memory with {iname}")


def _shape(t, name, shape):
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")


def _err(err, device):
    torch = _torch()
    if err is not None:
        _need(err, "err", torch.int32, 1, device)
        if err.shape[0] < 1:
            raise ValueError("err must hold at least one int32")


def store_raw(mem: Memory, layer: int, raw_k, raw_v, vis_rows, err=None, stream=None):
    """Capture one layer's pre-rotary K/V rows of the visual tokens (prcr_store_raw).
    A key-only memory stores keys only (raw_v may be None)."""
    torch = _torch()
    B, M, NL, H, D = mem.k.shape
    _need(raw_k, "raw_k", mem.k.dtype, 4, mem.device)
    if raw_k.shape[0] != B or tuple(raw_k.shape[2:]) != (H, D):
        raise ValueError("raw_k must be [B, S_src, H, D]")
    if mem.v is not None or raw_v is not None:
        _need(raw_v, "raw_v", mem.k.dtype, 4, mem.device)
        if raw_k.shape != raw_v.shape:
            raise ValueError("raw_k/raw_v must be [B, S_src, H, D]")
    _need(vis_rows, "vis_rows", torch.int32, 2, mem.device)
    if tuple(vis_rows.shape) != (B, M):
        raise ValueError("vis_rows must be [B, M_max]")
    _err(err, mem.device)
    st = lib().prcr_store_raw(ctypes.byref(mem.to_c()), int(layer), _ptr(raw_k), _ptr(raw_v),
                              int(raw_k.shape[1]), _ptr(vis_rows), _ptr(err),
                              _stream(stream, mem.device))
    _check("prcr_store_raw", st)


def reassign_coords(mem: Memory, sel_off, sel_idx, p_txt, mode: str = "pcr", l_ext: int = 2,
                    new_pos=None, next_pos=None, err=None, stream=None):
    """New (t, h, w) positions of the selected tokens and next text positions
    (prcr_reassign_coords).  Returns (new_pos [total_k, 3] float64, next_pos [B] int32)."""
    torch = _torch()
    total_k = _selection(mem, sel_off, sel_idx)
    B = mem.k.shape[0]
    _need(p_txt, "p_txt", torch.int32, 1, mem.device)
    _shape(p_txt, "p_txt", (B,))
    if new_pos is None:
        new_pos = torch.empty((total_k, 3), dtype=torch.float64, device=mem.device)
    if next_pos is None:
        next_pos = torch.empty((B,), dtype=torch.int32, device=mem.device)
    _need(new_pos, "new_pos", torch.float64, 2, mem.device)
    _need(next_pos, "next_pos", torch.int32, 1, mem.device)
    _shape(new_pos, "new_pos", (total_k, 3))
    _shape(next_pos, "next_pos", (B,))
    _no_alias([(("next_pos", next_pos), ("sel_off", sel_off)),
               (("next_pos", next_pos), ("mem.n_visual", mem.n_visual))])
    _err(err, mem.device)
    if mode not in MODES:
        raise ValueError(f"mode must be one of {sorted(MODES)}")
    st = lib().prcr_reassign_coords(ctypes.byref(mem.to_c()), _ptr(sel_off), _ptr(sel_idx), total_k,
                                    _ptr(p_txt), MODES[mode], int(l_ext), _ptr(new_pos),
                                    _ptr(next_pos), _ptr(err), _stream(stream, mem.device))
    _check("prcr_reassign_coords", st)
    return new_pos, next_pos


def rebind_inject(rope: Rope, mem: Memory, sel_off, sel_idx, new_pos, cache: Cache, cache_len,
                  new_cache_len=None, slot_mapping=None, err=None, stream=None):
    """Gather, rotate keys at new_pos, copy values and append to the cache
    (prcr_rebind_inject).  Returns (new_cache_len [B] int32, slot_mapping [total_k] int64)."""
    torch = _torch()
    total_k = _selection(mem, sel_off, sel_idx)
    B = mem.k.shape[0]
    cache.check_matches(mem)
    _need(new_pos, "new_pos", torch.float64, 2, mem.device)
    _need(cache_len, "cache_len", torch.int32, 1, mem.device)
    _shape(new_pos, "new_pos", (total_k, 3))
    _shape(cache_len, "cache_len", (B,))
    if new_cache_len is None:
        new_cache_len = torch.empty((B,), dtype=torch.int32, device=mem.device)
    if slot_mapping is None:
        slot_mapping = torch.empty((total_k,), dtype=torch.int64, device=mem.device)
    _need(new_cache_len, "new_cache_len", torch.int32, 1, mem.device)
    _need(slot_mapping, "slot_mapping", torch.int64, 1, mem.device)
    _shape(new_cache_len, "new_cache_len", (B,))
    _shape(slot_mapping, "slot_mapping", (total_k,))
    _no_alias([(("new_cache_len", new_cache_len), ("cache_len", cache_len)),
               (("new_cache_len", new_cache_len), ("sel_off", sel_off))])
    _err(err, mem.device)
    st = lib().prcr_rebind_inject(ctypes.byref(rope.to_c()), ctypes.byref(mem.to_c()), _ptr(sel_off),
                                  _ptr(sel_idx), total_k, _ptr(new_pos), ctypes.byref(cache.to_c()),
                                  _ptr(cache_len), _ptr(new_cache_len), _ptr(slot_mapping), _ptr(err),
                                  _stream(stream, mem.device))
    _check("prcr_rebind_inject", st)
    return new_cache_len, slot_mapping


def revisit(rope: Rope, mem: Memory, sel_off, sel_idx, p_txt, cache: Cache, cache_len,
            mode: str = "pcr", l_ext: int = 2, new_pos=None, next_pos=None, new_cache_len=None,
            slot_mapping=None, err=None, stream=None, store_positions: bool = True):
    """Reassignment + rebinding + injection in one launch (prcr_revisit).

    Returns (new_pos or None, next_pos, new_cache_len, slot_mapping)."""
    torch = _torch()
    total_k = _selection(mem, sel_off, sel_idx)
    B = mem.k.shape[0]
    cache.check_matches(mem)
    _need(p_txt, "p_txt", torch.int32, 1, mem.device)
    _need(cache_len, "cache_len", torch.int32, 1, mem.device)
    _shape(p_txt, "p_txt", (B,))
    _shape(cache_len, "cache_len", (B,))
    if new_pos is None and store_positions:
        new_pos = torch.empty((total_k, 3), dtype=torch.float64, device=mem.device)
    if new_pos is not None:
        _need(new_pos, "new_pos", torch.float64, 2, mem.device)
        _shape(new_pos, "new_pos", (total_k, 3))
    if next_pos is None:
        next_pos = torch.empty((B,), dtype=torch.int32, device=mem.device)
    if new_cache_len is None:
        new_cache_len = torch.empty((B,), dtype=torch.int32, device=mem.device)
    if slot_mapping is None:
        slot_mapping = torch.empty((total_k,), dtype=torch.int64, device=mem.device)
    _need(next_pos, "next_pos", torch.int32, 1, mem.device)
    _need(new_cache_len, "new_cache_len", torch.int32, 1, mem.device)
    _need(slot_mapping, "slot_mapping", torch.int64, 1, mem.device)
    _shape(next_pos, "next_pos", (B,))
    _shape(new_cache_len, "new_cache_len", (B,))
    _shape(slot_mapping, "slot_mapping", (total_k,))
    # Every wave of the single launch reads p_txt, cache_len, the offsets and the
    # visual counts while some waves write next_pos and the new lengths.
    _no_alias([(("next_pos", next_pos), ("p_txt", p_txt)),
               (("next_pos", next_pos), ("cache_len", cache_len)),
               (("next_pos", next_pos), ("sel_off", sel_off)),
               (("next_pos", next_pos), ("mem.n_visual", mem.n_visual)),
               (("next_pos", next_pos), ("new_cache_len", new_cache_len)),
               (("new_cache_len", new_cache_len), ("cache_len", cache_len)),
               (("new_cache_len", new_cache_len), ("sel_off", sel_off)),
               (("new_cache_len", new_cache_len), ("p_txt", p_txt))])
    _err(err, mem.device)
    if mode not in MODES:
        raise ValueError(f"mode must be one of {sorted(MODES)}")
    st = lib().prcr_revisit(ctypes.byref(rope.to_c()), ctypes.byref(mem.to_c()), _ptr(sel_off),
                            _ptr(sel_idx), total_k, _ptr(p_txt), MODES[mode], int(l_ext),
                            ctypes.byref(cache.to_c()), _ptr(cache_len), _ptr(new_pos),
                            _ptr(next_pos), _ptr(new_cache_len), _ptr(slot_mapping), _ptr(err),
                            _stream(stream, mem.device))
    _check("prcr_revisit", st)
    return new_pos, next_pos, new_cache_len, slot_mapping


def prefill_capture(rope: Rope, mem: Memory, layer: int, raw_k, raw_v, pos, n_tokens, vis_index,
                    cache: Cache, cache_start, write_coords: bool = True, err=None, stream=None):
    """One prefill layer, fused (prcr_prefill_capture): rotated K and V into the cache
    at the prompt's position ids, raw rows of visual tokens into the memory."""
    torch = _torch()
    B, M, NL, H, D = mem.k.shape
    cache.check_matches(mem)
    _need(raw_k, "raw_k", mem.k.dtype, 4, mem.device)
    _need(raw_v, "raw_v", mem.k.dtype, 4, mem.device)
    if raw_k.shape != raw_v.shape or raw_k.shape[0] != B or tuple(raw_k.shape[2:]) != (H, D):
        raise ValueError("raw_k/raw_v must be [B, S_src, H, D]")
    S = raw_k.shape[1]
    _need(pos, "pos", torch.int32, 3, mem.device)
    _shape(pos, "pos", (B, S, 3))
    _need(n_tokens, "n_tokens", torch.int32, 1, mem.device)
    _shape(n_tokens, "n_tokens", (B,))
    _need(vis_index, "vis_index", torch.int32, 2, mem.device)
    _shape(vis_index, "vis_index", (B, S))
    _need(cache_start, "cache_start", torch.int32, 1, mem.device)
    _shape(cache_start, "cache_start", (B,))
    _err(err, mem.device)
    st = lib().prcr_prefill_capture(ctypes.byref(rope.to_c()), ctypes.byref(mem.to_c()), int(layer),
                                    _ptr(raw_k), _ptr(raw_v), int(S), _ptr(pos), _ptr(n_tokens),
                                    _ptr(vis_index), int(bool(write_coords)),
                                    ctypes.byref(cache.to_c()), _ptr(cache_start), _ptr(err),
                                    _stream(stream, mem.device))
    _check("prcr_prefill_capture", st)


def _cache_dims(cache: Cache):
    """(n_layers, n_kv_heads, head_dim) of a cache tensor."""
    if cache.paged:
        NL, _, _, H, D = cache.k.shape
    else:
        _, NL, H, _, D = cache.k.shape
    return NL, H, D


def decode_workspace_bytes(cache: Cache, batch: int, n_q_heads: int) -> int:
    """Bytes of workspace prcr_decode_attention needs (prcr_decode_workspace_size)."""
    NL, H, D = _cache_dims(cache)
    out = ctypes.c_size_t(0)
    _check("prcr_decode_workspace_size",
           lib().prcr_decode_workspace_size(ctypes.byref(cache.to_c()), int(batch), int(n_q_heads),
                                            int(H), int(D), ctypes.byref(out)))
    return int(out.value)


def decode_attention(rope: Rope, cache: Cache, layer: int, q, q_pos, cache_len, scale=None,
                     out=None, workspace=None, err=None, stream=None):
    """One decode step of attention over one layer of the cache (prcr_decode_attention).
    q [B, Hq, D] raw queries; returns out float32 [B, Hq, D]."""
    torch = _torch()
    NL, H, D = _cache_dims(cache)
    _need(q, "q", cache.k.dtype, 3, cache.device)
    B, Hq = q.shape[0], q.shape[1]
    if q.shape[2] != D:
        raise ValueError("q head_dim differs from the cache's")
    if cache.paged and cache.block_table.shape[0] != B:
        raise ValueError("block_table must have one row per sequence")
    if not cache.paged and cache.k.shape[0] != B:
        raise ValueError("contiguous cache batch differs from q's")
    _need(q_pos, "q_pos", torch.int32, 1, cache.device)
    _shape(q_pos, "q_pos", (B,))
    _need(cache_len, "cache_len", torch.int32, 1, cache.device)
    _shape(cache_len, "cache_len", (B,))
    if out is None:
        out = torch.empty((B, Hq, D), dtype=torch.float32, device=cache.device)
    _need(out, "out", torch.float32, 3, cache.device)
    _shape(out, "out", (B, Hq, D))
    need = decode_workspace_bytes(cache, B, Hq)
    if workspace is None:
        workspace = torch.empty((max(need, 4) + 3) // 4, dtype=torch.float32, device=cache.device)
    _need(workspace, "workspace", None, None, cache.device)
    if workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace needs {need} bytes")
    _err(err, cache.device)
    sc = float(D) ** -0.5 if scale is None else float(scale)
    st = lib().prcr_decode_attention(ctypes.byref(rope.to_c()), ctypes.byref(cache.to_c()),
                                     _dtype_code(cache.k), int(B), int(NL), int(H), int(layer),
                                     _ptr(q), int(Hq), _ptr(q_pos), _ptr(cache_len), sc, _ptr(out),
                                     _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     _ptr(err), _stream(stream, cache.device))
    _check("prcr_decode_attention", st)
    return out


def decode_attention_static(rope: Rope, cache: Cache, layer: int, q, q_pos, cache_len, scale=None,
                            out=None, err=None, stream=None):
    """decode_attention whose split-K partials go to the library's static device buffer
    (prcr_decode_attention_static): no workspace, nothing allocated by the library.
    Calls that overlap on one GPU race on that buffer.  q [B, Hq, D] raw queries;
    returns out float32 [B, Hq, D] (allocated here by torch when not given)."""
    torch = _torch()
    NL, H, D = _cache_dims(cache)
    _need(q, "q", cache.k.dtype, 3, cache.device)
    B, Hq = q.shape[0], q.shape[1]
    if q.shape[2] != D:
        raise ValueError("q head_dim differs from the cache's")
    if cache.paged and cache.block_table.shape[0] != B:
        raise ValueError("block_table must have one row per sequence")
    if not cache.paged and cache.k.shape[0] != B:
        raise ValueError("contiguous cache batch differs from q's")
    _need(q_pos, "q_pos", torch.int32, 1, cache.device)
    _shape(q_pos, "q_pos", (B,))
    _need(cache_len, "cache_len", torch.int32, 1, cache.device)
    _shape(cache_len, "cache_len", (B,))
    if out is None:
        out = torch.empty((B, Hq, D), dtype=torch.float32, device=cache.device)
    _need(out, "out", torch.float32, 3, cache.device)
    _shape(out, "out", (B, Hq, D))
    _err(err, cache.device)
    sc = float(D) ** -0.5 if scale is None else float(scale)
    st = lib().prcr_decode_attention_static(ctypes.byref(rope.to_c()), ctypes.byref(cache.to_c()),
                                            _dtype_code(cache.k), int(B), int(NL), int(H),
                                            int(layer), _ptr(q), int(Hq), _ptr(q_pos),
                                            _ptr(cache_len), sc, _ptr(out), _ptr(err),
                                            _stream(stream, cache.device))
    _check("prcr_decode_attention_static", st)
    return out
