"""Plain CPU oracle for PRCR position-rebinding cache reuse.

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct reference
that the GPU path is checked against.  Only the test suite, the package smoke
check and the CPU-baseline leg of the benchmark may import it; the product path
never calls it and shares no code with it.

What it computes (Position Rebinding Cache Reuse, Sec. 3 and Algorithm 1):

* ``store_raw``        - Raw Visual Evidence Memory capture, Eq. (6)-(7).
* ``prefill_capture``  - one prefill layer: rotated keys and values into the
                         standard cache (Eq. (4)) and raw visual rows into the
                         memory (Eq. (6)-(7)).
* ``reassign``         - Position-Consistent Reinsertion, Eq. (8)-(10), plus the
                         other reinsertion rules named in Sec. 3.2 / Table 2.
* ``rotate_keys``      - RoPE rebinding of the raw keys at the new coordinates,
                         Eq. (12) (keys) with Eq. (4)'s rotation convention.
* ``decode_attention`` - one decode step of attention over the active cache,
                         Eq. (14), with the query at a text position.
* ``rebind_inject``    - gather of the selected memory rows (Eq. (11)), key
                         rebinding and value reuse (Eq. (12)), concatenation into
                         the active cache (Eq. (13)), next text position.

Precision: every floating-point step runs in float64; the only roundings are
(a) the reassigned position, kept as the correctly rounded float64 value of the
exact rational Eq. (10) defines, and (b) one final round-to-nearest-even into the
storage dtype (float32, or bfloat16 held as uint16 bit patterns).

Readings where the paper is silent (each one is a documented choice):

* R1  Eq. (8)-(10) are applied to all three M-RoPE axes (t, h, w) alike; text
      positions are (p, p, p).
* R2  An axis whose selected range is empty (p_max == p_min) uses u = 1/2, the
      centre of the reinsertion interval (Eq. (10) gives the same for K = 1).
* R3  ``p_txt`` is the position of the latest text token; the next text position
      under PCR is p_txt + 1.
* R5  LPA: p_j = p_txt + j, next = p_txt + K + 1.  UIR: p_j = p_txt + j/(K+1),
      next = p_txt + 1 (j = 1..K in selection order, all axes equal).
* R8  Rotary pairs are (x_i, x_{i+d/2}); inv_freq_i = theta^(-2i/d); pair i
      takes its position from axis(i) given by contiguous sections [s_t, s_h, s_w]
      or, when interleaved, h for i % 3 == 1 and i < 3 s_h, w for i % 3 == 2 and
      i < 3 s_w, t otherwise.
* SHIFT (second mode): p_a = (p_txt + 1) + (c_a - min_a), next = max p + 1.
* IDENTITY (direct reuse, Eq. (4)): p = original coordinates, next = p_txt + 1.

Parity unpinned: no value printed in the paper fixes the readings R1 (t axis), R2
(degenerate axis), the SHIFT next position and R5 (LPA, UIR); their tests pin them to
the readings above, not to the paper.

Layouts (all row-major, shared with the C ABI):
  memory K/V      [B][M_max][NL][H][D]   (per visual token, its per-layer rows)
  coords          [B][M_max][3] int32    (t, h, w)
  contiguous cache[B][NL][H][S_max][D]
  paged cache     [NL][n_blocks][block_size][H][D], block_table [B][max_blocks]
  slot_mapping    int64: contiguous b*S_max + s, paged block*block_size + offset
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

MODES = ("pcr", "shift", "identity", "lpa", "uir", "pcr_right")

# Error bits reported through the err word (bitwise OR of these).
ERR_INDEX = 1      # selected index outside [0, n_visual[b])
ERR_CAPACITY = 2   # slot beyond the cache capacity (S_max, or max_blocks * block_size)
ERR_BLOCK = 4      # block table entry outside [0, n_blocks)

BF16_MAX = float.fromhex("0x1.fep127")   # (2 - 2^-7) * 2^127


# --------------------------------------------------------------------------
# Rotary tables
# --------------------------------------------------------------------------
def inv_freq(theta: float, head_dim: int) -> np.ndarray:
    """RoPE frequencies theta^(-2i/d), i = 0..d/2-1, in float64 (reading R8)."""
    P = head_dim // 2
    return np.array([float(theta) ** (-(2.0 * i) / head_dim) for i in range(P)],
                    dtype=np.float64)


def pair_axis(head_dim: int, sections, interleaved: bool) -> np.ndarray:
    """Axis (0 = t, 1 = h, 2 = w) that rotary pair i takes its position from (R8)."""
    P = head_dim // 2
    s_t, s_h, s_w = (int(s) for s in sections)
    if s_t + s_h + s_w != P:
        raise ValueError("sections must sum to head_dim / 2")
    axis = np.zeros(P, dtype=np.int64)
    for i in range(P):
        if interleaved:
            if i % 3 == 1 and i < 3 * s_h:
                axis[i] = 1
            elif i % 3 == 2 and i < 3 * s_w:
                axis[i] = 2
            else:
                axis[i] = 0
        else:
            if i < s_t:
                axis[i] = 0
            elif i < s_t + s_h:
                axis[i] = 1
            else:
                axis[i] = 2
    return axis


# --------------------------------------------------------------------------
# Position reassignment, Sec. 3.2
# --------------------------------------------------------------------------
def reassign(coords_sel, p_txt: int, mode: str = "pcr", l_ext: int = 2, valid=None):
    """Reassigned positions for one sequence's selected tokens.

    coords_sel: int [K, 3] original (t, h, w) of the selected tokens in selection
    order.  valid: optional bool [K]; invalid tokens are left out of the range
    computation and get NaN positions.  Returns (new_pos float64 [K, 3], next_pos).
    """
    if mode not in MODES:
        raise ValueError(mode)
    c = np.asarray(coords_sel, dtype=np.int64).reshape(-1, 3)
    K = c.shape[0]
    ok = np.ones(K, dtype=bool) if valid is None else np.asarray(valid, dtype=bool)
    out = np.full((K, 3), np.nan, dtype=np.float64)
    p_txt = int(p_txt)
    L = int(l_ext)

    if mode == "identity":                       # direct reuse, Eq. (4)
        for j in range(K):
            if ok[j]:
                out[j] = c[j].astype(np.float64)
        return out, p_txt + 1

    if mode == "lpa":                            # reading R5
        for j in range(K):
            if ok[j]:
                out[j] = float(p_txt + j + 1)
        return out, p_txt + K + 1

    if mode == "uir":                            # reading R5
        for j in range(K):
            if ok[j]:
                out[j] = float(p_txt + Fraction(j + 1, K + 1))
        return out, p_txt + 1

    # Eq. (8): per-axis range over the selected subset.
    lo = [None, None, None]
    hi = [None, None, None]
    for a in range(3):
        vals = [int(c[j, a]) for j in range(K) if ok[j]]
        if vals:
            lo[a], hi[a] = min(vals), max(vals)

    if mode == "shift":
        top = None
        for j in range(K):
            if not ok[j]:
                continue
            for a in range(3):
                v = (p_txt + 1) + (int(c[j, a]) - lo[a])
                out[j, a] = float(v)
                top = v if top is None else max(top, v)
        return out, (p_txt + 1 if top is None else top + 1)

    # PCR, Eq. (9)-(10), exact rational arithmetic, one rounding to float64.  The
    # interval starts at p_txt - L (leftward, the paper's default) or, re-anchored
    # rightward (reading R6), at p_txt + 1.
    start = p_txt + 1 if mode == "pcr_right" else p_txt - L
    for j in range(K):
        if not ok[j]:
            continue
        for a in range(3):
            if hi[a] > lo[a]:
                u = Fraction(int(c[j, a]) - lo[a], hi[a] - lo[a])       # Eq. (9)
            else:
                u = Fraction(1, 2)                                        # R2
            p = start + (L + 1) * (1 + (K - 1) * u) / Fraction(K + 1)     # Eq. (10)
            out[j, a] = float(p)
    return out, p_txt + 1


def reassign_batch(coords, n_visual, sel_off, sel_idx, p_txt, mode="pcr", l_ext=2):
    """Batched reassignment over a CSR selection.

    Returns (new_pos float64 [total_k, 3], next_pos int64 [B], err int)."""
    coords = np.asarray(coords)
    sel_off = np.asarray(sel_off, dtype=np.int64)
    sel_idx = np.asarray(sel_idx, dtype=np.int64)
    B = len(sel_off) - 1
    new_pos = np.full((len(sel_idx), 3), np.nan, dtype=np.float64)
    next_pos = np.zeros(B, dtype=np.int64)
    err = 0
    for b in range(B):
        s0, s1 = int(sel_off[b]), int(sel_off[b + 1])
        idx = sel_idx[s0:s1]
        valid = (idx >= 0) & (idx < int(n_visual[b]))
        if not valid.all():
            err |= ERR_INDEX
        c = np.zeros((s1 - s0, 3), dtype=np.int64)
        c[valid] = coords[b, idx[valid]]
        pos, nxt = reassign(c, int(p_txt[b]), mode, l_ext, valid)
        new_pos[s0:s1] = pos
        next_pos[b] = nxt
    return new_pos, next_pos, err


# --------------------------------------------------------------------------
# Key rebinding, Eq. (12)
# --------------------------------------------------------------------------
def rotate_keys(x, pos, invf, axis):
    """RoPE of raw keys x [..., D] at positions pos [..., 3] (float64 throughout).

    Pair i = (x_i, x_{i+D/2}) is rotated by the angle pos[axis(i)] * invf[i]:
      y_i       = x_i cos - x_{i+D/2} sin
      y_{i+D/2} = x_{i+D/2} cos + x_i sin
    """
    x = np.asarray(x, dtype=np.float64)
    pos = np.asarray(pos, dtype=np.float64)
    P = x.shape[-1] // 2
    ang = pos[..., axis] * invf            # [..., P]
    c, s = np.cos(ang), np.sin(ang)
    lo, hi = x[..., :P], x[..., P:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


# --------------------------------------------------------------------------
# Storage dtypes
# --------------------------------------------------------------------------
def bf16_bits_to_f64(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    with np.errstate(invalid="ignore"):
        return b.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(y) -> np.ndarray:
    """Round float64 to the nearest bfloat16, ties to even; returns uint16 bits.

    A bfloat16 number has 8 significant bits, so inside [2^(e-1), 2^e) its
    spacing is 2^(e-8) (never below the subnormal spacing 2^-133).  Scaling by
    that power of two is exact, np.rint rounds half to even on the scaled
    significand, and scaling back is exact.  NaN maps to 0x7FC0.
    """
    y = np.asarray(y, dtype=np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        _, e = np.frexp(y)
        q = np.maximum(e - 8, -133)
        r = np.ldexp(np.rint(np.ldexp(y, -q)), q)
        r = np.where(np.abs(r) > BF16_MAX, np.copysign(np.inf, y), r)
        bits = (r.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    bits = np.where(np.isnan(y), np.uint16(0x7FC0), bits)
    return bits.astype(np.uint16)


def storage_to_f64(a, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def f64_to_storage(y, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return f64_to_bf16_bits(y)
    if dtype == "f32":
        with np.errstate(over="ignore"):      # beyond the float32 range: +-inf, as IEEE rounds
            return np.asarray(y, dtype=np.float64).astype(np.float32)
    raise ValueError(dtype)


# --------------------------------------------------------------------------
# Raw Visual Evidence Memory capture, Eq. (6)-(7)
# --------------------------------------------------------------------------
def store_raw(mem_k, mem_v, layer, raw_k, raw_v, vis_rows, n_visual):
    """Copy layer ``layer``'s pre-RoPE rows of the visual tokens into the memory.

    raw_k/raw_v: [B][S_src][H][D] projections of one layer; vis_rows [B][M_max]
    gives the source row of visual token m.  Returns (mem_k, mem_v, err) as new
    arrays; rows whose source index is outside [0, S_src) are skipped with
    ERR_INDEX.  A key-only memory (mem_v None) stores keys only: its values stay
    in the standard cache, where Eq. (4) put them unrotated.
    """
    mem_k = np.array(mem_k, copy=True)
    mem_v = None if mem_v is None else np.array(mem_v, copy=True)
    B, S_src = raw_k.shape[0], raw_k.shape[1]
    err = 0
    for b in range(B):
        for m in range(int(n_visual[b])):
            r = int(vis_rows[b, m])
            if r < 0 or r >= S_src:
                err |= ERR_INDEX
                continue
            mem_k[b, m, layer] = raw_k[b, r]
            if mem_v is not None:
                mem_v[b, m, layer] = raw_v[b, r]
    return mem_k, mem_v, err


# --------------------------------------------------------------------------
# Prefill capture fused with rotary: Eq. (4) and Eq. (6)-(7) for one layer
# --------------------------------------------------------------------------
def prefill_capture(rope: dict, mem: dict, layer: int, raw_k, raw_v, pos, n_tokens, vis_index,
                    write_coords: bool, cache: dict, cache_start):
    """One prefill layer: the standard cache gets RoPE(k_raw, p) and v_raw at slot
    cache_start[b] + s (Eq. (4)); visual rows (vis_index[b][s] = m >= 0) also go raw
    into the memory at [b][m][layer] (Eq. (6)-(7)), with their coordinates when
    write_coords.  A key-only memory (mem["v"] None) keeps no values: it records in
    mem["v_slot"][b][m] the cache slot cache_start[b] + s that holds the token's
    value row.  Returns updated copies {mem_k, mem_v, coords, v_slot, k, v, err}."""
    dtype = mem["dtype"]
    D = rope["head_dim"]
    invf = inv_freq(rope["theta"], D)
    axis = pair_axis(D, rope["sections"], rope["interleaved"])
    mk = np.array(mem["k"], copy=True)
    mv = None if mem["v"] is None else np.array(mem["v"], copy=True)
    vs = None if mem.get("v_slot") is None else np.array(mem["v_slot"], copy=True)
    co = np.array(mem["coords"], copy=True)
    ck, cv = np.array(cache["k"], copy=True), np.array(cache["v"], copy=True)
    B, S = raw_k.shape[0], raw_k.shape[1]
    M = mk.shape[1]
    err = 0
    for b in range(B):
        nt = int(n_tokens[b])
        if nt < 0 or nt > S:
            err |= ERR_INDEX
        for s in range(max(0, min(nt, S))):
            p = np.asarray(pos[b, s], dtype=np.float64)
            y = f64_to_storage(rotate_keys(storage_to_f64(raw_k[b, s], dtype), p, invf, axis), dtype)
            slot, where = slot_of(cache, b, int(cache_start[b]) + s)
            if slot is None:
                err |= where
            elif cache["paged"]:
                blk, off = where
                ck[layer, blk, off] = y
                cv[layer, blk, off] = raw_v[b, s]
            else:
                bb, ss = where
                ck[bb, layer, :, ss] = y
                cv[bb, layer, :, ss] = raw_v[b, s]
            m = int(vis_index[b, s])
            if m >= 0:
                if m >= int(mem["n_visual"][b]) or m >= M:
                    err |= ERR_INDEX
                    continue
                mk[b, m, layer] = raw_k[b, s]
                if mv is not None:
                    mv[b, m, layer] = raw_v[b, s]
                elif vs is not None:
                    vs[b, m] = int(cache_start[b]) + s if slot is not None else -1
                if write_coords:
                    co[b, m] = pos[b, s]
    return {"mem_k": mk, "mem_v": mv, "coords": co, "v_slot": vs, "k": ck, "v": cv, "err": err}


# --------------------------------------------------------------------------
# Gather + rebind + inject, Eq. (11)-(13)
# --------------------------------------------------------------------------
def slot_of(cache: dict, b: int, s: int):
    """Destination of logical slot s of sequence b: (slot_id, locator) or an error bit."""
    if cache["paged"]:
        bs = cache["block_size"]
        lb = s // bs
        if lb >= cache["max_blocks"]:
            return None, ERR_CAPACITY
        blk = int(cache["block_table"][b, lb])
        if blk < 0 or blk >= cache["n_blocks"]:
            return None, ERR_BLOCK
        return blk * bs + s % bs, (blk, s % bs)
    if s >= cache["s_max"]:
        return None, ERR_CAPACITY
    return b * cache["s_max"] + s, (b, s)


def rebind_inject(rope: dict, mem: dict, sel_off, sel_idx, new_pos, cache: dict, cache_len):
    """Reference for one rebind-and-inject call.

    rope:  {"head_dim", "sections", "interleaved", "theta"}
    mem:   {"k", "v", "n_visual", "dtype"} with k/v [B][M_max][NL][H][D].  A
           key-only memory has v None and "v_slot" [B][M_max]: token m's value
           rows are those of cache slot v_slot[b][m] of the same sequence, which
           must be one of its cache_len[b] filled slots (else ERR_INDEX).
    cache: {"paged", "k", "v", "s_max" | ("block_table", "block_size",
            "max_blocks", "n_blocks")}
    Returns dict(k, v, slot_mapping, new_cache_len, err); k/v are updated copies.
    """
    dtype = mem["dtype"]
    D = rope["head_dim"]
    invf = inv_freq(rope["theta"], D)
    axis = pair_axis(D, rope["sections"], rope["interleaved"])
    ck = np.array(cache["k"], copy=True)
    cv = np.array(cache["v"], copy=True)
    sel_off = np.asarray(sel_off, dtype=np.int64)
    sel_idx = np.asarray(sel_idx, dtype=np.int64)
    B = len(sel_off) - 1
    slot_mapping = np.full(len(sel_idx), -1, dtype=np.int64)
    new_len = np.zeros(B, dtype=np.int64)
    err = 0
    for b in range(B):
        s0, s1 = int(sel_off[b]), int(sel_off[b + 1])
        new_len[b] = int(cache_len[b]) + (s1 - s0)
        for j in range(s1 - s0):
            g = s0 + j
            m = int(sel_idx[g])
            if m < 0 or m >= int(mem["n_visual"][b]):
                err |= ERR_INDEX
                continue
            if mem["v"] is None:
                vsl = int(mem["v_slot"][b, m])
                if vsl < 0 or vsl >= int(cache_len[b]):
                    err |= ERR_INDEX
                    continue
                src, src_where = slot_of(cache, b, vsl)
                if src is None:
                    err |= src_where
                    continue
            slot, where = slot_of(cache, b, int(cache_len[b]) + j)
            if slot is None:
                err |= where
                continue
            slot_mapping[g] = slot
            x = storage_to_f64(mem["k"][b, m], dtype)                 # [NL][H][D], Eq. (11)
            y = f64_to_storage(rotate_keys(x, new_pos[g], invf, axis), dtype)  # Eq. (12)
            if mem["v"] is not None:                                  # value reuse, Eq. (12)
                vv = mem["v"][b, m]
            elif cache["paged"]:
                vv = np.array(cache["v"][:, src_where[0], src_where[1]], copy=True)
            else:
                vv = np.array(cache["v"][b, :, :, src_where[1]], copy=True)
            if cache["paged"]:                                        # Eq. (13)
                blk, off = where
                ck[:, blk, off] = y
                cv[:, blk, off] = vv
            else:
                bb, s = where
                ck[bb, :, :, s] = y
                cv[bb, :, :, s] = vv
    return {"k": ck, "v": cv, "slot_mapping": slot_mapping,
            "new_cache_len": new_len, "err": err}


def rebind_row(rope: dict, k_row, dtype: str, pos):
    """One raw key row (storage form) rebound at pos [3]: the key half of Eq. (12)."""
    D = rope["head_dim"]
    invf = inv_freq(rope["theta"], D)
    axis = pair_axis(D, rope["sections"], rope["interleaved"])
    return f64_to_storage(rotate_keys(storage_to_f64(k_row, dtype), pos, invf, axis), dtype)


def rebind_entry(rope: dict, mem: dict, b: int, m: int, layer: int, head: int, pos):
    """One rebound key row and its value row (storage dtype), for sampled checks."""
    y = rebind_row(rope, mem["k"][b, m, layer, head], mem["dtype"], pos)
    return y, np.array(mem["v"][b, m, layer, head], copy=True)


# --------------------------------------------------------------------------
# Decode attention over the active cache, Eq. (14)
# --------------------------------------------------------------------------
def cache_rows(cache: dict, layer: int, b: int, kv_head: int, n: int, which: str = "k"):
    """Rows of slots 0..n-1 of sequence b, one layer and KV head (storage form)."""
    t = cache[which]
    if cache["paged"]:
        bs = cache["block_size"]
        return np.stack([t[layer, cache["block_table"][b, s // bs], s % bs, kv_head]
                         for s in range(n)]) if n else t[layer, :0, 0, kv_head]
    return t[b, layer, kv_head, :n]


def decode_attention(rope: dict, cache: dict, layer: int, q, q_pos, cache_len, scale: float,
                     dtype: str):
    """out[b][qh] = softmax(scale * RoPE(q[b][qh], (p, p, p)) . K^T) V over the
    cache_len[b] keys of KV head qh // G (grouped-query attention), in float64;
    an empty cache gives zeros."""
    D = rope["head_dim"]
    invf = inv_freq(rope["theta"], D)
    axis = pair_axis(D, rope["sections"], rope["interleaved"])
    n_kv = cache["k"].shape[3] if cache["paged"] else cache["k"].shape[2]
    B, Hq = q.shape[0], q.shape[1]
    G = Hq // n_kv
    out = np.zeros((B, Hq, D), dtype=np.float64)
    for b in range(B):
        n = int(cache_len[b])
        if n == 0:
            continue
        p = np.full(3, float(q_pos[b]))
        for kvh in range(n_kv):
            K = storage_to_f64(cache_rows(cache, layer, b, kvh, n, "k"), dtype)
            V = storage_to_f64(cache_rows(cache, layer, b, kvh, n, "v"), dtype)
            for g in range(G):
                qh = kvh * G + g
                qr = rotate_keys(storage_to_f64(q[b, qh], dtype), p, invf, axis)
                s = (K @ qr) * scale
                w = np.exp(s - s.max())
                out[b, qh] = (w / w.sum()) @ V
    return out
