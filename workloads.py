"""Seeded synthetic inputs for the PRCR rebinding path.

Input generation only: index sets, coordinates, cache lengths, block tables and
random tensor contents.  Nothing here computes any step of the method; both the
GPU path and the CPU oracle receive the arrays built here.

Five workloads, shaped like the paper's setting (visual tokens of a Qwen-VL-style
decoder, an attention-driven selection of a relevant region plus scattered picks,
Sec. 2.1 and Eq. (3)).  The paper's own benchmarks (real images from its
evaluation suites) are not available; these synthetic inputs stand in for them.

  1  tiny fp32: 1 seq, 2 layers, 2 KV heads, d 64, sections [8,12,12], theta 1e6,
     16x16 grid, 6x6 sub-grid selected (rows 5-10, cols 3-8), contiguous cache of
     512 with 300 used.
  2  1 seq bf16 (Qwen2.5-VL-7B shape): 28 layers, 4 heads, d 128, [16,24,24],
     36x36 grid, 12x12 region at a seeded origin + 48 extra tokens, K with 4
     outlier channels x8 per (layer, head), cache length 1600 of 2048.
  3  32 seq bf16: 36 layers, 8 heads, d 128, interleaved (i mod 3) sections
     [22,21,21], theta 5e6, 64x32 grid, top-256 of i.i.d. N(0,1) scores, cache
     length U[2500, 4000] of 4256.
  4  video, 8 seq bf16: 28 layers, 4 heads, d 128, [16,24,24], 8 frames of 24x24,
     4 revisits of 1024 tokens from 2-4 consecutive frames with random boxes,
     cache starts at 4736 of 9216.
  5  paged, 64 seq bf16: 28 layers, 4 heads, d 128, [16,24,24], 48x48 grid, 16x16
     region + 256 extra, cache length U[2400, 6000], block size 16, blocks drawn
     from one globally shuffled pool.

``scale="small"`` keeps head_dim, dtype, axis map, grid and selection structure but
uses fewer sequences and layers, so the oracle finishes in seconds.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass, field

import numpy as np


@dataclass
class Workload:
    cfg: int
    name: str
    dtype: str                      # "f32" | "bf16"
    B: int
    NL: int
    H: int
    D: int
    M_max: int
    sections: tuple
    interleaved: bool
    theta: float
    coords: np.ndarray              # int32 [B][M_max][3]
    n_visual: np.ndarray            # int32 [B]
    sel_off: np.ndarray             # int32 [B+1]
    sel_idx: np.ndarray             # int32 [total_k]
    p_txt: np.ndarray               # int32 [B], latest text position
    cache_len: np.ndarray           # int32 [B]
    paged: bool = False
    s_max: int = 0
    block_size: int = 0
    block_table: np.ndarray | None = None   # int32 [B][max_blocks]
    max_blocks: int = 0
    n_blocks: int = 0
    revisits: list = field(default_factory=list)   # [(sel_off, sel_idx)] incl. the first
    decode_between: int = 0         # text tokens decoded between revisits
    outlier_channels: np.ndarray | None = None      # int [NL][H][4] (workload 2)
    seed: int = 0
    mode: str = "pcr"
    l_ext: int = 2

    @property
    def total_k(self) -> int:
        return int(self.sel_off[-1])

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def entries(self) -> int:
        """Rebound (sequence, token, layer, head) rows of one call."""
        return self.total_k * self.NL * self.H

    def algorithmic_bytes(self) -> int:
        """Read K + read V + write K + write V per entry."""
        return self.entries() * 4 * self.D * self.elem_bytes

    def rope(self) -> dict:
        return {"head_dim": self.D, "sections": tuple(self.sections),
                "interleaved": bool(self.interleaved), "theta": float(self.theta)}


def _grid_coords(frames: int, gh: int, gw: int) -> np.ndarray:
    t, h, w = np.meshgrid(np.arange(frames), np.arange(gh), np.arange(gw), indexing="ij")
    return np.stack([t.ravel(), h.ravel(), w.ravel()], axis=1).astype(np.int32)


def _csr(lists) -> tuple[np.ndarray, np.ndarray]:
    off = np.zeros(len(lists) + 1, dtype=np.int32)
    off[1:] = np.cumsum([len(x) for x in lists])
    idx = np.concatenate([np.asarray(x, dtype=np.int32) for x in lists]) if lists else \
        np.zeros(0, np.int32)
    return off, idx.astype(np.int32)


def _region_plus_random(rng, gh, gw, rh, rw, extra):
    h0 = int(rng.integers(0, gh - rh + 1))
    w0 = int(rng.integers(0, gw - rw + 1))
    region = [(h0 + i) * gw + (w0 + j) for i in range(rh) for j in range(rw)]
    rest = np.setdiff1d(np.arange(gh * gw), np.array(region))
    picks = rng.choice(rest, size=extra, replace=False)
    return np.sort(np.concatenate([np.array(region), picks]))


def _paged_tables(rng, lens, k_new, bs):
    need = [(int(l) + k_new + bs - 1) // bs for l in lens]
    n_blocks = int(sum(need))
    pool = rng.permutation(n_blocks).astype(np.int32)
    max_blocks = int(max(need))
    table = np.full((len(lens), max_blocks), -1, dtype=np.int32)
    pos = 0
    for b, n in enumerate(need):
        table[b, :n] = pool[pos:pos + n]
        pos += n
    return table, max_blocks, n_blocks


def make(cfg: int, scale: str = "full", seed: int | None = None) -> Workload:
    """Build workload ``cfg`` (1-5) at ``scale`` "full" or "small"."""
    if scale not in ("full", "small"):
        raise ValueError(scale)
    small = scale == "small"
    seed = 1000 + cfg if seed is None else int(seed)
    rng = np.random.Generator(np.random.PCG64(seed))

    if cfg == 1:
        gh = gw = 16
        coords = _grid_coords(1, gh, gw)[None]
        sel = [h * gw + w for h in range(5, 11) for w in range(3, 9)]
        off, idx = _csr([sel])
        return Workload(1, "tiny-f32", "f32", 1, 2, 2, 64, gh * gw, (8, 12, 12), False, 1e6,
                        coords, np.array([gh * gw], np.int32), off, idx,
                        np.array([299], np.int32), np.array([300], np.int32),
                        s_max=512, revisits=[(off, idx)], seed=seed)

    if cfg == 2:
        gh = gw = 36
        NL, H = (4 if small else 28), 4
        coords = _grid_coords(1, gh, gw)[None]
        sel = _region_plus_random(rng, gh, gw, 12, 12, 48)
        off, idx = _csr([sel])
        outl = np.stack([np.stack([rng.choice(128, 4, replace=False) for _ in range(H)])
                         for _ in range(NL)])
        return Workload(2, "qwen2.5-vl-7b-1seq", "bf16", 1, NL, H, 128, gh * gw,
                        (16, 24, 24), False, 1e6, coords, np.array([gh * gw], np.int32),
                        off, idx, np.array([1599], np.int32), np.array([1600], np.int32),
                        s_max=2048, revisits=[(off, idx)], outlier_channels=outl, seed=seed)

    if cfg == 3:
        gh, gw = 64, 32
        B, NL, H = (3, 3, 8) if small else (32, 36, 8)
        M = gh * gw
        coords = np.broadcast_to(_grid_coords(1, gh, gw), (B, M, 3)).copy()
        sels = []
        for _ in range(B):
            scores = rng.standard_normal(M)
            sels.append(np.sort(np.argsort(-scores, kind="stable")[:256]))
        off, idx = _csr(sels)
        lens = rng.integers(2500, 4001, size=B).astype(np.int32)
        return Workload(3, "32seq-interleaved", "bf16", B, NL, H, 128, M, (22, 21, 21), True,
                        5e6, coords, np.full(B, M, np.int32), off, idx, (lens - 1).astype(np.int32),
                        lens, s_max=4256, revisits=[(off, idx)], seed=seed)

    if cfg == 4:
        frames, gh, gw = 8, 24, 24
        B, NL, H = (2, 3, 4) if small else (8, 28, 4)
        M = frames * gh * gw
        coords = np.broadcast_to(_grid_coords(frames, gh, gw), (B, M, 3)).copy()
        revisits = []
        for _ in range(4):
            sels = []
            for _ in range(B):
                f = int(rng.integers(2, 5))
                t0 = int(rng.integers(0, frames - f + 1))
                side = min(gh, math.ceil(math.sqrt(1.25 * 1024 / f)))
                cand = []
                for t in range(t0, t0 + f):
                    h0 = int(rng.integers(0, gh - side + 1))
                    w0 = int(rng.integers(0, gw - side + 1))
                    cand += [t * gh * gw + (h0 + i) * gw + (w0 + j)
                             for i in range(side) for j in range(side)]
                cand = np.unique(np.array(cand))
                sels.append(np.sort(rng.choice(cand, size=1024, replace=False)))
            revisits.append(_csr(sels))
        off, idx = revisits[0]
        lens = np.full(B, 4736, np.int32)
        return Workload(4, "video-8seq", "bf16", B, NL, H, 128, M, (16, 24, 24), False, 1e6,
                        coords, np.full(B, M, np.int32), off, idx, (lens - 1).astype(np.int32),
                        lens, s_max=9216, revisits=revisits, decode_between=32, seed=seed)

    if cfg == 5:
        gh = gw = 48
        B, NL, H = (3, 3, 4) if small else (64, 28, 4)
        M = gh * gw
        coords = np.broadcast_to(_grid_coords(1, gh, gw), (B, M, 3)).copy()
        sels = [_region_plus_random(rng, gh, gw, 16, 16, 256) for _ in range(B)]
        off, idx = _csr(sels)
        lens = rng.integers(2400, 6001, size=B).astype(np.int32)
        table, max_blocks, n_blocks = _paged_tables(rng, lens, 512, 16)
        return Workload(5, "paged-64seq", "bf16", B, NL, H, 128, M, (16, 24, 24), False, 1e6,
                        coords, np.full(B, M, np.int32), off, idx, (lens - 1).astype(np.int32),
                        lens, paged=True, block_size=16, block_table=table,
                        max_blocks=max_blocks, n_blocks=n_blocks, revisits=[(off, idx)],
                        seed=seed)

    raise ValueError(f"unknown workload {cfg}")


# --------------------------------------------------------------------------
# Tensor contents
# --------------------------------------------------------------------------
def tp_shard(w: Workload, tp: int) -> Workload:
    """One GPU's share of workload w when its KV heads are split over tp GPUs
    (tensor parallelism): the same sequences, selection and caches with H / tp heads."""
    if w.H % tp != 0:
        raise ValueError(f"{w.H} KV heads do not split over {tp} GPUs")
    return dataclasses.replace(w, H=w.H // tp, name=f"{w.name}-tp{tp}-shard")


def one_d(w: Workload) -> Workload:
    """Workload w for a model with plain 1-D rotary positions (InternVL3.5's language
    model: every rotary pair on one axis): the same shapes and selection, each visual
    token's 1-D position m in t, h = w = 0, and the all-t axis map."""
    coords = np.zeros_like(w.coords)
    coords[:, :, 0] = np.arange(w.coords.shape[1], dtype=np.int32)[None, :]
    return dataclasses.replace(w, coords=coords, sections=(w.D // 2, 0, 0), interleaved=False,
                               theta=1e6, name=f"{w.name.split('-')[0]}-1d-rotary")


def with_capacity(w: Workload, s_max: int) -> Workload:
    """Workload w with a contiguous cache of s_max slots per sequence (the same
    sequences, selection and lengths; only the row stride of the cache changes)."""
    if w.paged:
        raise ValueError("the capacity of a paged cache is its block pool")
    need = int((w.cache_len.astype(np.int64) + np.diff(w.sel_off)).max())
    if s_max < need:
        raise ValueError(f"s_max {s_max} is below the {need} slots the revisit needs")
    return dataclasses.replace(w, s_max=int(s_max), name=f"{w.name}-smax{s_max}")


def value_slots(w: Workload) -> np.ndarray:
    """Value-slot table of a key-only memory for workload w, int32 [B][M_max]: the
    prompt is read as up to 64 text tokens followed by the visual tokens, so visual
    token m of sequence b sits at slot prefix + m, below the sequence's filled
    length (entries past n_visual[b] are -1)."""
    M = w.coords.shape[1]
    prefix = int(max(0, min(64, int(np.min(w.cache_len)) - M)))
    out = np.full((w.B, M), -1, np.int32)
    for b in range(w.B):
        n = int(w.n_visual[b])
        out[b, :n] = prefix + np.arange(n)
        assert n == 0 or prefix + n - 1 < int(w.cache_len[b])
    return out


def mem_shape(w: Workload) -> tuple:
    return (w.B, w.M_max, w.NL, w.H, w.D)


def cache_shape(w: Workload) -> tuple:
    if w.paged:
        return (w.NL, w.n_blocks, w.block_size, w.H, w.D)
    return (w.B, w.NL, w.H, w.s_max, w.D)


def _to_storage_torch(x32, dtype):
    """float32 torch tensor -> storage tensor (float32, or bfloat16 by torch's RNE cast)."""
    import torch
    return x32 if dtype == "f32" else x32.to(torch.bfloat16)


def _apply_outliers(w: Workload, k32):
    if w.outlier_channels is None:
        return k32
    for l in range(w.NL):
        for h in range(w.H):
            ch = [int(c) for c in w.outlier_channels[l, h]]
            k32[:, :, l, h, ch] *= 8.0
    return k32


def torch_values(w: Workload, device="cpu", chunk_elems: int = 1 << 28):
    """Seeded memory and pre-existing cache contents as torch tensors on ``device``.

    K, V ~ N(0,1) drawn in float32 (torch generator seeded from the workload seed),
    cast to the storage dtype; workload 2's K gets its outlier channels scaled x8.
    The pre-existing cache is filled with an independent N(0,1) pattern so that any
    stray write is visible.
    """
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(w.seed)
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16

    def randn(shape, outliers=False):
        out = torch.empty(shape, dtype=tdt, device=device)
        flat = out.view(shape[0], -1)
        per = max(1, chunk_elems // max(1, flat.shape[1]))
        for b0 in range(0, shape[0], per):
            b1 = min(shape[0], b0 + per)
            x = torch.randn((b1 - b0,) + tuple(shape[1:]), generator=g, device=device,
                            dtype=torch.float32)
            if outliers:
                x = _apply_outliers(w, x)
            out[b0:b1] = _to_storage_torch(x, w.dtype)
        return out

    return {"mem_k": randn(mem_shape(w), outliers=True), "mem_v": randn(mem_shape(w)),
            "cache_k": randn(cache_shape(w)), "cache_v": randn(cache_shape(w))}


def as_numpy_storage(t):
    """torch tensor -> numpy in the oracle's storage form (float32, or uint16 bits)."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def custom(B=3, NL=2, H=2, D=128, dtype="bf16", sections=(16, 24, 24), interleaved=False,
           theta=1e6, frames=1, gh=12, gw=10, ks=(5, 0, 9), lens=(3, 40, 17), paged=False,
           block_size=16, s_max=None, seed=7, spare_blocks=0) -> Workload:
    """A small workload with explicit per-sequence selection sizes ``ks`` and cache
    lengths ``lens`` (edge cases: empty and single-token selections, ragged row
    counts, odd block sizes).  Selections are sorted random subsets of the grid."""
    rng = np.random.Generator(np.random.PCG64(seed))
    M = frames * gh * gw
    coords = np.broadcast_to(_grid_coords(frames, gh, gw), (B, M, 3)).copy()
    sels = [np.sort(rng.choice(M, size=int(k), replace=False)) for k in ks]
    off, idx = _csr(sels)
    lens = np.asarray(lens, dtype=np.int32)
    kw = dict(revisits=[(off, idx)], seed=seed)
    if paged:
        table, max_blocks, n_blocks = _paged_tables(rng, lens, int(max(ks)), block_size)
        if spare_blocks:
            n_blocks += spare_blocks
        kw.update(paged=True, block_size=block_size, block_table=table, max_blocks=max_blocks,
                  n_blocks=n_blocks)
    else:
        kw.update(s_max=int(s_max if s_max is not None else int(lens.max()) + int(max(ks)) + 3))
    return Workload(0, "custom", dtype, B, NL, H, D, M, tuple(sections), bool(interleaved),
                    float(theta), coords, np.full(B, M, np.int32), off, idx,
                    (lens - 1).astype(np.int32), lens, **kw)


PAPER_MODELS = {
    # Table 3's operating points: decoder shape of the paper's Qwen3-VL models
    # (public configurations: 36 / 64 layers, 8 KV heads, head_dim 128, interleaved
    # M-RoPE [24, 20, 20], theta 5e6); 768 visual tokens per image (24 x 32 grid).
    "qwen3-vl-8b": dict(NL=36, H=8),
    "qwen3-vl-32b": dict(NL=64, H=8),
}


def paper_k(model: str, K: int, seed: int = 2000) -> Workload:
    """One sequence revisiting K of 768 visual tokens at a paper model's cache shape."""
    rng = np.random.Generator(np.random.PCG64(seed + K))
    shape = PAPER_MODELS[model]
    gh, gw = 24, 32
    M = gh * gw
    coords = _grid_coords(1, gh, gw)[None]
    off, idx = _csr([np.sort(rng.choice(M, size=K, replace=False))])
    lens = np.array([1024], np.int32)
    return Workload(6, f"{model}-K{K}", "bf16", 1, shape["NL"], shape["H"], 128, M, (24, 20, 20),
                    True, 5e6, coords, np.array([M], np.int32), off, idx,
                    (lens - 1).astype(np.int32), lens, s_max=1024 + K, revisits=[(off, idx)],
                    seed=seed + K)


def prompt(B=2, n_before=(5, 9), grid=((4, 6), (3, 5)), n_after=(3, 0), frames=(1, 2)):
    """Prompt layout of a multimodal prefill: text, one image (or video) of grid
    (gh, gw) x frames, text.  Position ids follow the M-RoPE convention: a text
    token at p is (p, p, p); the image starts at the current text offset q with
    (q + t, q + h, q + w); text resumes at 1 + the largest image position id.
    Returns pos int32 [B][S][3], vis_index int32 [B][S] (visual index m or -1),
    n_tokens int32 [B], n_visual int32 [B]."""
    rows = []
    for b in range(B):
        gh, gw = grid[b]
        tk = []
        vis = []
        q = 0
        for _ in range(n_before[b]):
            tk.append((q, q, q)); vis.append(-1); q += 1
        m = 0
        top = q
        for t in range(frames[b]):
            for h in range(gh):
                for w in range(gw):
                    tk.append((q + t, q + h, q + w)); vis.append(m); m += 1
                    top = max(top, q + t, q + h, q + w)
        q = top + 1
        for _ in range(n_after[b]):
            tk.append((q, q, q)); vis.append(-1); q += 1
        rows.append((tk, vis, m))
    S = max(len(r[0]) for r in rows)
    pos = np.zeros((B, S, 3), np.int32)
    vis_index = np.full((B, S), -1, np.int32)
    n_tokens = np.zeros(B, np.int32)
    n_visual = np.zeros(B, np.int32)
    for b, (tk, vis, m) in enumerate(rows):
        pos[b, :len(tk)] = tk
        vis_index[b, :len(vis)] = vis
        n_tokens[b] = len(tk)
        n_visual[b] = m
    return pos, vis_index, n_tokens, n_visual
