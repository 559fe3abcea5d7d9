"""GPU parity of bf16 decode attention (Eq. (14)) on batches that mix lengths: a few
long sequences among short ones (their splits then differ by up to 5x in keys),
single-sequence and many-head batches, empty sequences, whole-tile blocks (16, 48)
and blocks read an entry per key (8), and 1-8 query heads per KV head.  The oracle
checks sampled sequences, every query head; tolerance as in test_gpu_attention.py."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, to_dev

pytestmark = pytest.mark.gpu


# (paged, block size, batch, KV heads, G, lengths: (low, high, long ones))
CASES = [(False, 0, 32, 32, 8, (1100, 1300, (5000, 4500, 6000))),
         (True, 16, 32, 32, 8, (1100, 1300, (5000, 4500, 6000))),
         (False, 0, 2, 1, 1, (2990, 3000, ())),
         (True, 16, 64, 4, 4, (0, 6000, ())),
         (True, 48, 10, 2, 2, (0, 2000, ())),
         (True, 8, 20, 8, 4, (0, 3000, ())),
         (False, 0, 40, 8, 7, (0, 4000, (0, 0)))]


@pytest.mark.parametrize("paged,bs,B,H,G,spec", CASES)
def test_decode_mixed_lengths(paged, bs, B, H, G, spec):
    D = 128
    NL = 1 if B * H > 512 else 2                  # the two large cases: one layer
    layer = NL - 1
    lo, hi, longs = spec
    rng = np.random.default_rng(B * 131 + H * 7 + G + bs)
    lens = rng.integers(lo, hi + 1, B).astype(np.int32)
    long_at = rng.choice(B, len(longs), replace=False) if longs else np.array([], int)
    lens[long_at] = longs
    lens[rng.choice(np.setdiff1d(np.arange(B), long_at))] = 0
    Hq = H * G
    print(f"decode mixed lengths: paged={paged} block {bs}, {B} x {H} KV heads, G={G}, "
          f"lengths {int(lens.min())}-{int(lens.max())}", flush=True)
    g = torch.Generator(device=DEV)
    g.manual_seed(int(B * 1000 + H * 10 + G + bs))
    rnd = lambda *s: torch.randn(s, generator=g, device=DEV).to(torch.bfloat16)
    if paged:
        need = (lens + bs - 1) // bs
        max_blocks = max(int(need.max()), 1)
        n_blocks = int(need.sum()) + 1
        perm = 1 + rng.permutation(n_blocks - 1)
        table = np.full((B, max_blocks), -1, np.int32)
        o = 0
        for b in range(B):
            table[b, :need[b]] = perm[o:o + need[b]]
            o += need[b]
        k, v = rnd(NL, n_blocks, bs, H, D), rnd(NL, n_blocks, bs, H, D)
        cache = prcr.Cache(k, v, to_dev(table))
    else:
        cap = int(lens.max()) + 5
        k, v = rnd(B, NL, H, cap, D), rnd(B, NL, H, cap, D)
        cache = prcr.Cache(k, v)
    q = rnd(B, Hq, D)
    q_pos = rng.integers(0, 20000, B).astype(np.int32)
    rope = prcr.Rope(D, (16, 24, 24), False, 1e6)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q, to_dev(q_pos), to_dev(lens), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    out = out.cpu().numpy()

    # Sampled sequences (the long ones, an empty one, and others at random); the
    # oracle reads only their rows: a sub-cache (contiguous) or sub-pool (paged).
    sel = np.unique(np.concatenate([long_at, np.flatnonzero(lens == 0)[:1],
                                    rng.choice(B, min(B, 5), replace=False)])).astype(int)
    if paged:
        used = table[sel]
        ids = np.unique(used[used >= 0])
        remap = np.full(n_blocks, -1, np.int64)
        remap[ids] = np.arange(len(ids))
        sub_table = np.where(used >= 0, remap[np.maximum(used, 0)], -1).astype(np.int32)
        idx = torch.from_numpy(ids).to(DEV)
        sub = {"paged": True, "block_size": bs, "block_table": sub_table, "max_blocks": max_blocks,
               "n_blocks": max(len(ids), 1),
               "k": workloads.as_numpy_storage(k[:, idx].cpu()),
               "v": workloads.as_numpy_storage(v[:, idx].cpu())}
    else:
        idx = torch.from_numpy(sel).to(DEV)
        sub = {"paged": False, "s_max": cap, "k": workloads.as_numpy_storage(k[idx].cpu()),
               "v": workloads.as_numpy_storage(v[idx].cpu())}
    qs = workloads.as_numpy_storage(q.cpu())[sel]
    ref = oracle.decode_attention(rope.__dict__ | {"sections": rope.sections}, sub, layer, qs,
                                  q_pos[sel], lens[sel], D ** -0.5, "bf16")
    for i, b in enumerate(sel):
        n = int(lens[b])
        for kvh in range(H):
            vmax = np.abs(oracle.storage_to_f64(oracle.cache_rows(sub, layer, i, kvh, n, "v"),
                                                "bf16")).max() if n else 0.0
            for gg in range(G):
                qh = kvh * G + gg
                d = np.abs(out[b, qh] - ref[i, qh]).max()
                assert d <= 5e-5 * vmax + 1e-6, (int(b), qh, float(d), float(vmax))


@pytest.mark.parametrize("paged", [False, True])
def test_decode_batch_order_does_not_matter(paged):
    """The grid's rows take the sequences longest first; a sequence's result must not
    depend on which row takes it.  A permuted batch (queries, positions, lengths and
    cache rows or block-table rows permuted alike) gives the permuted outputs, bit for
    bit."""
    B, H, G, D, NL, layer, bs = 24, 4, 4, 128, 1, 0, 16
    rng = np.random.default_rng(2024 + paged)
    lens = rng.integers(0, 3000, B).astype(np.int32)
    lens[[3, 11]] = (4000, 4000)                  # a tie among the longest
    print(f"decode batch order, paged={paged}: {B} sequences, lengths {lens.min()}-{lens.max()}",
          flush=True)
    g = torch.Generator(device=DEV)
    g.manual_seed(2025 + paged)
    rnd = lambda *s: torch.randn(s, generator=g, device=DEV).to(torch.bfloat16)
    perm = rng.permutation(B)
    q, q_pos = rnd(B, H * G, D), rng.integers(0, 20000, B).astype(np.int32)
    rope = prcr.Rope(D, (16, 24, 24), False, 1e6)
    if paged:
        need = (lens + bs - 1) // bs
        max_blocks, n_blocks = int(need.max()), int(need.sum()) + 1
        pool = 1 + rng.permutation(n_blocks - 1)
        table = np.full((B, max_blocks), -1, np.int32)
        o = 0
        for b in range(B):
            table[b, :need[b]] = pool[o:o + need[b]]
            o += need[b]
        k, v = rnd(NL, n_blocks, bs, H, D), rnd(NL, n_blocks, bs, H, D)
        cache = prcr.Cache(k, v, to_dev(table))
        cache_p = prcr.Cache(k, v, to_dev(table[perm]))
    else:
        cap = int(lens.max())
        k, v = rnd(B, NL, H, cap, D), rnd(B, NL, H, cap, D)
        pi = torch.from_numpy(perm).to(DEV)
        cache = prcr.Cache(k, v)
        cache_p = prcr.Cache(k[pi].contiguous(), v[pi].contiguous())
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q, to_dev(q_pos), to_dev(lens), err=err)
    out_p = prcr.decode_attention(rope, cache_p, layer, q[torch.from_numpy(perm).to(DEV)].contiguous(),
                                  to_dev(q_pos[perm]), to_dev(lens[perm]), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    a = out.cpu().numpy()[perm].view(np.uint32)
    b = out_p.cpu().numpy().view(np.uint32)
    assert np.array_equal(a, b)
