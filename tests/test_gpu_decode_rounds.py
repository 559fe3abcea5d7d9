"""GPU parity of decode attention where one workgroup takes a whole sequence
(one split per sequence and KV head: batch x KV heads at least the number of
workgroups the library aims for) and a wave takes more than 64 tiles of 16 keys,
so that paged caches read their block-table entries in several rounds: contiguous
caches, paged caches whose blocks are whole tiles (16, 48) and paged caches read
an entry per key (8, 24), with 4 and 8 query heads per KV head.  The oracle checks
every long sequence and a sample of the short ones.  Tolerance as in
test_gpu_attention.py."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, to_dev

pytestmark = pytest.mark.gpu

# (paged, block size, batch, KV heads, G, lengths of the long sequences)
CASES = [(False, 0, 96, 8, 4, (4500, 4161)),
         (False, 0, 64, 8, 8, (4300,)),
         (True, 16, 192, 4, 4, (4100, 8300, 12400)),
         (True, 48, 192, 4, 4, (9000,)),
         (True, 8, 192, 4, 4, (4400, 8200)),
         (True, 24, 96, 8, 4, (5000,))]


@pytest.mark.parametrize("paged,bs,B,H,G,longs", CASES)
def test_decode_one_split_long_sequences(paged, bs, B, H, G, longs):
    D, NL, layer = 128, 1, 0
    rng = np.random.default_rng(B + H + G + bs)
    lens = rng.integers(0, 300, B).astype(np.int32)
    long_at = rng.choice(B, len(longs), replace=False)
    lens[long_at] = longs
    cap = int(max(longs))
    g = torch.Generator().manual_seed(int(cap + bs))
    rnd = lambda *s: torch.randn(s, generator=g).to(torch.bfloat16)
    if paged:
        need = (lens + bs - 1) // bs
        max_blocks = int(need.max())
        n_blocks = int(need.sum()) + 1
        perm = 1 + rng.permutation(n_blocks - 1)
        table = np.zeros((B, max_blocks), np.int32)
        o = 0
        for b in range(B):
            table[b, :need[b]] = perm[o:o + need[b]]
            o += need[b]
        k, v = rnd(NL, n_blocks, bs, H, D), rnd(NL, n_blocks, bs, H, D)
        cache_o = {"paged": True, "block_size": bs, "block_table": table, "max_blocks": max_blocks,
                   "n_blocks": n_blocks}
        cache = prcr.Cache(k.to(DEV), v.to(DEV), to_dev(table))
    else:
        k, v = rnd(B, NL, H, cap, D), rnd(B, NL, H, cap, D)
        cache_o = {"paged": False, "s_max": cap}
        cache = prcr.Cache(k.to(DEV), v.to(DEV))
    n_split = prcr.decode_workspace_bytes(cache, B, H * G) // (B * H * G * (D + 2) * 4)
    assert n_split == 1, n_split
    q = rnd(B, H * G, D)
    q_pos = rng.integers(0, 20000, B).astype(np.int32)
    print(f"decode, one split: paged={paged} block {bs}, {B} x {H} KV heads, G={G}, "
          f"long sequences {list(longs)}", flush=True)
    rope = prcr.Rope(D, (16, 24, 24), False, 1e6)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = prcr.decode_attention(rope, cache, layer, q.to(DEV), to_dev(q_pos), to_dev(lens), err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    out = out.cpu().numpy()
    sel = np.unique(np.concatenate([long_at, rng.choice(B, 6, replace=False)]))
    ko, vo = workloads.as_numpy_storage(k), workloads.as_numpy_storage(v)
    if paged:
        sub = dict(cache_o, block_table=table[sel], k=ko, v=vo)
    else:
        sub = dict(cache_o, k=ko[sel], v=vo[sel])
    ref = oracle.decode_attention(rope.__dict__ | {"sections": rope.sections}, sub, layer,
                                  workloads.as_numpy_storage(q)[sel], q_pos[sel], lens[sel],
                                  D ** -0.5, "bf16")
    for i, b in enumerate(sel):
        n = int(lens[b])
        for kvh in range(H):
            vmax = np.abs(oracle.storage_to_f64(oracle.cache_rows(sub, layer, i, kvh, n, "v"),
                                                "bf16")).max() if n else 0.0
            for gg in range(G):
                qh = kvh * G + gg
                d = np.abs(out[b, qh] - ref[i, qh]).max()
                assert d <= 5e-5 * vmax + 1e-6, (int(b), qh, n, d, vmax)
