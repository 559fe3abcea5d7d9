"""GPU parity of prcr_store_raw (Sec. 3.1, Eq. (6)-(7)) against the oracle's copy.

Every byte of the memory is compared, the rows the call must leave alone included (the
memory starts from random bytes).  The shapes span rows of 32 B to 32 KB (up to sixteen
rounds of a wave's loop), a key-only memory, odd and zero visual-token counts (a wave's second
token absent), bad source rows, and the 32-prompt prefill workload at full size, whose
memory is checked whole for sampled sequences.  Each test prints its case before
touching the GPU.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, to_dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _bits(t):
    """A tensor's element bit patterns as unsigned integers (NaN payloads included)."""
    a = workloads.as_numpy_storage(t)
    return a.view(np.uint32) if a.dtype == np.float32 else a


def _random_bits(shape, dtype, g):
    """Random bit patterns of the element type (finite or not: the copy moves bytes)."""
    if dtype == "f32":
        return torch.randint(-2**31, 2**31 - 1, shape, generator=g, dtype=torch.int32).view(torch.float32)
    return torch.randint(-2**15, 2**15 - 1, shape, generator=g, dtype=torch.int16).view(torch.bfloat16)


CASES = [
    # dtype, H, D, B, M, S, NL, key_only
    ("f32", 1, 8, 5, 9, 20, 2, False),      # 32-byte rows
    ("bf16", 3, 64, 6, 17, 40, 3, False),   # 384-byte rows
    ("bf16", 4, 128, 7, 33, 50, 2, False),  # 1 KB
    ("bf16", 8, 128, 9, 65, 80, 3, False),  # 2 KB
    ("f32", 16, 128, 3, 11, 30, 2, False),  # 8 KB: four rounds of the wave's loop
    ("f32", 64, 128, 2, 5, 9, 2, False),    # 32 KB: sixteen rounds
    ("bf16", 8, 128, 5, 21, 40, 2, True),   # key-only memory
    ("f32", 2, 96, 4, 7, 12, 1, True),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-H{c[1]}-D{c[2]}-B{c[3]}-M{c[4]}"
                         + ("-keyonly" if c[7] else ""))
def test_store_raw_shapes(case):
    dtype, H, D, B, M, S, NL, key_only = case
    _say(f"store_raw {dtype} H={H} D={D} B={B} M={M} S={S} NL={NL} key_only={key_only}")
    g = torch.Generator().manual_seed(1000 + H * D + B)
    rng = np.random.default_rng(H * D + B)
    raw_k = _random_bits((B, S, H, D), dtype, g)
    raw_v = _random_bits((B, S, H, D), dtype, g)
    mk = _random_bits((B, M, NL, H, D), dtype, g)
    mv = None if key_only else _random_bits((B, M, NL, H, D), dtype, g)
    vis = np.stack([rng.choice(S, M, replace=False) for _ in range(B)]).astype(np.int32)
    # ragged counts: empty, odd, full, and the rest random
    nvis = rng.integers(0, M + 1, B).astype(np.int32)
    nvis[0] = M
    nvis[1] = 0
    nvis[2 % B] = M - 1 if M % 2 == 0 else M
    if B > 3:
        nvis[3] = 1
    # bad source rows inside the counted range
    bad_b = [b for b in range(B) if nvis[b] > 0][:2]
    vis[bad_b[0], nvis[bad_b[0]] - 1] = S
    if len(bad_b) > 1:
        vis[bad_b[1], 0] = -1
    for b in range(B):
        vis[b, nvis[b]:] = -7            # past the count: never read, no error
    mem = prcr.Memory(mk.to(DEV), None if key_only else mv.to(DEV),
                      torch.zeros((B, M, 3), dtype=torch.int32, device=DEV), to_dev(nvis),
                      to_dev(np.zeros((B, M), np.int32)) if key_only else None)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    rk, rv = raw_k.to(DEV), raw_v.to(DEV)
    order = list(range(NL)) + [0]
    for layer in order:
        prcr.store_raw(mem, layer, rk, None if key_only else rv, to_dev(vis), err=err)
    torch.cuda.synchronize()
    ek = _bits(mk)
    ev = None if key_only else _bits(mv)
    e_all = 0
    for layer in order:
        ek, ev, e = oracle.store_raw(ek, ev, layer, _bits(raw_k), _bits(raw_v), vis, nvis)
        e_all |= e
    assert int(err.item()) == e_all == oracle.ERR_INDEX
    assert np.array_equal(_bits(mem.k), ek)
    if not key_only:
        assert np.array_equal(_bits(mem.v), ev)


def test_store_raw_full_size():
    """The 32-prompt prefill workload (32 x 2,560 rows, up to 2,048 visual tokens in a
    random sorted subset of the rows, 36 layers x 8 KV heads, d 128, bf16) at full size:
    three layers stored, then the whole memory of four sampled sequences against the
    oracle."""
    B, M, S, NL, H, D = 32, 2048, 2560, 36, 8, 128
    layers = (0, 17, 35)
    _say(f"store_raw full size B={B} M={M} S={S} NL={NL} H={H} D={D} bf16, layers {layers}")
    rng = np.random.default_rng(77)
    nvis = rng.integers(1500, M + 1, B).astype(np.int32)
    nvis[:3] = (M, M - 1, 1)
    vis = np.stack([np.sort(rng.choice(S, M, replace=False)) for _ in range(B)]).astype(np.int32)
    g = torch.Generator(device=DEV)
    g.manual_seed(78)
    raws = {}
    mem = prcr.Memory(torch.zeros((B, M, NL, H, D), dtype=torch.bfloat16, device=DEV),
                      torch.zeros((B, M, NL, H, D), dtype=torch.bfloat16, device=DEV),
                      torch.zeros((B, M, 3), dtype=torch.int32, device=DEV), to_dev(nvis))
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    vis_d = to_dev(vis)
    for layer in layers:
        rk = torch.randn((B, S, H, D), generator=g, device=DEV).to(torch.bfloat16)
        rv = torch.randn((B, S, H, D), generator=g, device=DEV).to(torch.bfloat16)
        prcr.store_raw(mem, layer, rk, rv, vis_d, err=err)
        raws[layer] = (rk, rv)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    for b in (0, 1, 2, int(rng.integers(3, B))):
        _say(f"  sequence {b}: n_visual {nvis[b]}")
        ek = np.zeros((1, M, NL, H, D), np.uint16)
        ev = np.zeros_like(ek)
        for layer in layers:
            rk, rv = raws[layer]
            ek, ev, e = oracle.store_raw(ek, ev, layer, workloads.as_numpy_storage(rk[b:b + 1].cpu()),
                                         workloads.as_numpy_storage(rv[b:b + 1].cpu()),
                                         vis[b:b + 1], nvis[b:b + 1])
            assert e == 0
        assert np.array_equal(workloads.as_numpy_storage(mem.k[b:b + 1].cpu()), ek)
        assert np.array_equal(workloads.as_numpy_storage(mem.v[b:b + 1].cpu()), ev)
