"""HIP graph capture of the two-call revisit (prcr_reassign_coords, then
prcr_rebind_inject: the step the bench times) and of prcr_store_raw.

Each graph is replayed several times, in a different order than the eager runs,
with new inputs written into the captured buffers and the target rows clobbered
by eager work in between.  Every replay must reproduce, bit for bit, the eager
calls on the same inputs (those are checked against the oracle elsewhere), and
replays on different inputs must differ.
"""
import numpy as np
import pytest
import torch

import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, Case, to_dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


@pytest.mark.parametrize("cfg", [3, 5])
def test_two_call_graph_replays_track_inputs(cfg):
    w = workloads.make(cfg, "small")
    _say(f"graph capture of reassign + rebind_inject (workload {cfg} small), 3 inputs")
    case = Case(w)
    mem, cache, rope = case.memory(), case.cache(), case.rope()
    so, si = to_dev(w.sel_off), to_dev(w.sel_idx)
    pt, cl = to_dev(w.p_txt), to_dev(w.cache_len)
    p0 = pt.clone()
    new_pos = torch.empty((w.total_k, 3), dtype=torch.float64, device=DEV)
    next_pos = torch.empty((w.B,), dtype=torch.int32, device=DEV)
    new_len = torch.empty((w.B,), dtype=torch.int32, device=DEV)
    slots = torch.empty((w.total_k,), dtype=torch.int64, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    outs = (cache.k, cache.v, new_pos, next_pos, new_len, slots)
    s = torch.cuda.Stream(device=DEV)
    torch.cuda.synchronize()

    def step():
        prcr.reassign_coords(mem, so, si, pt, "pcr", 2, new_pos, next_pos, err, s)
        prcr.rebind_inject(rope, mem, so, si, new_pos, cache, cl, new_len, slots, err, s)

    eager = []
    for r in range(3):
        pt.copy_(p0 + 7 * r)
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            step()
        torch.cuda.synchronize()
        eager.append([t.clone() for t in outs])
    assert not torch.equal(eager[0][2], eager[1][2])      # the inputs change the positions
    assert not torch.equal(_bits(eager[0][0]), _bits(eager[1][0]))

    if w.paged:
        rows = (slots // w.block_size, slots % w.block_size)
        def clobber():
            cache.k[:, rows[0], rows[1]] = 0
            cache.v[:, rows[0], rows[1]] = 0
    else:
        s_max = cache.k.shape[3]
        rows = (slots // s_max, slots % s_max)
        def clobber():
            cache.k[rows[0], :, :, rows[1]] = 0
            cache.v[rows[0], :, :, rows[1]] = 0

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        step()
    torch.cuda.synchronize()
    for r in (2, 0, 1, 2):
        pt.copy_(p0 + 7 * r)                        # new input into the captured buffer
        clobber()                                   # eager work on the target rows
        new_pos.zero_(); next_pos.zero_(); new_len.zero_(); slots.fill_(-7)
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(outs, eager[r])):
            assert torch.equal(_bits(a), _bits(b)), f"replay with input {r}, output {i}"
    assert int(err.item()) == 0


def test_store_raw_graph_replays_track_inputs():
    B, M, S, NL, H, D = 5, 40, 64, 3, 4, 128
    _say(f"graph capture of store_raw B={B} M={M} S={S} NL={NL} H={H} D={D} bf16, 3 inputs")
    g = torch.Generator(device=DEV)
    g.manual_seed(600)
    rng = np.random.default_rng(600)
    raws = [(torch.randn((B, S, H, D), generator=g, device=DEV).to(torch.bfloat16),
             torch.randn((B, S, H, D), generator=g, device=DEV).to(torch.bfloat16)) for _ in range(3)]
    nvis = np.array([40, 0, 17, 1, 33], np.int32)
    vis = to_dev(np.stack([np.sort(rng.choice(S, M, replace=False)) for _ in range(B)]).astype(np.int32))
    mem = prcr.Memory(torch.zeros((B, M, NL, H, D), dtype=torch.bfloat16, device=DEV),
                      torch.zeros((B, M, NL, H, D), dtype=torch.bfloat16, device=DEV),
                      torch.zeros((B, M, 3), dtype=torch.int32, device=DEV), to_dev(nvis))
    rk, rv = torch.empty_like(raws[0][0]), torch.empty_like(raws[0][1])
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    s = torch.cuda.Stream(device=DEV)
    torch.cuda.synchronize()

    def call():
        prcr.store_raw(mem, 1, rk, rv, vis, err, s)

    eager = []
    for r in range(3):
        rk.copy_(raws[r][0]); rv.copy_(raws[r][1])
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            call()
        torch.cuda.synchronize()
        eager.append((mem.k.clone(), mem.v.clone()))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        call()
    torch.cuda.synchronize()
    for r in (1, 2, 0, 1):
        rk.copy_(raws[r][0]); rv.copy_(raws[r][1])
        mem.k[:, :, 1] = 0                          # eager work on the target layer
        mem.v[:, :, 1] = 0
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize()
        assert torch.equal(_bits(mem.k), _bits(eager[r][0])), f"replay with input {r}"
        assert torch.equal(_bits(mem.v), _bits(eager[r][1])), f"replay with input {r}"
    assert not torch.equal(_bits(eager[0][0]), _bits(eager[1][0]))
    assert int(err.item()) == 0
