"""The bandwidth measurement's reference copies.  The pattern copy must touch
exactly the bytes the rebind touches: run on a small 32-sequence-shaped and a small
paged workload, every new slot row of the cache must equal the raw memory row of
its token (keys unrotated, values as they are) and every other cache byte must be
unchanged; the new slots are those of the rebind's own slot mapping.  The
streaming copy must copy."""
import numpy as np
import pytest
import torch

import bench
import paper_2606_26631_amd as prcr
import workloads
from gpu_util import DEV, Case, new_row_mask, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg", [3, 5])
def test_pattern_copy_writes_the_rebinds_slots(cfg):
    w = workloads.make(cfg, "small")
    print(f"pattern copy, workload {cfg} small: B={w.B} NL={w.NL} H={w.H} K={w.total_k}",
          flush=True)
    case = Case(w)
    mem, cache = case.memory(), case.cache()
    # the slots the rebind writes
    so, si = to_dev(w.sel_off), to_dev(w.sel_idx)
    new_pos, _ = prcr.reassign_coords(mem, so, si, to_dev(w.p_txt))
    scratch = prcr.Cache(cache.k.clone(), cache.v.clone(), cache.block_table)
    _, slots = prcr.rebind_inject(case.rope(), mem, so, si, new_pos, scratch, to_dev(w.cache_len))
    del scratch
    p = type("P", (), {})()
    p.w, p.mem, p.cache = w, mem, cache
    before_k, before_v = cache.k.clone(), cache.v.clone()
    bench.pattern_copy(p, steps=1, warmup=0)
    torch.cuda.synchronize()
    mask = torch.from_numpy(new_row_mask(w, slots.cpu().numpy())).to(DEV)
    for got, before, src in ((cache.k, before_k, mem.k), (cache.v, before_v, mem.v)):
        assert torch.equal(got[~mask], before[~mask])          # nothing else touched
        so_np, si_np = w.sel_off, w.sel_idx
        sl = slots.cpu().numpy()
        for g in range(w.total_k):
            b = int(np.searchsorted(so_np, g, side="right") - 1)
            m = int(si_np[g])
            sid = int(sl[g])
            if w.paged:
                dst = got[:, sid // w.block_size, sid % w.block_size]          # [NL][H][D]
            else:
                dst = got[sid // w.s_max, :, :, sid % w.s_max]                 # [NL][H][D]
            assert torch.equal(dst, src[b, m]), (g, b, m)


def test_stream_copy_copies():
    print("stream copy, 64 MiB", flush=True)
    src = torch.randint(0, 255, (64 << 20,), dtype=torch.uint8, device=DEV)
    dst = torch.zeros_like(src)
    L = bench.copyref_lib()
    assert L.prcr_copyref_stream(src.data_ptr(), dst.data_ptr(), src.numel(), 16384,
                                 torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    assert torch.equal(src, dst)


def test_prefill_pattern_copy_writes_the_prefills_rows():
    """The prefill pattern copy writes every prompt row raw into the cache slot the
    prefill uses (slot s of a contiguous cache) and every visual row into the memory,
    and nothing else."""
    B, NL, H, D, layer = 2, 3, 4, 128, 1
    pos, vis, n_tok, n_vis = workloads.prompt(B, n_before=(5, 9), grid=((4, 6), (3, 5)),
                                              n_after=(3, 0), frames=(1, 2))
    S, M = pos.shape[1], int(n_vis.max())
    print(f"prefill pattern copy: B={B} S={S} M={M} H={H}", flush=True)
    g = torch.Generator(device=DEV)
    g.manual_seed(77)
    raw_k = torch.randn((B, S, H, D), generator=g, device=DEV).to(torch.bfloat16)
    raw_v = torch.randn((B, S, H, D), generator=g, device=DEV).to(torch.bfloat16)
    ck = torch.randn((B, NL, H, S + 4, D), generator=g, device=DEV).to(torch.bfloat16)
    cv, mk, mv = ck.clone() + 1, torch.randn((B, M, NL, H, D), generator=g, device=DEV).to(
        torch.bfloat16), None
    mv = mk.clone() + 1
    before = [x.clone() for x in (ck, cv, mk, mv)]
    L = bench.copyref_lib()
    assert L.prcr_copyref_prefill(raw_k.data_ptr(), raw_v.data_ptr(), to_dev(vis).data_ptr(),
                                  to_dev(n_tok).data_ptr(), ck.data_ptr(), cv.data_ptr(),
                                  mk.data_ptr(), mv.data_ptr(), B, S, H, NL, layer, S + 4, M,
                                  torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    exp = [x.clone() for x in before]
    for b in range(B):
        for s in range(int(n_tok[b])):
            exp[0][b, layer, :, s] = raw_k[b, s]
            exp[1][b, layer, :, s] = raw_v[b, s]
            m = int(vis[b, s])
            if m >= 0:
                exp[2][b, m, layer] = raw_k[b, s]
                exp[3][b, m, layer] = raw_v[b, s]
    for got, want in zip((ck, cv, mk, mv), exp):
        assert torch.equal(got, want)
