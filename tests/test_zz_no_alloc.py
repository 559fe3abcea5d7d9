"""prcr_decode_attention_static, the decode entry point that allocates nothing: its
split-K partials live in the library's static device buffer.  Through the C ABI
(ctypes binding) it must give what prcr_decode_attention gives with a caller
workspace, on two calls in a row (the second with a smaller input, so the buffer
holds the first call's partials when the second starts), and refuse, before any
launch, a shape whose partials exceed the buffer."""
import ctypes

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


def _inputs(B, NL, H, G, D, cap, lens, paged, seed):
    g = torch.Generator().manual_seed(seed)
    rnd = lambda *s: torch.randn(s, generator=g).to(torch.bfloat16)
    rng = np.random.default_rng(seed)
    if paged:
        bs = 16
        need = (cap + bs - 1) // bs
        table = rng.permutation(B * need).astype(np.int32).reshape(B, need)
        k, v = rnd(NL, B * need, bs, H, D), rnd(NL, B * need, bs, H, D)
        cache_o = {"paged": True, "block_size": bs, "block_table": table, "max_blocks": need,
                   "n_blocks": B * need}
    else:
        k, v = rnd(B, NL, H, cap, D), rnd(B, NL, H, cap, D)
        cache_o = {"paged": False, "s_max": cap}
    cache_o["k"], cache_o["v"] = workloads.as_numpy_storage(k), workloads.as_numpy_storage(v)
    cache = prcr.Cache(k.to(DEV), v.to(DEV), to_dev(cache_o["block_table"]) if paged else None)
    q = rnd(B, H * G, D)
    q_pos = rng.integers(0, 20000, B).astype(np.int32)
    return cache, cache_o, q, q_pos, np.asarray(lens, np.int32)


@pytest.mark.parametrize("paged", [False, True], ids=["contiguous", "paged"])
def test_static_matches_workspace_entry_point(paged):
    D, layer = 128, 1
    rope = prcr.Rope(D, (16, 24, 24), False, 1e6)
    # call 1: 8 sequences x 4 KV heads x 4 query heads per KV head, up to 3000 keys;
    # call 2: a smaller problem, 3 sequences x 2 KV heads x 2 query heads per KV head
    shapes = [dict(B=8, NL=2, H=4, G=4, cap=3072, lens=[0, 1, 3000, 777, 2048, 5, 64, 2999],
                   seed=11),
              dict(B=3, NL=2, H=2, G=2, cap=1024, lens=[1000, 3, 0], seed=12)]
    for i, sh in enumerate(shapes):
        cache, cache_o, q, q_pos, lens = _inputs(sh["B"], sh["NL"], sh["H"], sh["G"], D, sh["cap"],
                                                 sh["lens"], paged, sh["seed"])
        need = prcr.decode_workspace_bytes(cache, sh["B"], sh["H"] * sh["G"])
        _say(f"static decode call {i + 1}: paged={paged} B={sh['B']} H={sh['H']} G={sh['G']} "
             f"partials {need} bytes")
        assert 0 < need <= prcr.binding.STATIC_SCRATCH_BYTES
        qd, qp, cl = q.to(DEV), to_dev(q_pos), to_dev(lens)
        err_s = torch.zeros(1, dtype=torch.int32, device=DEV)
        err_w = torch.zeros(1, dtype=torch.int32, device=DEV)
        out_s = prcr.decode_attention_static(rope, cache, layer, qd, qp, cl, err=err_s)
        out_w = prcr.decode_attention(rope, cache, layer, qd, qp, cl, err=err_w)
        torch.cuda.synchronize()
        assert int(err_s.item()) == 0 and int(err_w.item()) == 0
        # the same kernels over the same partial layout: identical results
        assert torch.equal(out_s, out_w), float((out_s - out_w).abs().max())
        # and within the decode tolerance of the oracle
        ref = oracle.decode_attention(rope.__dict__ | {"sections": rope.sections}, cache_o, layer,
                                      workloads.as_numpy_storage(q), q_pos, lens, D ** -0.5, "bf16")
        out = out_s.cpu().numpy()
        for b in range(sh["B"]):
            for kvh in range(sh["H"]):
                n = int(lens[b])
                vmax = np.abs(oracle.storage_to_f64(
                    oracle.cache_rows(cache_o, layer, b, kvh, n, "v"), "bf16")).max() if n else 0.0
                for g in range(sh["G"]):
                    qh = kvh * sh["G"] + g
                    assert np.abs(out[b, qh] - ref[b, qh]).max() <= 5e-5 * vmax + 1e-6
        _say(f"  call {i + 1} equal to the workspace entry point")


def test_static_refuses_partials_beyond_its_buffer():
    """65535 sequences x 32 query heads need ~1 GB of partials: PRCR_ERR_SCRATCH,
    returned on the host before anything is launched (output left untouched)."""
    D = 128
    rope = prcr.Rope(D, (16, 24, 24), False, 1e6)
    B, H, Hq = 65535, 4, 32
    _say("static decode: oversized shape refused")
    k = torch.zeros((1, 1, H, 16, D), dtype=torch.bfloat16, device=DEV)
    cc = prcr.binding.CCache(0, k.data_ptr(), k.data_ptr(), 16, None, 0, 0, 0)
    q = torch.zeros((B, Hq, D), dtype=torch.bfloat16, device=DEV)
    pos = torch.zeros(B, dtype=torch.int32, device=DEV)
    out = torch.full((B, Hq, D), 7.0, dtype=torch.float32, device=DEV)
    need = ctypes.c_size_t(0)
    L = prcr.lib()
    assert L.prcr_decode_workspace_size(ctypes.byref(cc), B, Hq, H, D, ctypes.byref(need)) == 0
    assert need.value > prcr.binding.STATIC_SCRATCH_BYTES
    st = L.prcr_decode_attention_static(ctypes.byref(rope.to_c()), ctypes.byref(cc), 1, B, 1, H, 0,
                                        q.data_ptr(), Hq, pos.data_ptr(), pos.data_ptr(), 0.088,
                                        out.data_ptr(), None, None)
    assert st == 9
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
