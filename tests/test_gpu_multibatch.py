"""Whole-output GPU parity at the launch shapes of the full-size workloads.

On large problems the rebinding kernel gives each wavefront several load batches
of one token's (layer, head) rows: the next batch is in flight while the current
one is rotated and stored, rows past the wave's run reload its last row, and the
last row group of a token can end in a partial batch.  The shapes here are chosen
so that the launch takes that form, with every key, value and untouched cache
byte compared against the oracle (Eq. (11)-(13)), not a sample:

  * 36 layers x 8 KV heads, 1024 selected tokens: 80 rows per wave (5 batches)
    and a last group of 48, the 32-sequence workload's own launch shape;
  * 35 x 8: the last group of 40 rows ends in a half batch;
  * 28 x 4, 4096 tokens, paged: 64 rows per wave (4 batches) and 48, the paged
    workload's own launch shape;
  * 27 x 4, paged: the last group of 44 rows ends in a partial batch.

Each runs as the two-call path and as the single-launch revisit.
"""
import pytest

import workloads
from gpu_util import Case, assert_parity, run_both

pytestmark = pytest.mark.gpu

CASES = {
    "contiguous-36x8": dict(B=4, NL=36, H=8, sections=(22, 21, 21), interleaved=True, theta=5e6,
                            gh=32, gw=24, ks=(256, 256, 256, 256), lens=(300, 17, 500, 650),
                            seed=31),
    "contiguous-35x8-partial": dict(B=4, NL=35, H=8, sections=(22, 21, 21), interleaved=True,
                                    theta=5e6, gh=32, gw=24, ks=(256, 256, 256, 256),
                                    lens=(64, 401, 0, 333), seed=32),
    "paged-28x4": dict(B=8, NL=28, H=4, sections=(16, 24, 24), gh=32, gw=24, ks=(512,) * 8,
                       lens=(100, 513, 0, 37, 260, 16, 999, 1), paged=True, block_size=16,
                       seed=33),
    "paged-27x4-partial": dict(B=8, NL=27, H=4, sections=(16, 24, 24), gh=32, gw=24,
                               ks=(512,) * 8, lens=(5, 300, 48, 700, 2, 129, 64, 33), paged=True,
                               block_size=16, seed=34),
}


def _say(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("fused", [False, True], ids=["two-call", "fused"])
@pytest.mark.parametrize("name", sorted(CASES))
def test_full_launch_shape_whole_output(name, fused):
    w = workloads.custom(D=128, dtype="bf16", **CASES[name])
    _say(f"{name} {'fused' if fused else 'two-call'}: B={w.B} NL={w.NL} H={w.H} "
         f"K={w.total_k} rows={w.total_k * w.NL * w.H}")
    case = Case(w)
    gpu, ref = run_both(case, w.sel_off, w.sel_idx, w.p_txt, w.cache_len, fused=fused)
    exact, n = assert_parity(case, gpu, ref)
    assert n == w.total_k * w.NL * w.H * w.D          # every rebound key element compared
    _say(f"  keys bit-exact {exact}/{n}")
