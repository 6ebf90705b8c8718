"""GPU parity of reskv_build_cache at the largest settings it accepts (App. D,
Algorithm 1 with r given; scores App. B.2.2; selection Sec. 5.2; partition
and summaries Sec. 5.3, App. B.3): 1024 scoring rows per KV head (G = 16,
w = 64), 4096 residual entries, and 64 Lloyd rounds. Every head gets the
full construction checks (scores, exact selection, rows, the Lloyd replay of
every round, summaries).
"""

import numpy as np
import pytest

from paper_2607_29591_amd import synth
from tests.build_check import check_head, run_build

pytestmark = pytest.mark.gpu


def layer(seed, dtype, d, G, hkv, s, budget, res, window, n_heavy=8):
    wl = synth.tiny_workload(s=s, d=d, hq=G * hkv, hkv=hkv, budget=budget, res=0, window=window, dtype=dtype,
                             n_heavy=n_heavy)
    wl.res = np.asarray(res, np.int64).reshape(1, 1, hkv)
    x = synth.gen_layer(wl, 0, seed=seed, n_decode=1)
    x["K_host"], x["V_host"], x["q_host"] = x["K"], x["V"], x["q_obs"]
    return wl, x


def test_build_1024_scoring_rows():
    """G * w = 1024 window rows per KV head (four 256-row chunks per key
    group); one head with residual entries, one without."""
    wl, x = layer(1, "bf16", 128, 16, 2, 3000, 300, [64, 0], 64)
    got = run_build(wl, x)
    for h in range(2):
        check_head(wl, x, got, 0, h, lloyd_info=False)


def test_build_4096_residual_entries():
    """r = 4096 = the largest residual capacity: 4096 Lloyd groups over the
    ~11.6K evicted tokens of a 12000-token context with a 4500-slot budget."""
    wl, x = layer(2, "bf16", 128, 4, 1, 12000, 4500, [4096], 8, n_heavy=32)
    got = run_build(wl, x)
    check_head(wl, x, got, 0, 0, lloyd_info=False)


def test_build_64_lloyd_rounds():
    """T = 64, the largest round count: every round's assignment replayed."""
    wl, x = layer(3, "f32", 64, 4, 2, 2000, 200, [32, 7], 8)
    got = run_build(wl, x, iters=64)
    for h in range(2):
        check_head(wl, x, got, 0, h, iters=64, lloyd_info=False)
