"""GPU parity of reskv_build_cache on seeded random geometries (App. D,
Algorithm 1 with r given; scores App. B.2.2; selection Sec. 5.2; partition
and summaries Sec. 5.3, App. B.3).

Each seed draws the storage type, head dim, group size, KV heads, batch, and
per sequence a context length, budget and heavy-token count, per head a
residual count, plus the observation window and the pooling taps; every
(sequence, KV head) gets the full construction checks (scores, exact
selection on the GPU's scores, rows, Lloyd replay, summaries).
"""

import numpy as np
import pytest

from paper_2607_29591_amd import synth
from tests.build_check import check_head, run_build

pytestmark = pytest.mark.gpu


def draw_case(seed):
    rng = np.random.default_rng(2000 + seed)
    dtype = ["bf16", "f32"][seed % 2]
    d = [64, 128][(seed // 2) % 2]
    G = int(rng.choice([1, 2, 4, 7, 8]))
    hkv = int(rng.choice([1, 2]))
    batch = int(rng.integers(1, 4))
    window = int(rng.choice([1, 4, 8, 16]))
    pool = int(rng.choice([0, 1, 3, 7]))
    ctx = [int(rng.integers(30, 2600)) for _ in range(batch)]
    budget = [int(rng.integers(max(8, window + 2), 300)) for _ in range(batch)]
    n_heavy = [int(rng.integers(1, 8)) for _ in range(batch)]
    res = np.array([[[int(rng.integers(0, budget[b])) for _ in range(hkv)] for b in range(batch)]])
    return rng, dtype, d, G, hkv, batch, window, pool, ctx, budget, n_heavy, res


@pytest.mark.parametrize("seed", list(range(30)))
def test_build_random_geometry(seed):
    rng, dtype, d, G, hkv, batch, window, pool, ctx, budget, n_heavy, res = draw_case(seed)
    wl = synth.tiny_workload(s=max(ctx), d=d, hq=G * hkv, hkv=hkv, budget=max(budget), res=0, window=window,
                             dtype=dtype, batch=batch)
    wl.ctx, wl.budget, wl.n_heavy, wl.res = ctx, budget, n_heavy, res
    x = synth.gen_layer(wl, 0, seed=30 + seed, n_decode=1)
    x["K_host"], x["V_host"], x["q_host"] = x["K"], x["V"], x["q_obs"]
    got = run_build(wl, x, pool=pool)
    for b in range(batch):
        for h in range(hkv):
            check_head(wl, x, got, b, h, pool=pool if pool > 0 else 5, lloyd_info=False)


def draw_long_case(seed):
    rng = np.random.default_rng(3000 + seed)
    dtype = ["bf16", "f32"][seed % 2]
    d = [128, 64][(seed // 2) % 2]
    G = int(rng.choice([1, 4, 7]))
    hkv = int(rng.choice([1, 2]))
    window = int(rng.choice([4, 8, 32]))
    ctx = [int(rng.integers(8193, 40000))]
    budget = [int(rng.integers(64, 1100))]
    n_heavy = [int(rng.integers(4, 64))]
    res = np.array([[[int(rng.integers(0, 65)) for _ in range(hkv)]]])
    return dtype, d, G, hkv, window, ctx, budget, n_heavy, res


@pytest.mark.parametrize("seed", list(range(8)))
def test_build_random_long_context(seed):
    """Contexts of 8K-40K tokens: the top-k selection spans several 8192-score
    blocks with thresholds wherever the draw puts them."""
    dtype, d, G, hkv, window, ctx, budget, n_heavy, res = draw_long_case(seed)
    wl = synth.tiny_workload(s=ctx[0], d=d, hq=G * hkv, hkv=hkv, budget=budget[0], res=0, window=window,
                             dtype=dtype, batch=1)
    wl.n_heavy, wl.res = n_heavy, res
    x = synth.gen_layer(wl, 0, seed=60 + seed, n_decode=1)
    x["K_host"], x["V_host"], x["q_host"] = x["K"], x["V"], x["q_obs"]
    got = run_build(wl, x)
    for h in range(hkv):
        check_head(wl, x, got, 0, h, lloyd_info=False)
