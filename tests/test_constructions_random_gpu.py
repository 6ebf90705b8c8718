"""GPU parity of the AdaKV and validation-proxy constructions on seeded
random geometries (App. B.2.2 AdaKV allocation, reading R26; Sec. 5.5.1
validation loss and margin rule, App. D Algorithm 1, App. B.3 grid).

AdaKV: each seed draws the storage type, head dim, group size, KV heads,
batch, per-sequence contexts and budgets, per-head residual counts, the
safeguard and the slot capacity; every sequence gets the allocation checks
and every head the construction checks. Proxy: each seed draws the group
size, window and validation rows, contexts and budgets; every head gets
the decision rule, the bit equality with its chosen candidate and the
candidates' losses (the checks of the proxy tests).
"""

import numpy as np
import pytest

from paper_2607_29591_amd import synth
from tests.build_check import run_build
from tests.test_adakv_gpu import check_sequence
from tests.test_proxy_gpu import GRID, check_proxy

pytestmark = pytest.mark.gpu


def draw_adakv(seed):
    rng = np.random.default_rng(4000 + seed)
    dtype = ["bf16", "f32"][seed % 2]
    d = [128, 64][(seed // 2) % 2]
    G = int(rng.choice([1, 2, 4, 7]))
    hkv = int(rng.choice([2, 3, 4]))
    batch = int(rng.integers(1, 4))
    window = int(rng.choice([4, 8]))
    ctx = [int(rng.integers(40, 3000)) for _ in range(batch)]
    budget = [int(rng.integers(16, 200)) for _ in range(batch)]
    res = np.array([[[int(rng.integers(0, b)) for _ in range(hkv)] for b in budget]])
    alpha = float(rng.choice([0.0, 0.2, 0.5, 1.0]))
    C = int(max(budget) * rng.uniform(1.0, 2.5))
    return dtype, d, G, hkv, batch, window, ctx, budget, res, alpha, C


@pytest.mark.parametrize("seed", list(range(12)))
def test_adakv_random_geometry(seed):
    dtype, d, G, hkv, batch, window, ctx, budget, res, alpha, C = draw_adakv(seed)
    wl = synth.tiny_workload(s=max(ctx), d=d, hq=G * hkv, hkv=hkv, budget=max(budget), res=0, window=window,
                             dtype=dtype, batch=batch)
    wl.ctx, wl.budget, wl.res = ctx, budget, res
    x = synth.gen_layer(wl, 0, seed=80 + seed, n_decode=1)
    x["K_host"], x["V_host"], x["q_host"] = x["K"], x["V"], x["q_obs"]
    got = run_build(wl, x, adakv=alpha, slot_cap=C)
    for b in range(batch):
        check_sequence(wl, x, got, b, alpha, C, window)


def draw_proxy(seed):
    rng = np.random.default_rng(5000 + seed)
    dtype = ["bf16", "f32"][seed % 2]
    d = [128, 64][(seed // 2) % 2]
    G = int(rng.choice([1, 4, 7]))
    hkv = int(rng.choice([1, 2]))
    batch = int(rng.integers(1, 3))
    window = int(rng.choice([8, 16, 32]))
    val = int(rng.integers(2, window // 2 + 1))
    ctx = [int(rng.integers(60, 2000)) for _ in range(batch)]
    budget = [int(rng.integers(32, 200)) for _ in range(batch)]
    return dtype, d, G, hkv, batch, window, val, ctx, budget


@pytest.mark.parametrize("seed", list(range(6)))
def test_proxy_random_geometry(seed):
    dtype, d, G, hkv, batch, window, val, ctx, budget = draw_proxy(seed)
    wl = synth.tiny_workload(s=max(ctx), d=d, hq=G * hkv, hkv=hkv, budget=max(budget), res=0, window=window,
                             dtype=dtype, batch=batch)
    wl.ctx, wl.budget = ctx, budget
    # residual capacity for the largest candidate of the grid
    wl.res = np.full((1, batch, hkv), int(np.floor(max(GRID) * max(budget) + 0.5)))
    x = synth.gen_layer(wl, 0, seed=90 + seed, n_decode=1)
    x["K_host"], x["V_host"], x["q_host"] = x["K"], x["V"], x["q_obs"]
    rep, got = check_proxy(wl, x, GRID, val, 0.01)
    assert rep["heads"] == batch * hkv
