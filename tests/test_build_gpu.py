"""GPU parity of reskv_build_cache against the fp64 oracle (App. D, Algorithm 1
with r given; scores App. B.2.2; selection Sec. 5.2; partition and summaries
Sec. 5.3, App. B.3), then decode over the GPU-built cache (Sec. 5.4)."""

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import reskv as rk
from paper_2607_29591_amd import synth
from tests.build_check import check_head, run_build
from tests.helpers import TOL, decode_on_gpu, rel_err_rows

pytestmark = pytest.mark.gpu


def host_copies(x):
    x["K_host"], x["V_host"], x["q_host"] = x["K"], x["V"], x["q_obs"]
    return x


def small(seed, dtype="f32", d=64, s=300, hq=8, hkv=2, budget=64, res=(16, 0), window=8, batch=1, n_heavy=4):
    wl = synth.tiny_workload(s=s, d=d, hq=hq, hkv=hkv, budget=budget, res=0, window=window, dtype=dtype,
                             batch=batch, n_heavy=n_heavy)
    wl.res = np.asarray(res, np.int64).reshape(1, batch, hkv)
    x = host_copies(synth.gen_layer(wl, 0, seed=seed, n_decode=2))
    return wl, x


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [64, 128])
def test_build_small(dtype, d):
    wl, x = small(1, dtype=dtype, d=d, s=700, budget=96, res=(40, 0))
    got = run_build(wl, x)
    for h in range(wl.hkv):
        check_head(wl, x, got, 0, h)


def test_build_ragged_batch_gqa7_and_edge_cases():
    """G = 7; per-sequence lengths and budgets; one sequence shorter than its
    budget (every token main); r = 0; r larger than the evicted set; a
    protected window longer than the main budget."""
    wl = synth.tiny_workload(s=600, d=128, hq=14, hkv=2, budget=64, res=0, window=8, dtype="bf16", batch=4)
    wl.ctx = [600, 50, 333, 90]
    wl.budget = [64, 64, 48, 80]
    wl.n_heavy = [4, 2, 3, 2]
    wl.res = np.array([[[16, 0], [8, 30], [47, 1], [40, 79]]])
    x = host_copies(synth.gen_layer(wl, 0, seed=2, n_decode=1))
    got = run_build(wl, x)
    for b in range(4):
        for h in range(2):
            check_head(wl, x, got, b, h)
    got2 = run_build(wl, x, recent=70)
    for b in range(4):
        for h in range(2):
            check_head(wl, x, got2, b, h, recent=70)


@pytest.mark.parametrize("recent", [None, 4])
def test_build_window_covers_the_sequence(recent):
    """s = w, the largest window the boundary accepts: every position is a
    window query position and the scored range [0, s - |P|) shrinks with the
    protected window. With the default protected window (|P| = min(w, m, s)
    = m) every main slot is protected and no top-k is taken; with |P| = 4
    the top-k runs on [0, s - 4). A 4-token sequence (w = s = 4, budget 2,
    r = 1) sits beside a 40-token one."""
    wl = synth.tiny_workload(s=40, d=64, hq=8, hkv=2, budget=24, res=0, window=40, dtype="f32", batch=1, n_heavy=2)
    wl.res = np.array([[[8, 0]]])
    x = host_copies(synth.gen_layer(wl, 0, seed=21, n_decode=1))
    got = run_build(wl, x, recent=recent)
    for h in range(2):
        check_head(wl, x, got, 0, h, recent=recent)
    wl = synth.tiny_workload(s=4, d=64, hq=8, hkv=2, budget=2, res=0, window=4, dtype="f32", batch=1, n_heavy=1)
    wl.res = np.array([[[1, 0]]])
    x = host_copies(synth.gen_layer(wl, 0, seed=22, n_decode=1))
    got = run_build(wl, x, recent=None if recent is None else 1)
    for h in range(2):
        check_head(wl, x, got, 0, h, recent=None if recent is None else 1)


def test_build_ties_take_lowest_positions():
    """Identical keys and queries give identical window scores; zero-padded
    pooling lowers the two positions at each end of the scored range, so the
    tied interior positions are taken lowest first (2, 3, ...)."""
    wl, x = small(3, dtype="bf16", d=64, s=200, budget=40, res=(8, 8))
    x["K"][:] = 1.0
    x["q_obs"][:] = 0.5
    host_copies(x)
    got = run_build(wl, x)
    for h in range(wl.hkv):
        check_head(wl, x, got, 0, h)
        assert got["main_idx"][0, h, :32].tolist() == list(range(2, 26)) + list(range(192, 200))


@pytest.mark.parametrize("s", [20000, 16392])
def test_build_ties_across_selection_blocks(s):
    """All scores equal over 20000 positions (three 8192-score selection
    blocks, the last partial) or over exactly two full blocks (16384 scored
    positions): the tie ranks run across the blocks, so the top-scored
    tokens are the lowest interior positions and the seeds the next ones."""
    wl, x = small(3, dtype="bf16", d=64, s=s, budget=600, res=(64, 32))
    x["K"][:] = 1.0
    x["q_obs"][:] = 0.5
    host_copies(x)
    got = run_build(wl, x)
    for h in range(wl.hkv):
        check_head(wl, x, got, 0, h)
        k_top = 600 - wl.res[0, 0, h] - wl.window
        assert got["main_idx"][0, h, :k_top].tolist() == list(range(2, 2 + k_top))


def test_build_workload0_and_decode():
    """The fp32 toy workload end to end: construction parity, then decode of
    the 8 queries over the GPU-built cache."""
    wl = synth.workload(0)
    x = host_copies(synth.gen_layer(wl, 0))
    got = run_build(wl, x)
    for h in range(wl.hkv):
        check_head(wl, x, got, 0, h)
    shape = rk.make_shape(wl.batch, wl.hq, wl.hkv, wl.d, wl.dtype, wl.slot_cap, wl.res_cap)
    for step in range(wl.steps):
        q = x["q_dec"][step].astype(np.float64)
        out = decode_on_gpu(shape, dict(tau_scalar=0.25, alpha=12.0, g_min=0.0, beta=1.0), q, got["kc"],
                            got["vc"], got["logc"], got["res_len"], got["main_len"], dbg=False)["out"]
        ref, *_ = orc.decode(q, got["kc"], got["vc"], got["logc"], got["res_len"], got["main_len"],
                             0.25, 12.0, 0.0, 1.0)
        assert rel_err_rows(out, ref).max() <= TOL["f32"]


@pytest.mark.parametrize("s,budget,res,iters", [(4000, 1600, (1500, 1030), 2), (8192, 4200, (4096, 0), 1)])
def test_build_many_groups(s, budget, res, iters):
    """More than 1024 residual groups per head, up to the 4096 entries a
    construction accepts: the group offsets take several column passes and
    a group index spans 11 to 12 bits in the stable placement; both update
    variants run in the two-round case."""
    wl, x = small(31, dtype="bf16", d=128, s=s, hq=8, hkv=2, budget=budget, res=res, window=16, n_heavy=8)
    assert wl.res_cap == max(res)
    got = run_build(wl, x, iters=iters)
    for h in range(wl.hkv):
        check_head(wl, x, got, 0, h, iters=iters)


@pytest.mark.parametrize("dtype,d,hq,hkv,window", [("bf16", 128, 16, 2, 20), ("bf16", 64, 16, 1, 24),
                                                  ("f32", 64, 8, 1, 40), ("f32", 128, 8, 2, 40)])
def test_build_many_window_rows(dtype, d, hq, hkv, window):
    """More than 128 window rows (G w = 160, 384, 320, 160): the scoring
    passes stage the rows in one or two 256-row chunks (bf16, fp32 at d 64)
    or in 128-row chunks (fp32 at d 128), with a partial last chunk."""
    res = (48, 16)[:hkv]
    wl, x = small(41, dtype=dtype, d=d, s=1500, hq=hq, hkv=hkv, budget=200, res=res, window=window, n_heavy=6)
    assert wl.group * window > 128
    got = run_build(wl, x)
    for h in range(wl.hkv):
        check_head(wl, x, got, 0, h)


def test_build_is_deterministic():
    wl, x = small(4, dtype="bf16", d=128, s=2000, budget=256, res=(64, 32), window=16)
    a = run_build(wl, x)
    b = run_build(wl, x)
    for k in ("kc", "vc", "logc", "main_idx", "assign", "scores"):
        np.testing.assert_array_equal(a[k], b[k])


@pytest.mark.parametrize("scorer", ["h2o", "tova", "pool3", "pool9", "pool31"])
def test_build_alternative_scorers(scorer):
    """The compared scorers of App. B.2.2 through the same selection and
    residual path: H2O (accumulated window attention, no pooling, 64 recent
    tokens), TOVA (last-token window w = 1, no pooling, 1 recent token), and
    3-, 9- and 31-tap (the largest accepted) pooling; ragged lengths, G = 4,
    bf16, d = 128."""
    window, recent, pool = {"h2o": (8, 64, 1), "tova": (1, 1, 1), "pool3": (8, 8, 3), "pool9": (8, 8, 9),
                            "pool31": (8, 8, 31)}[scorer]
    wl = synth.tiny_workload(s=900, d=128, hq=8, hkv=2, budget=160, res=0, window=window, dtype="bf16", batch=2,
                             n_heavy=6)
    wl.ctx = [900, 517]
    wl.res = np.array([[[24, 0], [40, 7]]])
    x = host_copies(synth.gen_layer(wl, 0, seed=21, n_decode=1))
    got = run_build(wl, x, recent=recent, pool=pool)
    for b in range(2):
        for h in range(2):
            check_head(wl, x, got, b, h, recent=recent, pool=pool)
