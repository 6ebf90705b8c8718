"""Pins for the oracle's AdaKV cross-head allocation (App. B.2.2 compared
methods: AdaKV allocates the retained budget across KV heads from SnapKV
scores with a safeguard coefficient; reading R26)."""

import itertools
import math

import numpy as np
import pytest

from oracle import reskv_oracle as orc


def kept_mass(scores, kk):
    return sum(np.sort(np.asarray(sc))[::-1][:k].sum() for sc, k in zip(scores, kk))


@pytest.mark.parametrize("seed", range(12))
def test_allocation_maximises_kept_score_brute_force(seed):
    """With distinct scores the allocation is the feasible split of largest
    kept score: floor(alpha k) <= k'_h <= cap_h, sum k'_h = min(K, sum cap)."""
    rng = np.random.default_rng(seed)
    H = 3
    n = rng.integers(2, 7, size=H)
    scores = [rng.random(int(x)) for x in n]
    k_top = [int(rng.integers(0, x + 1)) for x in n]
    cap = [int(min(x, rng.integers(k, x + 2))) for x, k in zip(n, k_top)]
    alpha = float(rng.choice([0.0, 0.2, 0.5]))
    kk = orc.adakv_allocate(scores, k_top, alpha, cap)
    floors = [math.floor(alpha * k) for k in k_top]
    target = min(sum(k_top), sum(cap))
    best, arg = -1.0, None
    for cand in itertools.product(*[range(f, c + 1) for f, c in zip(floors, cap)]):
        if sum(cand) != target:
            continue
        v = kept_mass(scores, cand)
        if v > best:
            best, arg = v, cand
    assert list(kk) == list(arg)


def test_alpha_zero_is_global_top_k():
    rng = np.random.default_rng(3)
    scores = [rng.random(40), rng.random(25), rng.random(33)]
    k_top = [10, 5, 12]
    kk = orc.adakv_allocate(scores, k_top, 0.0, [40, 25, 33])
    cat = np.concatenate(scores)
    head = np.concatenate([np.full(len(s), h) for h, s in enumerate(scores)])
    top = np.argsort(-cat, kind="stable")[:sum(k_top)]
    assert kk == [int((head[top] == h).sum()) for h in range(3)]


def test_alpha_one_keeps_the_uniform_split():
    rng = np.random.default_rng(4)
    scores = [rng.random(30) * (h + 1) for h in range(4)]
    assert orc.adakv_allocate(scores, [7, 3, 9, 0], 1.0, [30] * 4) == [7, 3, 9, 0]


def test_ties_go_to_the_lower_head_and_caps_bind():
    scores = [np.array([0.5, 0.5, 0.1]), np.array([0.5, 0.5, 0.9])]
    # K = 2, alpha 0: 0.9 first, then the first 0.5 of head 0
    assert orc.adakv_allocate(scores, [1, 1], 0.0, [3, 3]) == [1, 1]
    # K = 4: 0.9, then the four 0.5 go head 0 first
    assert orc.adakv_allocate(scores, [2, 2], 0.0, [3, 3]) == [2, 2]
    # head 1 capped at 1: the rest spills to head 0
    assert orc.adakv_allocate(scores, [2, 2], 0.0, [3, 1]) == [3, 1]


def test_build_heads_adakv_uniform_matches_build_head():
    """alpha = 1 keeps every head's uniform budget: the records equal
    build_head's, head by head."""
    rng = np.random.default_rng(5)
    s, d, G, w, budget = 120, 8, 2, 6, 40
    Ks = [rng.normal(size=(s, d)) for _ in range(3)]
    Vs = [rng.normal(size=(s, d)) for _ in range(3)]
    Qws = [rng.normal(size=(G, w, d)) for _ in range(3)]
    res = [8, 0, 5]
    recs = orc.build_heads_adakv(Ks, Vs, Qws, budget, res, w, 3, 1.0, 64, "f32")
    for h in range(3):
        ref = orc.build_head(Ks[h], Vs[h], Qws[h], budget - res[h], res[h], w, 3, "f32")
        np.testing.assert_array_equal(recs[h]["main_idx"], ref["main_idx"])
        np.testing.assert_array_equal(recs[h]["kc"], ref["kc"])


def test_build_heads_adakv_moves_budget_to_concentrated_heads():
    """The ranking is by attention mass, so a head whose window attention
    sits on a few tokens per row (large, spread keys) takes budget from a
    head whose attention is flat (near-identical keys: every token holds a
    small share); the total is conserved, the flat head keeps its floor, and
    the recent tokens stay protected in every head."""
    rng = np.random.default_rng(6)
    s, d, G, w, budget = 200, 8, 2, 6, 48
    base = rng.normal(size=d)
    Ks = [rng.normal(size=(s, d)) * 3, 0.02 * rng.normal(size=(s, d)) + base]
    Vs = [rng.normal(size=(s, d)) for _ in range(2)]
    Qws = [rng.normal(size=(G, w, d)), rng.normal(size=(G, w, d)) * 0.1]
    recs = orc.build_heads_adakv(Ks, Vs, Qws, budget, [4, 4], w, 2, 0.2, 96, "f32")
    k = [r["k_top"] for r in recs]
    assert sum(k) == 2 * (budget - 4 - w)
    assert k[0] > k[1] >= math.floor(0.2 * (budget - 4 - w))
    for r in recs:
        assert set(range(s - w, s)) <= set(r["main_idx"].tolist())
        assert r["main_len"] == w + r["k_top"]
