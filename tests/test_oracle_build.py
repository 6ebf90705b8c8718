"""Pins for the oracle's construction: window scores (App. B.2.2), main
selection (Sec. 5.2), Lloyd partition and summaries (Sec. 5.3, App. B.3),
and the end-to-end invariants of the built cache (Sec. 3.1, 3.2, 5.3, 5.4).
"""

import itertools
import json
import math
import os
import warnings

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def sdpa(q, K, V):
    q = torch.as_tensor(np.asarray(q), dtype=torch.float64)[None, None, None, :]
    K = torch.as_tensor(np.asarray(K), dtype=torch.float64)[None, None]
    V = torch.as_tensor(np.asarray(V), dtype=torch.float64)[None, None]
    return torch.nn.functional.scaled_dot_product_attention(q, K, V)[0, 0, 0].numpy()


# ----------------------------------------------------------------- scores

def brute_raw(K, Qw):
    """Pure-Python loops: per window row, softmax over the keys it can see."""
    s, d = len(K), len(K[0])
    G, w = len(Qw), len(Qw[0])
    raw = [0.0] * s
    for h in range(G):
        for i in range(w):
            pos = s - w + i
            logits = [sum(Qw[h][i][c] * K[p][c] for c in range(d)) / math.sqrt(d) for p in range(pos + 1)]
            top = max(logits)
            ex = [math.exp(x - top) for x in logits]
            tot = sum(ex)
            for p in range(pos + 1):
                raw[p] += ex[p] / tot
    return raw


def test_scores_hand_example_golden():
    g = json.load(open(os.path.join(GOLD, "scores_hand_example.json")))
    K = np.array([[0.0], [math.log(2)], [math.log(3)]])
    Qw = np.array([[[1.0]]])
    raw = orc.window_raw_scores(K, Qw)
    np.testing.assert_allclose(raw, [1 / 6, 2 / 6, 3 / 6], rtol=1e-15)
    n = orc.scored_length(3, g["m"], g["window"])
    pooled = orc.pool5(raw[:n])
    np.testing.assert_allclose(pooled, [0.5, 0.5], rtol=1e-15)
    main, ev, seeds = orc.select_main(pooled, 3, g["m"], g["window"], 1)
    assert main.tolist() == g["expected"]["main_idx"]
    assert ev.tolist() == g["expected"]["evicted"]
    assert seeds.tolist() == [1]


@pytest.mark.parametrize("seed", range(6))
def test_window_scores_brute_force(seed):
    rng = np.random.default_rng(seed)
    s = int(rng.integers(3, 13))
    d = int(rng.integers(1, 5))
    G = int(rng.integers(1, 4))
    w = int(rng.integers(1, s + 1))
    K = rng.normal(size=(s, d)) * 2
    Qw = rng.normal(size=(G, w, d)) * 2
    np.testing.assert_allclose(orc.window_raw_scores(K, Qw), brute_raw(K.tolist(), Qw.tolist()), rtol=1e-12)


def test_window_mass_closed_form():
    """Every window row distributes mass 1 over the keys it sees: sum raw = G*w."""
    rng = np.random.default_rng(3)
    K = rng.normal(size=(300, 16)) * 3
    Qw = rng.normal(size=(4, 16, 16)) * 3
    raw = orc.window_raw_scores(K, Qw)
    assert raw.sum() == pytest.approx(64.0, rel=1e-12)
    # the last key is seen only by the last row of each head
    assert raw[-1] <= 4.0 + 1e-12


def test_pool5_matches_convolution():
    rng = np.random.default_rng(4)
    for n in [1, 2, 3, 4, 5, 6, 17, 100]:
        raw = rng.random(n)
        np.testing.assert_allclose(orc.pool5(raw), np.convolve(raw, np.ones(5), mode="same")[:n] if n >= 5
                                   else np.convolve(raw, np.ones(5), mode="full")[2:2 + n], rtol=1e-14)


# -------------------------------------------------------------- selection

@pytest.mark.parametrize("seed", range(8))
def test_select_matches_python_sort(seed):
    rng = np.random.default_rng(seed)
    s = int(rng.integers(10, 200))
    m = int(rng.integers(1, s))
    P = int(rng.integers(0, 20))
    r = int(rng.integers(0, s))
    n = orc.scored_length(s, m, P)
    # coarse scores force many exact ties
    scores = rng.integers(0, 6, size=n).astype(float) / 4
    main, ev, seeds = orc.select_main(scores, s, m, P, r)
    order = sorted(range(n), key=lambda i: (-scores[i], i))
    p = min(P, m, s)
    k_top = m - p
    assert main.tolist() == sorted(order[:k_top] + list(range(n, s)))
    assert ev.tolist() == sorted(order[k_top:])
    assert seeds.tolist() == sorted(order[k_top:k_top + r])
    assert len(main) == m and set(main) | set(ev) == set(range(s)) and not set(main) & set(ev)
    assert set(range(s - p, s)) <= set(main.tolist())


def test_select_all_equal_takes_lowest():
    main, ev, seeds = orc.select_main(np.ones(90), 100, 30, 10, 5)
    assert main.tolist() == list(range(20)) + list(range(90, 100))
    assert seeds.tolist() == list(range(20, 25))


def test_select_everything_fits():
    main, ev, seeds = orc.select_main(np.zeros(0), 10, 16, 4, 3)
    assert main.tolist() == list(range(10)) and ev.size == 0 and seeds.size == 0


# ------------------------------------------------------------------ Lloyd

def test_lloyd_matches_sklearn():
    """Centres after T rounds equal scikit-learn's Lloyd k-means from the same
    initial centres (no empty clusters arise on this data)."""
    from sklearn.cluster import KMeans
    rng = np.random.default_rng(0)
    for trial in range(4):
        r = 6
        cent = rng.normal(size=(r, 5)) * 4
        X = np.concatenate([c + rng.normal(size=(40, 5)) for c in cent])
        init = X[rng.choice(X.shape[0], r, replace=False)]
        for T in (1, 2, 4):
            _, mu, _ = orc.lloyd(X, init, T)
            with warnings.catch_warnings():
                warnings.simplefilter("ignore")
                km = KMeans(n_clusters=r, init=init, n_init=1, max_iter=T, tol=0.0,
                            algorithm="lloyd").fit(X)
            np.testing.assert_allclose(mu, km.cluster_centers_, rtol=1e-10, atol=1e-12)


def test_lloyd_objective_nonincreasing_and_counts():
    rng = np.random.default_rng(1)
    X = rng.normal(size=(500, 8))
    init = X[:16]
    objs = []
    for T in range(1, 7):
        a, mu, hist = orc.lloyd(X, init, T)
        objs.append(orc.lloyd_objective(X, a, 16))
        assert np.bincount(a, minlength=16).sum() == 500
    assert all(b <= a + 1e-9 for a, b in zip(objs, objs[1:]))


def test_lloyd_single_cluster_closed_form():
    rng = np.random.default_rng(2)
    KE, VE = rng.normal(size=(50, 6)), rng.normal(size=(50, 6))
    a, mu, _ = orc.lloyd(KE, KE[:1], 4)
    kb, vb, c, lc = orc.residual_entries(KE, VE, a, mu, 1, 6)
    np.testing.assert_allclose(kb[0], KE.mean(0), rtol=1e-13)
    np.testing.assert_allclose(vb[0], VE.mean(0), rtol=1e-13)
    assert c[0] == 50 and lc[0] == pytest.approx(math.log(50))


def test_lloyd_brute_force_partition_optimum():
    """On well-separated tiny sets, Lloyd from the right seeds reaches the
    exhaustive minimum of the partition objective (Sec. 5.3)."""
    rng = np.random.default_rng(3)
    for trial in range(5):
        cents = np.array([[0, 0], [10, 0], [0, 10]], float)
        X = np.concatenate([c + rng.normal(scale=0.5, size=(int(rng.integers(1, 3)) + 1, 2)) for c in cents])
        n, r = X.shape[0], 3
        best = min(orc.lloyd_objective(X, np.array(lab), r)
                   for lab in itertools.product(range(r), repeat=n))
        init = X[[0, np.argmax(X[:, 0]), np.argmax(X[:, 1])]]
        a, mu, _ = orc.lloyd(X, init, 4)
        assert orc.lloyd_objective(X, a, r) == pytest.approx(best, rel=1e-12)


def test_lloyd_assignment_ties_lowest_centre():
    X = np.array([[0.0, 0.0], [1.0, 0.0]])
    cents = np.array([[0.5, 1.0], [0.5, -1.0]])   # equidistant from both points
    a, _ = orc.assign_nearest(X, cents)
    assert a.tolist() == [0, 0]


# ------------------------------------------------------ end-to-end cache

def tiny(seed, s=60, d=8, budget=16, res=4, window=4, dtype="f32"):
    wl = synth.tiny_workload(s=s, d=d, budget=budget, res=res, window=window, dtype=dtype)
    return wl, synth.gen_layer(wl, 0, seed=seed, n_decode=3)


def built(wl, x, budget=None, res=None, g_dtype=None):
    b = np.asarray(x["budget"]) if budget is None else np.asarray(budget)
    rc = np.asarray(x["res"]) if res is None else np.asarray(res)
    cap = int(max(b.max(), wl.max_ctx))
    return orc.build_cache(x["K"], x["V"], x["q_obs"], x["seq_len"], b, rc, wl.window, 4,
                           g_dtype or wl.dtype, cap, max(1, int(rc.max())))


def test_cache_holding_every_token_is_full_attention():
    wl, x = tiny(1)
    c = built(wl, x, budget=[80], res=[[0, 0]])
    out, *_ = orc.decode(x["q_dec"][0], c["kc"], c["vc"], c["logc"], c["res_len"], c["main_len"],
                         0.25, 12.0, 0.0, 1.0)
    for h in range(wl.hq):
        kv = h // wl.group
        np.testing.assert_allclose(out[0, h], sdpa(x["q_dec"][0, 0, h], x["K"][0, kv], x["V"][0, kv]),
                                   rtol=1e-12, atol=1e-14)


def test_zero_residual_is_eviction_over_main():
    wl, x = tiny(2)
    c = built(wl, x, res=[[0, 0]])
    out, *_ = orc.decode(x["q_dec"][1], c["kc"], c["vc"], c["logc"], c["res_len"], c["main_len"],
                         0.25, 12.0, 0.0, 1.0)
    for h in range(wl.hq):
        kv = h // wl.group
        idx = c["main_idx"][0, kv, :c["main_len"][0, kv]]
        np.testing.assert_allclose(out[0, h], sdpa(x["q_dec"][1, 0, h], x["K"][0, kv, idx], x["V"][0, kv, idx]),
                                   rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_singleton_residuals_reproduce_full_attention(dtype):
    """Entries built from one evicted token each are exact tokens; with the gate
    held at 1 the main + residual layout reproduces full attention (R12).
    A fixed budget always evicts more tokens than it has residual slots, so
    the singleton entries are formed here from the built main set directly."""
    wl, x = tiny(3, s=30, budget=24, res=10, dtype=dtype)
    c = built(wl, x)
    for kv in range(wl.hkv):
        rec = c["records"][(0, kv)]
        E = rec["evicted"]
        K, V = x["K"][0, kv, :30], x["V"][0, kv, :30]
        kb, vb, cnt, logc = orc.residual_entries(K[E], V[E], np.arange(E.size), K[E], E.size, wl.d)
        assert (cnt == 1).all()
        m = c["main_len"][0, kv]
        r = c["res_len"][0, kv]
        Km = c["kc"][0, kv, r:r + m]
        Vm = c["vc"][0, kv, r:r + m]
        for h in range(kv * wl.group, (kv + 1) * wl.group):
            q = x["q_dec"][0, 0, h]
            out, dbg = orc.decode_head(q, Km, Vm, orc.round_to_dtype(kb, dtype),
                                       orc.round_to_dtype(vb, dtype), logc, 0.25, 12.0, 1.0, 1.0)
            np.testing.assert_allclose(out, sdpa(q, K, V), rtol=1e-12, atol=1e-14)


def test_cache_layout_and_counts():
    wl, x = tiny(4, s=200, budget=40, res=12)
    c = built(wl, x)
    for kv in range(wl.hkv):
        rec = c["records"][(0, kv)]
        m = 40 - 12
        assert c["main_len"][0, kv] == m and c["res_len"][0, kv] == 12
        assert rec["counts"].sum() == 200 - m
        idx = c["main_idx"][0, kv, :m]
        assert (np.diff(idx) > 0).all()
        np.testing.assert_array_equal(c["kc"][0, kv, 12:12 + m], x["K"][0, kv, idx])
        np.testing.assert_array_equal(c["vc"][0, kv, 12:12 + m], x["V"][0, kv, idx])
        # protected recent window kept
        assert set(range(200 - wl.window, 200)) <= set(idx.tolist())
        # the residual entries are the means of their groups
        E = rec["evicted"]
        for j in range(12):
            mem = E[rec["assign"] == j]
            if mem.size:
                np.testing.assert_allclose(c["vc"][0, kv, j], x["V"][0, kv, mem].astype(float).mean(0), rtol=1e-6)


def test_bf16_storage_rounding():
    vals = np.array([1.0, 1.00390625, 1.005859375, 1.0 + 3 * 2 ** -9, -2.5e-39, 3.0e38, 1e39, 0.0])
    r = orc.round_to_dtype(vals, "bf16")
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa -> 1
    assert r[1] == 1.0
    assert r[2] == 1.0078125
    assert r[3] == 1.0 + 2 ** -7
    assert r[6] == np.inf
    # agree with torch's float32 -> bf16 conversion on float32-representable input
    f = np.random.default_rng(0).normal(size=1000).astype(np.float32)
    t = torch.as_tensor(f).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(orc.round_to_dtype(f.astype(np.float64), "bf16"), t)


def test_heavy_tokens_are_kept():
    """On the synthetic workload the window queries attend to heavy keys, so
    the selection keeps them (a sanity check of score direction)."""
    wl = synth.tiny_workload(s=400, d=16, budget=64, res=8, window=8, n_heavy=6)
    rng_heavy = None
    x = synth.gen_layer(wl, 0, seed=5, n_decode=1)
    c = built(wl, x)
    for kv in range(wl.hkv):
        norms = np.linalg.norm(x["K"][0, kv], axis=1)
        heavy = np.argsort(-norms)[:6]
        assert set(heavy.tolist()) <= set(c["main_idx"][0, kv, :56].tolist())
