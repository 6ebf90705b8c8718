"""Pins for the oracle's construction-time validation proxy (Sec. 5.5.1,
validation-loss and margin equations; App. D, Algorithm 1; App. B.3 for the
grid, the 96/32 query split and delta).
"""

import math

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc

GRID = [0.0, 0.05, 0.10, 0.15, 0.20]


def sdpa(q, K, V):
    q = torch.as_tensor(np.asarray(q), dtype=torch.float64)[None, None, None, :]
    K = torch.as_tensor(np.asarray(K), dtype=torch.float64)[None, None]
    V = torch.as_tensor(np.asarray(V), dtype=torch.float64)[None, None]
    return torch.nn.functional.scaled_dot_product_attention(q, K, V)[0, 0, 0].numpy()


def test_candidate_counts_closed_form():
    # 0.05 * 2048 = 102.4, 0.10 * 2048 = 204.8, ... rounded to nearest
    assert orc.candidate_counts(2048, GRID) == [0, 102, 205, 307, 410]
    assert orc.candidate_counts(512, GRID) == [0, 26, 51, 77, 102]
    assert orc.candidate_counts(40, [0.0, 0.0625, 0.1875]) == [0, 3, 8]  # 2.5 -> 3, 7.5 -> 8


@pytest.mark.parametrize("losses,counts,delta,want", [
    ([1.0, 0.5, 0.7], [0, 8, 16], 0.01, 8),           # clear win
    ([1.0, 0.995, 0.999], [0, 8, 16], 0.01, 0),       # inside the margin
    ([1.0, 0.989, 0.999], [0, 8, 16], 0.01, 8),       # just outside the margin
    ([1.0, 0.5, 0.5], [0, 16, 8], 0.0, 8),            # tie among r > 0 -> smaller r
    ([0.0, 0.0, 0.0], [0, 8, 16], 0.01, 0),           # nothing to gain
    ([1.0, 0.2, 0.4], [0, 8, 16], 1.0, 0),            # delta = 1 never enables
    ([0.5, 1.0], [8, 0], 0.0, 8),                     # the zero count need not come first
])
def test_proxy_choice_rule(losses, counts, delta, want):
    r, i = orc.proxy_choice(losses, counts, delta)
    assert r == want and counts[i] == want


def brute_fit_raw(K, Qw, fit):
    """Loops: fit row (h, i) at position s - w + i, softmax over keys <= pos."""
    s, d = K.shape
    G, w, _ = Qw.shape
    raw = np.zeros(s)
    for h in range(G):
        for i in range(fit):
            pos = s - w + i
            lg = [float(Qw[h, i] @ K[p]) / math.sqrt(d) for p in range(pos + 1)]
            top = max(lg)
            e = [math.exp(x - top) for x in lg]
            z = sum(e)
            for p in range(pos + 1):
                raw[p] += e[p] / z
    return raw


@pytest.mark.parametrize("seed", [0, 1])
def test_fit_rows_keep_their_window_positions(seed):
    rng = np.random.default_rng(seed)
    s, d, G, w, fit = 14, 4, 2, 5, 3
    K, Qw = rng.normal(size=(s, d)), rng.normal(size=(G, w, d))
    np.testing.assert_allclose(orc.window_raw_scores(K, Qw, fit), brute_fit_raw(K, Qw, fit), rtol=1e-12)
    # scoring with only the fit rows differs from scoring the whole window
    assert not np.allclose(orc.window_raw_scores(K, Qw, fit), orc.window_raw_scores(K, Qw))


def test_zero_budget_loss_is_eviction_error():
    """L_0 = mean over validation queries of ||attention over M - full attention||^2,
    computed independently with torch SDPA over the kept rows."""
    rng = np.random.default_rng(3)
    s, d, G, w, val = 80, 8, 2, 8, 2
    K, V, Qw = rng.normal(size=(s, d)), rng.normal(size=(s, d)), rng.normal(size=(G, w, d))
    res = orc.validation_proxy(K, V, Qw, 32, GRID, 4, 3, val, 0.01, 0.25, 12.0, 0.0, 1.0, "f32")
    assert res["counts"][0] == 0
    main = res["records"][0]["main_idx"]
    vq = Qw[:, w - val:].reshape(-1, d)
    want = np.mean([((sdpa(q, K[main], V[main]) - sdpa(q, K, V)) ** 2).sum() for q in vq])
    assert abs(res["losses"][0] - want) <= 1e-12 * max(1.0, want)


def test_candidate_loss_matches_gated_decode_of_its_cache():
    """Each candidate's loss is the mean squared error of the oracle decode
    over that candidate's own cache (the decode itself is pinned elsewhere)."""
    rng = np.random.default_rng(4)
    s, d, G, w, val = 90, 8, 2, 8, 2
    K, V, Qw = rng.normal(size=(s, d)), rng.normal(size=(s, d)), rng.normal(size=(G, w, d))
    res = orc.validation_proxy(K, V, Qw, 40, GRID, 4, 3, val, 0.01, 0.25, 12.0, 0.0, 1.0, "f32")
    vq = Qw[:, w - val:].reshape(-1, d)
    for r, rec, loss in zip(res["counts"], res["records"], res["losses"]):
        assert rec["res_len"] == r and rec["main_len"] == 40 - r
        n = rec["main_len"]
        errs = []
        for q in vq:
            o, _ = orc.decode_head(q, rec["kc"][r:r + n], rec["vc"][r:r + n], rec["kc"][:r], rec["vc"][:r],
                                   rec["logc"], 0.25, 12.0, 0.0, 1.0)
            errs.append(((o - sdpa(q, K, V)) ** 2).sum())
        assert abs(loss - np.mean(errs)) <= 1e-12 * max(1.0, loss)


def test_no_eviction_keeps_zero():
    """s <= b - max r: every candidate keeps every token, the losses are
    identical and the proxy keeps r = 0."""
    rng = np.random.default_rng(5)
    s, d, G, w = 20, 4, 2, 6
    K, V, Qw = rng.normal(size=(s, d)), rng.normal(size=(s, d)), rng.normal(size=(G, w, d))
    res = orc.validation_proxy(K, V, Qw, 40, GRID, 4, 3, 2, 0.01, 0.25, 12.0, 0.0, 1.0, "f32")
    assert res["r"] == 0
    assert max(res["losses"]) <= 1e-25
    assert len(set(res["losses"])) == 1


def test_chosen_record_is_the_build_with_that_count():
    rng = np.random.default_rng(6)
    s, d, G, w, val = 100, 8, 2, 8, 2
    K, V, Qw = rng.normal(size=(s, d)), rng.normal(size=(s, d)), rng.normal(size=(G, w, d))
    res = orc.validation_proxy(K, V, Qw, 40, GRID, 4, 3, val, 0.01, 0.25, 12.0, 0.0, 1.0, "f32")
    r = res["r"]
    rec = orc.build_head(K, V, Qw, 40 - r, r, 4, 3, "f32", fit_rows=w - val)
    np.testing.assert_array_equal(rec["main_idx"], res["record"]["main_idx"])
    np.testing.assert_array_equal(rec["kc"], res["record"]["kc"])
    assert r in res["counts"]
    r_star = min((x for x in zip(res["losses"], res["counts"]) if x[1] > 0))
    if r > 0:
        assert r == r_star[1] and r_star[0] < 0.99 * res["losses"][0]
    else:
        assert r_star[0] >= 0.99 * res["losses"][0]


def test_diffuse_heads_gain_from_residuals():
    """A group of many similar evicted tokens carries mass the main cache
    cannot: with diffuse validation queries some r > 0 must win."""
    rng = np.random.default_rng(7)
    s, d, G, w, val = 160, 8, 2, 8, 4
    base = rng.normal(size=d)
    K = 0.05 * rng.normal(size=(s, d)) + base        # near-identical keys: diffuse attention
    V = rng.normal(size=(s, d))
    Qw = 0.3 * rng.normal(size=(G, w, d))
    res = orc.validation_proxy(K, V, Qw, 48, GRID, 4, 4, val, 0.01, 0.25, 12.0, 0.0, 1.0, "f32")
    assert res["r"] > 0
    assert min(res["losses"][1:]) < 0.99 * res["losses"][0]
