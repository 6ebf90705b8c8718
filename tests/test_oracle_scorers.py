"""Pins for the oracle's score pooling and the alternative scorers of
App. B.2.2 (compared methods): H2O (accumulated attention of the
observation queries, no pooling, 64 protected recent tokens) and TOVA
(last-token window, no pooling, 1 protected recent token), both feeding the
same selection and residual path (readings R23, R24)."""

import math

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc


@pytest.mark.parametrize("k", [1, 3, 5, 7, 9])
@pytest.mark.parametrize("n", [1, 2, 4, 6, 9, 40])
def test_pool_is_zero_padded_convolution(k, n):
    raw = np.random.default_rng(k * 100 + n).random(n)
    want = np.convolve(raw, np.ones(k), mode="full")[k // 2:k // 2 + n]
    np.testing.assert_allclose(orc.pool(raw, k), want, rtol=1e-14, atol=0)


def test_pool_one_is_identity_and_pool5_is_snapkv():
    raw = np.random.default_rng(1).random(37)
    assert np.array_equal(orc.pool(raw, 1), raw)
    assert np.array_equal(orc.pool5(raw), orc.pool(raw, 5))


def torch_softmax_rows(q, K):
    lg = torch.as_tensor(K) @ torch.as_tensor(q) / math.sqrt(K.shape[1])
    return torch.softmax(lg, dim=0).numpy()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tova_scores_are_last_query_attention(seed):
    """w = 1: each head's last prefill query attends to every token; the
    score of position p is the sum over the G heads of its softmax weight."""
    rng = np.random.default_rng(seed)
    s, d, G, m, r = 60, 8, 3, 20, 4
    K, V = rng.normal(size=(s, d)), rng.normal(size=(s, d))
    Qw = rng.normal(size=(G, 1, d))
    rec = orc.build_head(K, V, Qw, m, r, 1, 3, "f32", pool_kernel=1)
    w = sum(torch_softmax_rows(Qw[h, 0], K) for h in range(G))
    n = s - 1  # one protected token
    np.testing.assert_allclose(rec["scores"], w[:n], rtol=1e-12)
    # main = the last token + the top m - 1 by score (ties to the lower position)
    order = np.lexsort((np.arange(n), -w[:n]))
    want = np.sort(np.concatenate([order[:m - 1], [s - 1]]))
    np.testing.assert_array_equal(rec["main_idx"], want)


def test_h2o_scores_are_unpooled_window_mass():
    """Pool kernel 1: the scores are the accumulated causal attention of the
    observation queries, computed here with torch softmax row by row."""
    rng = np.random.default_rng(5)
    s, d, G, w, m, recent = 200, 8, 2, 6, 90, 64
    K, V = rng.normal(size=(s, d)), rng.normal(size=(s, d))
    Qw = rng.normal(size=(G, w, d))
    rec = orc.build_head(K, V, Qw, m, 8, recent, 3, "f32", pool_kernel=1)
    acc = np.zeros(s)
    for h in range(G):
        for i in range(w):
            pos = s - w + i
            acc[:pos + 1] += torch_softmax_rows(Qw[h, i], K[:pos + 1])
    n = s - recent
    np.testing.assert_allclose(rec["scores"], acc[:n], rtol=1e-12)
    assert set(range(n, s)) <= set(rec["main_idx"].tolist())  # the 64 recent tokens are kept
    assert rec["main_idx"].size == m


def test_pooling_changes_selection():
    """The same inputs select differently with and without pooling (so the
    pool kernel reaches the selection)."""
    rng = np.random.default_rng(9)
    s, d, G, w = 300, 8, 2, 8
    K, V = rng.normal(size=(s, d)), rng.normal(size=(s, d))
    Qw = rng.normal(size=(G, w, d))
    a = orc.build_head(K, V, Qw, 60, 0, 8, 2, "f32", pool_kernel=1)["main_idx"]
    b = orc.build_head(K, V, Qw, 60, 0, 8, 2, "f32", pool_kernel=5)["main_idx"]
    assert not np.array_equal(a, b)
