"""Pins for the oracle's two-branch decode (Sec. 6.1: main branch and
residual branch merged through log-sum-exp statistics) and the ablation
with separate normalisations (Sec. 6.6 ablation table; reading R25, parity
unpinned against the paper, pinned to its limits here)."""

import math

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc


def sdpa(q, K, V, bias=None):
    q = torch.as_tensor(np.asarray(q, np.float64))[None, None, None, :]
    K = torch.as_tensor(np.asarray(K, np.float64))[None, None]
    V = torch.as_tensor(np.asarray(V, np.float64))[None, None]
    mask = None if bias is None else torch.as_tensor(np.asarray(bias, np.float64))[None, None, None, :]
    return torch.nn.functional.scaled_dot_product_attention(q, K, V, attn_mask=mask)[0, 0, 0].numpy()


def case(seed, n=40, r=6, d=16, empty=(2,)):
    rng = np.random.default_rng(seed)
    q = rng.normal(size=d)
    Km, Vm = rng.normal(size=(n, d)), rng.normal(size=(n, d))
    Kr, Vr = rng.normal(size=(r, d)), rng.normal(size=(r, d))
    logc = np.log(rng.integers(1, 30, size=r).astype(float))
    for j in empty:
        logc[j] = -np.inf
    return q, Km, Vm, Kr, Vr, logc


@pytest.mark.parametrize("seed", range(4))
def test_branches_against_torch(seed):
    q, Km, Vm, Kr, Vr, logc = case(seed)
    beta = 0.7
    om, lm, orr, lr = orc.decode_branches(q, Km, Vm, Kr, Vr, logc, beta)
    np.testing.assert_allclose(om, sdpa(q, Km, Vm), rtol=1e-12, atol=1e-14)
    lg = torch.as_tensor(Km @ q / math.sqrt(len(q)))
    assert lm == pytest.approx(float(torch.logsumexp(lg, 0)), rel=1e-13)
    live = np.isfinite(logc)
    np.testing.assert_allclose(orr, sdpa(q, Kr[live], Vr[live], beta * logc[live]), rtol=1e-12, atol=1e-14)
    lres = torch.as_tensor(Kr[live] @ q / math.sqrt(len(q)) + beta * logc[live])
    assert lr == pytest.approx(float(torch.logsumexp(lres, 0)), rel=1e-13)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("tau,g_min", [(0.25, 0.0), (0.9, 0.0), (-1.0, 0.3), (0.25, 1.0)])
def test_shared_merge_equals_shared_softmax_decode(seed, tau, g_min):
    """The log-sum-exp merge of the branches reproduces the single shared
    softmax of decode_head (Sec. 6.1)."""
    q, Km, Vm, Kr, Vr, logc = case(seed)
    out, dbg = orc.decode_head(q, Km, Vm, Kr, Vr, logc, tau, 12.0, g_min, 1.0)
    om, lm, orr, lr = orc.decode_branches(q, Km, Vm, Kr, Vr, logc, 1.0)
    merged = orc.merge_branches(om, lm, orr, lr, dbg["gate"], "shared")
    np.testing.assert_allclose(merged, out, rtol=1e-11, atol=1e-13)


def test_separate_merge_limits():
    q, Km, Vm, Kr, Vr, logc = case(7)
    om, lm, orr, lr = orc.decode_branches(q, Km, Vm, Kr, Vr, logc, 1.0)
    # g = 0: eviction attention over the main rows
    np.testing.assert_allclose(orc.merge_branches(om, lm, orr, lr, 0.0, "separate"), sdpa(q, Km, Vm), rtol=1e-12)
    # g = 1: the residual branch alone, softmax with the log-count bias
    live = np.isfinite(logc)
    np.testing.assert_allclose(orc.merge_branches(om, lm, orr, lr, 1.0, "separate"),
                               sdpa(q, Kr[live], Vr[live], logc[live]), rtol=1e-12)
    # no populated entry: the main branch whatever the gate
    none = np.full_like(logc, -np.inf)
    om2, lm2, or2, lr2 = orc.decode_branches(q, Km, Vm, Kr, Vr, none, 1.0)
    assert lr2 == -np.inf and not or2.any()
    np.testing.assert_allclose(orc.merge_branches(om2, lm2, or2, lr2, 0.8, "separate"), sdpa(q, Km, Vm), rtol=1e-12)
    # and the two merges differ when both branches carry mass
    g = 0.5
    assert not np.allclose(orc.merge_branches(om, lm, orr, lr, g, "separate"),
                           orc.merge_branches(om, lm, orr, lr, g, "shared"))
