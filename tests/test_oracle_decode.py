"""Pins for the oracle's decode (Sec. 3.1, 3.2, 4.2, 5.4, 5.5.2; App. A.1-A.2).

Each test checks the oracle against something other than itself: a library
attention routine, a closed form, or a hand-derived example.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def sdpa(q, K, V):
    """torch's scaled_dot_product_attention in float64 on the CPU."""
    q = torch.as_tensor(np.asarray(q), dtype=torch.float64)[None, None, None, :]
    K = torch.as_tensor(np.asarray(K), dtype=torch.float64)[None, None]
    V = torch.as_tensor(np.asarray(V), dtype=torch.float64)[None, None]
    return torch.nn.functional.scaled_dot_product_attention(q, K, V)[0, 0, 0].numpy()


def rand_qkv(seed, s=37, d=16, scale=1.5):
    rng = np.random.default_rng(seed)
    return (rng.normal(size=d) * scale, rng.normal(size=(s, d)), rng.normal(size=(s, d)))


def test_hand_example_golden():
    g = json.load(open(os.path.join(GOLD, "decode_hand_example.json")))
    ln3 = math.log(3.0)
    km = np.array([[0, 0, 0, 0], [ln3, 0, 0, 0]], float)
    out, dbg = orc.decode_head(np.array(g["q"]), km, np.array(g["v_main"]),
                               np.array(g["k_res"]), np.array(g["v_res"]),
                               np.log(np.array(g["count_res"], float)),
                               g["tau"], g["alpha"], g["g_min"], g["beta"])
    gate = 1.0 / (1.0 + math.exp(6.0))
    assert dbg["p_max"] == pytest.approx(0.75, rel=1e-15)
    assert dbg["gate"] == pytest.approx(gate, rel=1e-14)
    expect = np.array([1.0, 3.0, 2 * gate, 0.0]) / (4 + 2 * gate)
    np.testing.assert_allclose(out, expect, rtol=1e-14, atol=1e-16)


def test_full_attention_matches_library():
    for seed in range(5):
        q, K, V = rand_qkv(seed)
        np.testing.assert_allclose(orc.full_attention(q, K, V), sdpa(q, K, V), rtol=1e-12, atol=1e-14)


def test_no_residual_is_eviction_attention():
    """R = empty reduces the shared softmax to eviction attention (Sec. 3.2, 5.4)."""
    for seed in range(5):
        q, K, V = rand_qkv(seed)
        kept = np.sort(np.random.default_rng(seed).choice(K.shape[0], 11, replace=False))
        out, _ = orc.decode_head(q, K[kept], V[kept], np.zeros((0, K.shape[1])),
                                 np.zeros((0, K.shape[1])), np.zeros(0), 0.25, 12.0, 0.0, 1.0)
        np.testing.assert_allclose(out, sdpa(q, K[kept], V[kept]), rtol=1e-12, atol=1e-14)
        # the oracle's eviction attention over the kept rows (Sec. 3.2) is
        # the same library result, and equals the r = 0 decode
        ev = orc.evict_attention(q, K, V, kept)
        np.testing.assert_allclose(ev, sdpa(q, K[kept], V[kept]), rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(out, ev, rtol=1e-12, atol=1e-14)
    # unsorted kept indices select the same rows
    q, K, V = rand_qkv(11)
    kept = np.array([30, 2, 17, 5])
    np.testing.assert_allclose(orc.evict_attention(q, K, V, kept), sdpa(q, K[np.sort(kept)], V[np.sort(kept)]),
                               rtol=1e-12, atol=1e-14)


def test_empty_entries_contribute_nothing():
    q, K, V = rand_qkv(3)
    kept = np.arange(20)
    o0, _ = orc.decode_head(q, K[kept], V[kept], np.zeros((0, 16)), np.zeros((0, 16)),
                            np.zeros(0), 0.25, 12.0, 0.0, 1.0)
    o1, d1 = orc.decode_head(q, K[kept], V[kept], K[20:23], V[20:23],
                             np.array([-np.inf] * 3), 0.25, 12.0, 0.0, 1.0)
    np.testing.assert_array_equal(o0, o1)
    assert d1["lse_res"] == -np.inf


def test_singleton_entries_with_gate_off_give_full_attention():
    """c_j = 1 entries are exact tokens; with g = 1 the shared softmax is full
    attention (Sec. 5.3 entry reconstruction; reading R12)."""
    for seed in range(5):
        q, K, V = rand_qkv(seed)
        M = np.arange(0, 37, 3)
        E = np.setdiff1d(np.arange(37), M)
        out, dbg = orc.decode_head(q, K[M], V[M], K[E], V[E], np.zeros(E.size), 0.25, 12.0, 1.0, 1.0)
        assert dbg["gate"] == 1.0
        np.testing.assert_allclose(out, sdpa(q, K, V), rtol=1e-12, atol=1e-14)


def test_lse_split_and_decomposition():
    """Z_S = Z_M + Z_E and N_S = N_M + N_E (Sec. 4.2; App. A.1)."""
    for seed in range(5):
        q, K, V = rand_qkv(seed, scale=3.0)
        rng = np.random.default_rng(100 + seed)
        M = np.sort(rng.choice(37, 15, replace=False))
        E = np.setdiff1d(np.arange(37), M)
        zS, nS, cS = orc.zn_stats(q, K, V, np.arange(37))
        zM, nM, cM = orc.zn_stats(q, K, V, M)
        zE, nE, cE = orc.zn_stats(q, K, V, E)
        a = torch.as_tensor(K @ q / 4.0)
        lse_lib = float(torch.logsumexp(a, 0))
        assert math.log(zS) + cS == pytest.approx(lse_lib, rel=1e-13)
        assert np.logaddexp(math.log(zM) + cM, math.log(zE) + cE) == pytest.approx(lse_lib, rel=1e-13)
        np.testing.assert_allclose(nM * math.exp(cM - cS) + nE * math.exp(cE - cS), nS, rtol=1e-12)
        np.testing.assert_allclose(nS / zS, sdpa(q, K, V), rtol=1e-12, atol=1e-14)


def test_eviction_error_closed_form():
    """o_S - o_M = (Z_M N_E - Z_E N_M) / (Z_M (Z_M + Z_E))  (App. A.1)."""
    for seed in range(5):
        q, K, V = rand_qkv(seed, scale=2.0)
        rng = np.random.default_rng(200 + seed)
        M = np.sort(rng.choice(37, 9, replace=False))
        E = np.setdiff1d(np.arange(37), M)
        zM, nM, cM = orc.zn_stats(q, K, V, M)
        zE, nE, cE = orc.zn_stats(q, K, V, E)
        c = max(cM, cE)
        zM, nM = zM * math.exp(cM - c), nM * math.exp(cM - c)
        zE, nE = zE * math.exp(cE - c), nE * math.exp(cE - c)
        closed = (zM * nE - zE * nM) / (zM * (zM + zE))
        np.testing.assert_allclose(closed, sdpa(q, K, V) - sdpa(q, K[M], V[M]), rtol=1e-9, atol=1e-13)


def test_residual_entry_error_bounds():
    """|Z_j - c e^{abar}| <= c e^{abar}(e^eta - 1) and the numerator bound with
    V = max ||v_p|| (App. A.2), for the oracle's own residual entries."""
    rng = np.random.default_rng(7)
    d = 8
    for trial in range(20):
        c = int(rng.integers(1, 9))
        center = rng.normal(size=d)
        KE = center + rng.normal(scale=0.3, size=(c, d))
        VE = rng.normal(size=(c, d))
        kbar, vbar, cnt, logc = orc.residual_entries(KE, VE, np.zeros(c, np.int64), KE.mean(0, keepdims=True), 1, d)
        q = rng.normal(size=d) * 2
        abar = float(kbar[0] @ q) / math.sqrt(d)
        a = KE @ q / math.sqrt(d)
        eta = float(np.abs(a - abar).max())
        Zj = float(np.exp(a).sum())
        Nj = np.exp(a) @ VE
        approx_z = cnt[0] * math.exp(abar)
        assert abs(Zj - approx_z) <= approx_z * ((math.exp(eta) - 1) * (1 + 1e-12) + 1e-14)
        Vmax = float(np.linalg.norm(VE, axis=1).max())
        err = float(np.linalg.norm(Nj - approx_z * vbar[0]))
        assert err <= approx_z * Vmax * ((math.exp(eta) - 1) * (1 + 1e-9) + 1e-13)


def test_gate_closed_forms():
    """p_max is the largest main-only attention weight; g = max(g_min,
    sigmoid((tau - p_max) * alpha)) (Sec. 5.5.2)."""
    q, K, V = rand_qkv(11, scale=2.0)
    _, dbg = orc.decode_head(q, K, V, np.zeros((0, 16)), np.zeros((0, 16)), np.zeros(0), 0.25, 12.0, 0.0, 1.0)
    w = torch.softmax(torch.as_tensor(K @ q / 4.0), 0)
    assert dbg["p_max"] == pytest.approx(float(w.max()), rel=1e-13)
    p = dbg["p_max"]
    assert orc.gate_value(p, p, 12.0, 0.0) == 0.5
    assert orc.gate_value(p, 0.3, 12.0, 1.0) == 1.0
    assert orc.gate_value(0.75, 0.25, 12.0, 0.0) == pytest.approx(1 / (1 + math.exp(6)), rel=1e-14)
    taus = np.linspace(-2, 2, 41)
    gs = [orc.gate_value(p, t, 12.0, 0.0) for t in taus]
    assert all(b >= a for a, b in zip(gs, gs[1:]))
    assert orc.gate_value(p, 0.0, 12.0, 0.3) >= 0.3


def test_uniform_logits_closed_form():
    """q = 0: every logit is 0, p_max = 1/m, and the output is
    (sum_M v + g sum_j c_j vbar_j) / (m + g sum_j c_j)."""
    rng = np.random.default_rng(5)
    m, r, d = 7, 3, 6
    Km, Vm = rng.normal(size=(m, d)), rng.normal(size=(m, d))
    Kr, Vr = rng.normal(size=(r, d)), rng.normal(size=(r, d))
    cnt = np.array([4.0, 1.0, 9.0])
    out, dbg = orc.decode_head(np.zeros(d), Km, Vm, Kr, Vr, np.log(cnt), 0.25, 12.0, 0.0, 1.0)
    g = 1.0 / (1.0 + math.exp(-(0.25 - 1.0 / m) * 12.0))
    assert dbg["gate"] == pytest.approx(g, rel=1e-14)
    expect = (Vm.sum(0) + g * (cnt[:, None] * Vr).sum(0)) / (m + g * cnt.sum())
    np.testing.assert_allclose(out, expect, rtol=1e-13)
    # beta = 0.5 puts c_j^0.5 in place of c_j
    out2, _ = orc.decode_head(np.zeros(d), Km, Vm, Kr, Vr, np.log(cnt), 0.25, 12.0, 0.0, 0.5)
    c2 = np.sqrt(cnt)
    np.testing.assert_allclose(out2, (Vm.sum(0) + g * (c2[:, None] * Vr).sum(0)) / (m + g * c2.sum()), rtol=1e-13)


def test_slot_permutation_invariance():
    q, K, V = rand_qkv(21)
    rng = np.random.default_rng(1)
    Km, Vm, Kr, Vr = K[:20], V[:20], K[20:30], V[20:30]
    logc = np.log(rng.integers(1, 6, size=10).astype(float))
    o1, _ = orc.decode_head(q, Km, Vm, Kr, Vr, logc, 0.1, 12.0, 0.0, 1.0)
    pm, pr = rng.permutation(20), rng.permutation(10)
    o2, _ = orc.decode_head(q, Km[pm], Vm[pm], Kr[pr], Vr[pr], logc[pr], 0.1, 12.0, 0.0, 1.0)
    np.testing.assert_allclose(o1, o2, rtol=1e-13)


def test_batched_decode_gqa_mapping():
    """Query head h reads KV head h // (Hq/Hkv)."""
    rng = np.random.default_rng(9)
    B, Hq, Hkv, C, d = 2, 6, 2, 12, 4
    q = rng.normal(size=(B, Hq, d))
    kc, vc = rng.normal(size=(B, Hkv, C, d)), rng.normal(size=(B, Hkv, C, d))
    logc = np.log(rng.integers(1, 4, size=(B, Hkv, 3)).astype(float))
    res_len = np.full((B, Hkv), 3)
    main_len = np.array([[9, 5], [7, 8]])
    out, lm, lr, gate = orc.decode(q, kc, vc, logc, res_len, main_len, 0.25, 12.0, 1.0, 1.0)
    for b in range(B):
        for h in range(Hq):
            kv = h // 3
            n = main_len[b, kv]
            K = np.concatenate([kc[b, kv, 3:3 + n], kc[b, kv, :3]])
            V = np.concatenate([vc[b, kv, 3:3 + n], vc[b, kv, :3]])
            # with g = 1 the residual entries are tokens with log-count offsets:
            # repeat each entry c_j times to reach plain attention
            cnt = np.exp(logc[b, kv]).round().astype(int)
            Kx = np.concatenate([K[:n]] + [np.repeat(K[n + j:n + j + 1], cnt[j], 0) for j in range(3)])
            Vx = np.concatenate([V[:n]] + [np.repeat(V[n + j:n + j + 1], cnt[j], 0) for j in range(3)])
            np.testing.assert_allclose(out[b, h], sdpa(q[b, h], Kx, Vx), rtol=1e-12, atol=1e-14)
