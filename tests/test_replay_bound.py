"""The Lloyd-replay tolerance of the construction checks (Sec. 5.3 partition
objective, solved by Lloyd rounds, App. B.3) is tight enough to tell a
distance computed with the split-bf16 centres (hi + lo) from one that drops
the lo part, and loose enough for fp32 accumulation in any order.

The "kernel" assignments below are simulated on the CPU from the same
definition (argmin over ||mu||^2 - 2 k.mu with the centres stored as the
kernel stores them, products summed in float32); the replay itself is the
one the GPU parity tests run (tests/build_check.replay_round)."""

import numpy as np
import pytest

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import synth
from tests.build_check import replay_round


def head(dtype, d, s=8192, budget=512, r=64, seed=5):
    wl = synth.tiny_workload(s=s, d=d, hq=4, hkv=1, budget=budget, res=r, window=32, n_heavy=16, dtype=dtype)
    x = synth.gen_layer(wl, 0, seed=seed, n_decode=1)
    K = x["K"][0, 0].astype(np.float64)
    Qw = x["q_obs"][0].astype(np.float64)
    m = budget - r
    n = orc.scored_length(s, m, 32)
    sc = orc.pool5(orc.window_raw_scores(K, Qw)[:n])
    _, ev, seeds = orc.select_main(sc, s, m, 32, r)
    return K[ev], K[seeds]


def split(mu32):
    hi = orc.round_to_dtype(mu32, "bf16")
    lo = orc.round_to_dtype(mu32 - hi, "bf16")
    return hi, lo


def kernel_like(KE, mu, mode):
    """Assignment as a kernel would make it: centres rounded to fp32 (and for
    bf16 split into hi + lo, or hi only), products summed in float32."""
    mu32 = mu.astype(np.float32).astype(np.float64)
    nrm = np.float32((mu32 * mu32).sum(axis=1))
    k32 = KE.astype(np.float32)
    if mode == "f32":
        acc = k32 @ mu32.astype(np.float32).T
    else:
        hi, lo = split(mu32)
        acc = k32 @ hi.astype(np.float32).T
        if mode == "hi+lo":
            acc = acc + k32 @ lo.astype(np.float32).T
    delta = nrm[None, :] - np.float32(2.0) * acc
    return np.argmin(delta, axis=1)


def rounds(KE, seeds, mode, dtype, T=4):
    """T simulated rounds, each replayed against the exact fp64 means of the
    previous round's groups; returns the number of tokens outside the bound
    per round."""
    mu = seeds.copy()
    out = []
    for _ in range(T):
        a = kernel_like(KE, mu, mode)
        bad, _ = replay_round(KE, mu, a, dtype)
        out.append(int(bad.sum()))
        for j in range(mu.shape[0]):
            mem = a == j
            if mem.any():
                mu[j] = KE[mem].mean(axis=0)
    return out


def test_replay_ranking_is_the_oracle_distance():
    """The replay ranks by ||mu||^2 - 2 k.mu; its argmin equals the oracle's
    direct-difference nearest centre."""
    KE, seeds = head("bf16", 128, s=2048, budget=256, r=16)
    a_ref, dist = orc.assign_nearest(KE, seeds)
    bad, worst = replay_round(KE, seeds, a_ref, "bf16")
    assert not bad.any() and worst <= 0.0


def test_split_bf16_passes_and_hi_only_fails():
    KE, seeds = head("bf16", 128)
    ok = rounds(KE, seeds, "hi+lo", "bf16")
    assert sum(ok) == 0, ok
    # the first round's centres are bf16 keys (lo = 0): only later rounds can
    # tell hi-only from hi + lo
    bad = rounds(KE, seeds, "hi", "bf16")
    assert sum(bad[1:]) >= 10, bad


def test_fp32_cache_passes():
    KE, seeds = head("f32", 64, s=4096, budget=256, r=32)
    assert sum(rounds(KE, seeds, "f32", "f32")) == 0


def test_planted_second_best_is_caught():
    """Moving one token with a clear gap to its second-nearest centre is
    outside the bound."""
    KE, seeds = head("bf16", 128, s=2048, budget=256, r=16)
    a, dist = orc.assign_nearest(KE, seeds)
    srt = np.sort(dist, axis=1)
    p = int(np.argmax(srt[:, 1] - srt[:, 0]))
    a2 = a.copy()
    a2[p] = int(np.argsort(dist[p])[1])
    bad, worst = replay_round(KE, seeds, a2, "bf16")
    assert bad.sum() == 1 and bad[p] and worst > 1.0


@pytest.mark.parametrize("d", [64, 128])
def test_bound_scale(d):
    """At the workload's shapes the bound is typically a few 1e-5 of the
    distance itself (||k - mu||^2), the relative scale the parity contract
    names."""
    KE, seeds = head("bf16", d, s=2048, budget=256, r=16)
    mu = seeds
    nrm = (mu * mu).sum(axis=1)
    A = np.abs(KE) @ np.abs(mu).T
    dist = (KE * KE).sum(axis=1)[:, None] + nrm[None, :] - 2 * KE @ mu.T
    e = 2.0 * (2.0 ** -16 + 2.0 ** -24 + 2 * d * 2.0 ** -24) * A
    live = dist > 0  # a seed token sits on its own centre
    rel = np.median(2 * e[live] / dist[live])
    assert rel < 1e-4, rel
