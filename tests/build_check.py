"""Runs reskv_build_cache through the C ABI and checks it against the oracle.

Parity contract for construction (scores, selection, Lloyd, entries):
  * scores: |gpu - oracle| <= 1e-4 * |oracle| + 1e-30 per scored position;
  * selection from the GPU's own fp32 scores is exact: the oracle's selection
    run on those scores reproduces main_idx bit for bit;
  * main_idx equals the oracle's own fp64 selection except where the oracle's
    scores at the k_top boundary are closer than twice the score tolerance,
    absolute floor included (certified near-ties, counted and returned): a
    window row's probabilities below fp32's normal range are zero in the
    kernel, so where fewer than k_top positions score above the floor the
    kernel's choice among its zero scores is the lowest positions;
  * Lloyd replay: in every round each evicted token's GPU group is an
    eps-argmin of the fp64 distances to the centres the oracle recomputes from
    the GPU's previous round (the first round uses the seeds the oracle selects
    from the GPU scores), with eps the error bound of the kernel's distance
    arithmetic derived in replay_bound();
  * counts equal the oracle's recount of the GPU's last assignment; stored
    mean keys/values are within one storage ulp of the fp64 means of the GPU's
    groups (fp32 caches: 1e-6 relative); empty groups have log-count -inf.
"""

import math

import numpy as np
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import reskv as rk

SCORE_RTOL = 1e-4
SCORE_ATOL = 1e-30  # scores below fp32's normal range carry no relative precision


def to_dev(x, dtype):
    t = torch.as_tensor(np.asarray(x, np.float32))
    return (t.to(torch.bfloat16) if dtype == "bf16" else t).cuda().contiguous()


class HostView:
    """Host float64 copies of slices of a device tensor, made on indexing."""

    def __init__(self, t):
        self.t = t

    def __getitem__(self, idx):
        return self.t[idx].float().cpu().numpy().astype(np.float64)


def run_build(wl, x, layer=0, dbg=True, recent=None, iters=None, keep_device=False, host_cache=True, fit=0,
              res=None, pool=0, adakv=None, slot_cap=None, reserve=0, centers=True):
    """Build one layer on the GPU; returns host numpy copies of the outputs
    (and the device tensors under "dev" when keep_device is set). `fit` > 0
    scores with the leading `fit` window rows only; `res` overrides x["res"];
    `pool` is the pooling kernel (0: the default 5); `adakv` = a safeguard
    builds through reskv_build_cache_adakv with `reserve` slots per head kept
    for decode appends; `slot_cap` overrides C; `centers` (with `dbg`)
    exports every round's Lloyd centres."""
    B, Hkv, d = wl.batch, wl.hkv, wl.d
    S = x["K"].shape[2]
    C, Rcap = wl.slot_cap if slot_cap is None else slot_cap, wl.res_cap
    T = wl.lloyd_iters if iters is None else iters
    shape = rk.make_shape(B, wl.hq, Hkv, d, wl.dtype, C, Rcap)
    params = rk.BuildParams(S, wl.window, wl.window if recent is None else recent, T, fit, pool)
    res = np.asarray(x["res"] if res is None else res, np.int32).reshape(-1)
    K = x["K"] if torch.is_tensor(x["K"]) else to_dev(x["K"], wl.dtype)
    V = x["V"] if torch.is_tensor(x["V"]) else to_dev(x["V"], wl.dtype)
    Q = x["q_obs"] if torch.is_tensor(x["q_obs"]) else to_dev(x["q_obs"], wl.dtype)
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    kc = torch.full((B, Hkv, C, d), 7.0, dtype=tdt, device="cuda")
    vc = torch.full((B, Hkv, C, d), 7.0, dtype=tdt, device="cuda")
    logc = torch.full((B, Hkv, Rcap), 7.0, device="cuda")
    main_idx = torch.full((B, Hkv, C), -7, dtype=torch.int32, device="cuda")
    res_len = torch.full((B * Hkv,), -7, dtype=torch.int32, device="cuda")
    main_len = torch.full((B * Hkv,), -7, dtype=torch.int32, device="cuda")
    dbg_s = torch.empty((B, Hkv, S), device="cuda") if dbg else None
    dbg_a = torch.empty((T, B, Hkv, S), dtype=torch.int32, device="cuda") if dbg else None
    dbg_c = torch.full((T, B, Hkv, Rcap, d), float("nan"), device="cuda") if dbg and centers else None
    if adakv is None:
        nws = rk.reskv_build_workspace_size(shape, params, x["seq_len"], x["budget"], res)
    else:
        nws = rk.reskv_build_adakv_workspace_size(shape, params, adakv, reserve, x["seq_len"], x["budget"], res)
    assert nws > 0
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    if adakv is None:
        rk.reskv_build_cache(shape, params, K, V, x["seq_len"], Q, x["budget"], res, kc, vc, logc, main_idx,
                             res_len, main_len, ws, dbg_scores=dbg_s, dbg_assign=dbg_a, dbg_centers=dbg_c)
    else:
        rk.reskv_build_cache_adakv(shape, params, adakv, reserve, K, V, x["seq_len"], Q, x["budget"], res, kc, vc,
                                   logc, main_idx, res_len, main_len, ws, dbg_scores=dbg_s, dbg_assign=dbg_a,
                                   dbg_centers=dbg_c)
    torch.cuda.synchronize()
    out = dict(logc=logc.cpu().numpy().astype(np.float64), main_idx=main_idx.cpu().numpy(),
               res_len=res_len.cpu().numpy().reshape(B, Hkv), main_len=main_len.cpu().numpy().reshape(B, Hkv))
    if host_cache:
        out["kc"] = kc.float().cpu().numpy().astype(np.float64)
        out["vc"] = vc.float().cpu().numpy().astype(np.float64)
    else:
        out["kc"], out["vc"] = HostView(kc), HostView(vc)
    if keep_device:
        out["dev"] = dict(kc=kc, vc=vc, logc=logc, res_len=res_len, main_len=main_len, main_idx=main_idx)
    if dbg:
        out["scores"] = dbg_s.cpu().numpy().astype(np.float64)
        out["assign"] = dbg_a.cpu().numpy()
    if dbg_c is not None:
        out["centers"] = HostView(dbg_c)
    return out


def ulp(x, dtype):
    """Spacing of the storage format at |x| (bf16: 8 significant bits)."""
    x = np.abs(np.asarray(x, np.float64))
    if dtype == "bf16":
        e = np.floor(np.log2(np.maximum(x, 2.0 ** -126)))
        return np.exp2(e - 7)
    return np.maximum(x, 1e-30) * 2.0 ** -23


# Lloyd replay tolerance. The kernel ranks centres by
#   delta_pj = ||mu_j||^2 - 2 k_p . mu_j   (= ||k_p - mu_j||^2 - ||k_p||^2)
# with mu_j the fp32 rounding of the group mean; bf16 caches split mu_j into
# hi = bf16(mu_j) and lo = bf16(mu_j - hi), both rounded to nearest even, and
# run the products k . hi and k . lo on MFMA (bf16 x bf16 products are exact in
# fp32) with fp32 accumulation; ||mu_j||^2 is an fp64 sum rounded to fp32 and
# delta is formed by one fp32 fma. With A_pj = sum_i |k_pi| |mu_ji| and
# u = 2^-24, the kernel's delta differs from the exact one by at most
#   e_pj = 2 (u_split + u + gamma) A_pj + u (3 ||mu_j||^2 + |delta_pj|)
# where u_split = 2^-16 bounds |mu - hi - lo| / |mu| per element (lo's own
# rounding, 2^-8 of |mu - hi| <= 2^-8 |mu|), u covers the fp32 rounding of the
# mean, and gamma = n u bounds the fp32 accumulation of the n = 2D hi and lo
# products (worst case, any summation order). fp32 caches have no split
# (u_split = 0) and round each of the D products: gamma = (D + 1) u.
# A token assigned to a while the exact argmin is j* must satisfy
#   delta_pa - delta_pj* <= e_pa + e_pj*.
# A kernel that dropped the lo part would err by up to 2^-8 A (bf16 rounding
# of mu itself), 128 times the split term, and fails this bound.
U32 = 2.0 ** -24
U_SPLIT = 2.0 ** -16


def replay_bound(d, dtype):
    """(u_split, gamma) of the kernel's distance arithmetic at head_dim d."""
    if dtype == "bf16":
        return U_SPLIT, 2 * d * U32
    return 0.0, (d + 1) * U32


def replay_round(KE, mu, a, dtype):
    """Check one Lloyd round: the tokens KE [n, d] were assigned a [n] against
    centres mu [r', d] (fp64: the exact means of the previous round's
    groups). Returns (mask of tokens outside the bound, largest excess of the
    chosen centre over the exact best in units of the bound)."""
    KE = np.asarray(KE, np.float64)
    mu = np.asarray(mu, np.float64)
    n = KE.shape[0]
    nrm = (mu * mu).sum(axis=1)
    delta = nrm[None, :] - 2.0 * (KE @ mu.T)
    A = np.abs(KE) @ np.abs(mu).T
    u_split, gamma = replay_bound(KE.shape[1], dtype)
    e = 2.0 * (u_split + U32 + gamma) * A + U32 * (3.0 * nrm[None, :] + np.abs(delta))
    rows = np.arange(n)
    jstar = np.argmin(delta, axis=1)
    excess = delta[rows, a] - delta[rows, jstar]
    tol = e[rows, a] + e[rows, jstar]
    bad = excess > tol
    return bad, float((excess / tol).max()) if n else 0.0


def check_head(wl, x, got, b, h, recent=None, iters=None, full_oracle=True, replay=True, fit=None, r=None, pool=5,
               k_top=None, lloyd_info=True):
    """All construction checks for one (b, kv head). Returns a report dict.
    `fit` = leading window rows that scored (None: all); `r` overrides
    x["res"]; `pool` = pooling kernel; `k_top` = the head's top-k count when
    a cross-head allocation set it (None: the uniform m - |P|);
    `lloyd_info` also runs the oracle's own Lloyd from the same seeds and
    reports its agreement (information only, slow at full size)."""
    recent = wl.window if recent is None else recent
    T = wl.lloyd_iters if iters is None else iters
    G = wl.group
    s = int(x["seq_len"][b])
    r = int(x["res"][b][h]) if r is None else int(r)
    m = int(x["budget"][b]) - r
    K = np.asarray(x["K_host"][b, h, :s], np.float64)
    V = np.asarray(x["V_host"][b, h, :s], np.float64)
    Qw = np.asarray(x["q_host"][b, h * G:(h + 1) * G], np.float64)
    rep = dict(near_ties=0, lloyd_agree=None)
    assert got["res_len"][b, h] == r
    ml = int(got["main_len"][b, h])
    P = min(recent, m, s)
    kt = m - P if (k_top is None or s <= m) else int(k_top)
    assert ml == (s if s <= m else P + kt)
    midx = got["main_idx"][b, h, :ml].astype(np.int64)
    if s <= m:
        assert (midx == np.arange(s)).all()
        assert np.isinf(got["logc"][b, h, :r]).all() and (got["logc"][b, h, :r] < 0).all()
        np.testing.assert_array_equal(got["kc"][b, h, r:r + ml], K)
        return rep
    n = orc.scored_length(s, m, recent)
    gs = got["scores"][b, h, :n]
    # (ii) score parity
    if full_oracle:
        raw = orc.window_raw_scores(K, Qw, fit)
        ref = orc.pool(raw[:n], pool)
        err = np.abs(gs - ref)
        assert (err <= SCORE_RTOL * np.abs(ref) + SCORE_ATOL).all(), \
            f"score err {(err / np.maximum(np.abs(ref), 1e-30)).max():.2e}"
    # (i) exact selection on the GPU's own scores
    main_g, ev_g, seeds_g = orc.select_top(gs, s, n, kt, r)
    np.testing.assert_array_equal(midx, main_g)
    # (iii) end-to-end selection against the oracle's fp64 scores, with
    # certified near-ties at the k_top boundary
    if full_oracle:
        main_o, _, _ = orc.select_top(ref, s, n, kt, r)
        if not np.array_equal(main_o, main_g):
            srt = np.sort(ref)[::-1]
            gap = abs(srt[kt - 1] - srt[kt]) if 0 < kt < n else 0.0
            assert gap <= 2 * (SCORE_RTOL * srt[max(kt - 1, 0)] + SCORE_ATOL), \
                "selection differs outside a near-tie"
            rep["near_ties"] += 1
    # cache main rows are exact copies
    np.testing.assert_array_equal(got["kc"][b, h, r:r + ml], K[midx])
    np.testing.assert_array_equal(got["vc"][b, h, r:r + ml], V[midx])
    if r == 0 or not replay:
        return rep
    # (iv) Lloyd replay
    KE = K[ev_g]
    nE = ev_g.size
    r_eff = min(r, nE)
    mu = K[seeds_g].copy()
    assign = None
    rep["replay_worst"] = 0.0
    for it in range(T):
        a = got["assign"][it, b, h][ev_g]
        assert (a >= 0).all() and (a < r_eff).all()
        if "centers" in got:
            # the exported centres of this round are the fp32 roundings of the
            # means the oracle recomputes (round 0: the seed keys, exactly);
            # rows past r' are zero
            cg = got["centers"][it, b, h]
            ref32 = mu[:r_eff].astype(np.float32).astype(np.float64)
            ulp32 = np.spacing(np.abs(ref32).astype(np.float32)).astype(np.float64)
            assert (np.abs(cg[:r_eff] - ref32) <= ulp32).all(), f"round {it}: centres differ from the group means"
            if it == 0:
                np.testing.assert_array_equal(cg[:r_eff], K[seeds_g])
            assert (cg[r_eff:] == 0).all()
        bad, worst = replay_round(KE, mu[:r_eff], a, wl.dtype)
        rep["replay_worst"] = max(rep["replay_worst"], worst)
        assert not bad.any(), f"round {it}: {bad.sum()} tokens not at an eps-argmin (worst {worst:.2f} of the bound)"
        for j in range(r_eff):
            mem = a == j
            if mem.any():
                mu[j] = KE[mem].mean(axis=0)
        assign = a
    cnt = np.bincount(assign, minlength=r)
    lc = got["logc"][b, h, :r]
    for j in range(r):
        if cnt[j] == 0:
            assert lc[j] == -np.inf
            assert (got["vc"][b, h, j] == 0).all()
        else:
            assert abs(lc[j] - math.log(cnt[j])) <= 1e-6 * max(1.0, math.log(cnt[j]))
            km = KE[assign == j].mean(axis=0)
            vm = V[ev_g][assign == j].mean(axis=0)
            assert (np.abs(got["kc"][b, h, j] - km) <= ulp(km, wl.dtype) * 1.0001).all(), f"kbar {j}"
            assert (np.abs(got["vc"][b, h, j] - vm) <= ulp(vm, wl.dtype) * 1.0001).all(), f"vbar {j}"
    assert cnt.sum() == nE
    if full_oracle and lloyd_info:
        a_o, _, _ = orc.lloyd(KE, K[seeds_g], T)
        rep["lloyd_agree"] = float((a_o == assign).mean())
    return rep
