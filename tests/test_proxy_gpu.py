"""GPU parity of reskv_build_cache_proxy, the construction-time validation
proxy (Sec. 5.5.1, validation-loss and margin equations; App. D, Algorithm 1;
App. B.3 for the grid, the 96/32 fit/validation split and delta).

Per (b, kv head) the checks are:
  * every candidate cache, rebuilt alone by reskv_build_cache with the same
    count and the fit rows, passes the construction parity checks against the
    oracle (scores with the fit rows, exact selection, Lloyd replay, entries);
  * the GPU loss of every candidate agrees with the fp64 oracle loss of that
    candidate's GPU cache: |sqrt(L_gpu) - sqrt(L_ref)| <= E, where E bounds
    the RMS of two decode errors (the candidate's and the uncompressed
    reference's), each at most sqrt(d) * e_dec * max|o| in L2 for a
    per-element relative decode error e_dec: 2^-17 for bf16 caches (the
    probabilities enter the MFMA as a bf16 hi + lo pair, 16 significant
    bits), 1e-6 for fp32 caches (fp32 products and accumulation);
  * the chosen count follows the margin rule applied to the GPU's own fp32
    losses exactly (replayed in float32), and the outputs are bit-identical to
    the chosen candidate's cache;
  * the chosen count equals the oracle's own validation proxy (fp64 caches
    and losses) except where the oracle's decision is within the loss bound of
    flipping (certified near-ties, counted) or the oracle's candidate caches
    differ from the GPU's at a certified selection near-tie.
"""

import math

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import reskv as rk
from paper_2607_29591_amd import synth
from tests.build_check import check_head, run_build

pytestmark = pytest.mark.gpu

GRID = (0.0, 0.05, 0.10, 0.15, 0.20)
E_DEC = {"f32": 1e-6, "bf16": 8e-6}
GATE = dict(tau_scalar=0.25, alpha=12.0, g_min=0.0, beta=1.0)


def host_copies(x):
    x["K_host"], x["V_host"], x["q_host"] = x["K"], x["V"], x["q_obs"]
    return x


def to_dev(a, dtype):
    if torch.is_tensor(a):
        return a
    t = torch.as_tensor(np.asarray(a, np.float32))
    return (t.to(torch.bfloat16) if dtype == "bf16" else t).cuda().contiguous()


def run_proxy(wl, x, grid, val, delta, gate=GATE, recent=None):
    B, Hkv, d = wl.batch, wl.hkv, wl.d
    S = x["K"].shape[2]
    C, Rcap = wl.slot_cap, wl.res_cap
    shape = rk.make_shape(B, wl.hq, Hkv, d, wl.dtype, C, Rcap)
    params = rk.BuildParams(S, wl.window, wl.window if recent is None else recent, wl.lloyd_iters, 0)
    proxy = rk.make_proxy(grid, val, delta)
    g = rk.make_gate(**gate)
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    kc = torch.full((B, Hkv, C, d), 7.0, dtype=tdt, device="cuda")
    vc = torch.full((B, Hkv, C, d), 7.0, dtype=tdt, device="cuda")
    logc = torch.full((B, Hkv, Rcap), 7.0, device="cuda")
    main_idx = torch.full((B, Hkv, C), -7, dtype=torch.int32, device="cuda")
    res_len = torch.full((B * Hkv,), -7, dtype=torch.int32, device="cuda")
    main_len = torch.full((B * Hkv,), -7, dtype=torch.int32, device="cuda")
    val_loss = torch.full((B * Hkv, len(grid)), float("nan"), device="cuda")
    nws = rk.reskv_build_proxy_workspace_size(shape, params, proxy, x["seq_len"], x["budget"])
    assert nws > 0, rk.last_error()
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    rk.reskv_build_cache_proxy(shape, params, proxy, g, to_dev(x["K"], wl.dtype), to_dev(x["V"], wl.dtype),
                               x["seq_len"], to_dev(x["q_obs"], wl.dtype), x["budget"], kc, vc, logc, main_idx,
                               res_len, main_len, ws, val_loss=val_loss)
    torch.cuda.synchronize()
    return dict(kc=kc.float().cpu().numpy().astype(np.float64), vc=vc.float().cpu().numpy().astype(np.float64),
                logc=logc.cpu().numpy().astype(np.float64), main_idx=main_idx.cpu().numpy(),
                res_len=res_len.cpu().numpy().reshape(B, Hkv), main_len=main_len.cpu().numpy().reshape(B, Hkv),
                val_loss=val_loss.cpu().numpy().reshape(B, Hkv, len(grid)))


def margin_rule_f32(losses, counts, delta):
    """The margin rule replayed in float32 on the GPU's fp32 losses."""
    L = np.asarray(losses, np.float32)
    i0 = counts.index(0)
    best = None
    for i, r in enumerate(counts):
        if r <= 0:
            continue
        if best is None or L[i] < L[best] or (L[i] == L[best] and r < counts[best]):
            best = i
    if best is not None and L[best] < np.float32(np.float32(1.0) - np.float32(delta)) * L[i0]:
        return best
    return i0


def cache_loss(targets, vq, kc, vc, logc, r, n, gate):
    """fp64 oracle loss of a given cache against the full-attention outputs
    `targets` of the queries `vq`; also the largest |output| seen."""
    errs, omax = [], 0.0
    for q, t in zip(vq, targets):
        o, _ = orc.decode_head(q, kc[r:r + n], vc[r:r + n], kc[:r], vc[:r], logc[:r], gate["tau_scalar"],
                               gate["alpha"], gate["g_min"], gate["beta"])
        errs.append(float(((o - t) ** 2).sum()))
        omax = max(omax, float(np.abs(o).max()), float(np.abs(t).max()))
    return float(np.mean(errs)), omax


def check_proxy(wl, x, grid, val, delta, gate=GATE, full_heads=None):
    """Every head: the decision rule, bit equality with the chosen
    candidate and the loss of every candidate; the heads in `full_heads`
    (all when None) also get the construction checks of every candidate
    and the end-to-end comparison with the oracle's proxy."""
    got = run_proxy(wl, x, grid, val, delta, gate)
    fit = wl.window - val
    G, d = wl.group, wl.d
    rep = dict(decision_ties=0, cache_ties=0, chose_res=0, heads=0, loss_dev=0.0)
    cand = []
    for f in grid:  # each candidate rebuilt alone for the whole batch
        counts_b = [orc.candidate_counts(int(x["budget"][b]), [f])[0] for b in range(wl.batch)]
        res = np.repeat(np.asarray(counts_b, np.int32)[:, None], wl.hkv, axis=1)
        cand.append((res, run_build(wl, x, fit=fit, res=res, host_cache=wl.max_ctx <= 4096)))
    for b in range(wl.batch):
        s = int(x["seq_len"][b])
        budget = int(x["budget"][b])
        counts = orc.candidate_counts(budget, grid)
        for h in range(wl.hkv):

            rep["heads"] += 1
            full = full_heads is None or (b, h) in full_heads
            K = np.asarray(x["K_host"][b, h, :s], np.float64)
            V = np.asarray(x["V_host"][b, h, :s], np.float64)
            Qw = np.asarray(x["q_host"][b, h * G:(h + 1) * G], np.float64)
            vq = Qw[:, fit:].reshape(-1, d)
            targets = [orc.full_attention(q, K, V) for q in vq]
            Lg = got["val_loss"][b, h]
            # the GPU decision follows its own losses
            pick = margin_rule_f32(Lg, counts, delta)
            r = counts[pick]
            assert got["res_len"][b, h] == r
            rep["chose_res"] += r > 0
            # outputs are the chosen candidate's cache, bit for bit
            res_c, cb = cand[pick]
            ml = int(cb["main_len"][b, h])
            assert got["main_len"][b, h] == ml
            np.testing.assert_array_equal(got["kc"][b, h, :r + ml], cb["kc"][b, h, :r + ml])
            np.testing.assert_array_equal(got["vc"][b, h, :r + ml], cb["vc"][b, h, :r + ml])
            np.testing.assert_array_equal(got["logc"][b, h], cb["logc"][b, h])
            np.testing.assert_array_equal(got["main_idx"][b, h, :ml], cb["main_idx"][b, h, :ml])
            # every candidate: construction parity and its loss
            Lref, E = [], []
            for i, (res_c, cb) in enumerate(cand):
                rc = int(res_c[b, h])
                assert rc == counts[i]
                if full:
                    cr = check_head(wl, x, cb, b, h, fit=fit, r=rc)
                    rep["cache_ties"] += cr["near_ties"]
                n = int(cb["main_len"][b, h])
                lr, omax = cache_loss(targets, vq, cb["kc"][b, h], cb["vc"][b, h], cb["logc"][b, h], rc, n, gate)
                e = 2.0 * math.sqrt(d) * E_DEC[wl.dtype] * omax + 1e-6 * math.sqrt(lr) + 1e-12
                dev = abs(math.sqrt(max(Lg[i], 0.0)) - math.sqrt(lr))
                rep["loss_dev"] = max(rep["loss_dev"], dev / e)
                assert dev <= e, f"b{b} h{h} cand {i}: loss {Lg[i]:.6e} vs {lr:.6e}"
                Lref.append(lr)
                E.append(e)
            # end to end against the oracle's own proxy
            if not full:
                continue
            res_o = orc.validation_proxy(K, V, Qw, budget, list(grid), wl.window, wl.lloyd_iters, val, delta,
                                         gate["tau_scalar"], gate["alpha"], gate["g_min"], gate["beta"], wl.dtype)
            if res_o["r"] != r:
                Lo = res_o["losses"]
                same_caches = all(abs(math.sqrt(a) - math.sqrt(c)) <= e for a, c, e in zip(Lo, Lref, E))
                if same_caches:
                    # a decision inside the loss bound: the best r > 0 against the margin,
                    # or two counts > 0 within the bound of each other
                    pos = [i for i, c in enumerate(counts) if c > 0]
                    i0 = counts.index(0)
                    thr = math.sqrt((1.0 - delta) * Lo[i0])
                    emax = max(E)
                    near = any(abs(math.sqrt(Lo[i]) - thr) <= 2 * emax for i in pos)
                    near |= any(abs(math.sqrt(Lo[i]) - math.sqrt(Lo[j])) <= 2 * emax
                                for i in pos for j in pos if i != j)
                    assert near, f"b{b} h{h}: proxy chose r={r}, oracle r={res_o['r']}"
                    rep["decision_ties"] += 1
                else:
                    assert rep["cache_ties"] > 0, f"b{b} h{h}: candidate caches differ without a near-tie"
    return rep, got


def diffuse_queries(x, wl, heads, scale, seed):
    """Replace the window queries of the given (b, kv head) groups by
    scale * N(0, 1): attention spread over many tokens, where the evicted
    mass matters (the recipe's heavy-key queries attend to few tokens)."""
    rng = np.random.default_rng(seed)
    G = wl.group
    for b, h in heads:
        q = scale * rng.normal(size=(G,) + x["q_obs"].shape[2:])
        if wl.dtype == "bf16":
            q = torch.as_tensor(q, dtype=torch.float32).to(torch.bfloat16).float().numpy()
        x["q_obs"][b, h * G:(h + 1) * G] = q
    return host_copies(x)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_proxy_paper_split(dtype, d):
    """G = 4, w = 32, 8 validation rows per head: 96 fit / 32 validation
    queries (two decode chunks of 16), grid {0, .05, .10, .15, .20}, delta
    0.01; two sequences with different lengths; kv head 0 of each sequence
    with diffuse queries (residual entries pay), kv head 1 with the
    heavy-key queries (the main cache holds nearly all the mass)."""
    wl = synth.tiny_workload(s=1500, d=d, hq=8, hkv=2, budget=160, res=0, window=32, dtype=dtype, batch=2,
                             n_heavy=6)
    wl.ctx = [1500, 900]
    wl.budget = [160, 120]
    wl.res = np.full((1, 2, 2), 32)  # capacity for the largest candidate (0.2 * 160)
    x = synth.gen_layer(wl, 0, seed=11, n_decode=1)
    x = diffuse_queries(x, wl, [(0, 0), (1, 0)], 0.1, 11)
    rep, got = check_proxy(wl, x, GRID, 8, 0.01)
    print(rep)
    assert (got["res_len"][:, 0] > 0).all(), rep  # diffuse heads take residual entries


def test_proxy_ragged_gqa7_and_all_main():
    """G = 7 with 3 validation rows (21 queries: chunks of 11 with one padded
    query); one sequence shorter than every candidate's main budget (all
    candidates keep every token); a recent window longer than some m."""
    wl = synth.tiny_workload(s=800, d=128, hq=14, hkv=2, budget=96, res=0, window=12, dtype="bf16", batch=3,
                             n_heavy=4)
    wl.ctx = [800, 60, 431]
    wl.budget = [96, 96, 80]
    wl.res = np.full((1, 3, 2), 20)
    x = host_copies(synth.gen_layer(wl, 0, seed=12, n_decode=1))
    rep, got = check_proxy(wl, x, GRID, 3, 0.01)
    print(rep)
    assert rep["heads"] == 6


def test_proxy_diffuse_heads_take_residuals():
    """Near-identical keys give diffuse attention that the main cache cannot
    carry: some r > 0 must win on the GPU as in the oracle."""
    wl = synth.tiny_workload(s=600, d=64, hq=4, hkv=2, budget=64, res=0, window=16, dtype="f32", batch=1)
    wl.res = np.full((1, 1, 2), 13)
    x = synth.gen_layer(wl, 0, seed=13, n_decode=1)
    rng = np.random.default_rng(13)
    for h in range(2):
        base = rng.normal(size=64)
        x["K"][0, h, :600] = (0.05 * rng.normal(size=(600, 64)) + base).astype(np.float32)
    x["q_obs"][:] = (0.3 * rng.normal(size=x["q_obs"].shape)).astype(np.float32)
    host_copies(x)
    rep, got = check_proxy(wl, x, GRID, 4, 0.01)
    print(rep)
    assert rep["chose_res"] == 2, rep


def test_proxy_delta_one_never_enables():
    wl = synth.tiny_workload(s=500, d=64, hq=4, hkv=2, budget=64, res=0, window=16, dtype="f32", batch=1)
    wl.res = np.full((1, 1, 2), 13)
    x = host_copies(synth.gen_layer(wl, 0, seed=14, n_decode=1))
    got = run_proxy(wl, x, GRID, 4, 1.0)
    assert (got["res_len"] == 0).all()
    assert np.isfinite(got["val_loss"]).all()


def test_proxy_llama8b_layer():
    """The Llama-3.1-8B-shaped layer at full size (32 q / 8 KV heads, d 128,
    bf16, context 32768, budget 512, window 32) with the proxy settings of
    App. B.3: 96 fit / 32 validation queries, grid {0, .05, .10, .15, .20},
    i.e. counts {0, 26, 51, 77, 102}, delta 0.01. KV heads 0-3 get diffuse
    window queries. Every head: decision rule, bit equality, the loss of
    every candidate; heads 0 and 5: construction parity of every candidate
    and the oracle's own proxy."""
    from tests.build_check import HostView
    wl = synth.workload(1)
    wl.res = np.full((1, 1, wl.hkv), 102)  # residual capacity of the largest candidate
    x = synth.gen_layer_device(wl, 0, torch.device("cuda"), n_decode=1)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    G, w, d = wl.group, wl.window, wl.d
    x["q_obs"][0, :4 * G] = (0.1 * torch.randn((4 * G, w, d), generator=gen, device="cuda")).to(torch.bfloat16)
    x["K_host"], x["V_host"], x["q_host"] = HostView(x["K"]), HostView(x["V"]), HostView(x["q_obs"])
    rep, got = check_proxy(wl, x, GRID, 8, 0.01, full_heads=[(0, 0), (0, 5)])
    print(rep)
    assert (got["res_len"][0, :4] > 0).all(), got["res_len"]
