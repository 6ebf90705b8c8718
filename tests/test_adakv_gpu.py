"""GPU parity of reskv_build_cache_adakv against the fp64 oracle: AdaKV's
cross-head budget allocation (App. B.2.2 compared methods: the kept budget
is allocated across KV heads from SnapKV scores, safeguard 0.2; reading R26)
followed by the residual construction (Sec. 5.3) and decode (Sec. 5.4).

Per sequence:
  * exact allocation on the GPU's own fp32 scores: the oracle's
    adakv_allocate run on them reproduces every head's top-k count;
  * end-to-end allocation against the oracle's fp64 scores, except at a
    certified near-tie of the cross-head ranking (the last slot handed out
    and the first one passed over lie within the score tolerance);
  * per head, every construction check of reskv_build_cache with the
    allocated count (score parity, exact selection, Lloyd replay, entries);
  * safeguard 1 reproduces reskv_build_cache bit for bit.
"""

import math

import numpy as np
import pytest

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import synth
from tests.build_check import SCORE_ATOL, SCORE_RTOL, check_head, run_build
from tests.helpers import TOL, decode_on_gpu, rel_err_rows

pytestmark = pytest.mark.gpu


def host_copies(x):
    x["K_host"], x["V_host"], x["q_host"] = x["K"], x["V"], x["q_obs"]
    return x


def heads_of(wl, x, b, C, recent):
    """Uniform sizes of the live heads of sequence b (those with s > m)."""
    s = int(x["seq_len"][b])
    live, k_top, cap, prot = [], [], [], []
    for h in range(wl.hkv):
        r = int(x["res"][b][h])
        m = int(x["budget"][b]) - r
        if s <= m:
            continue
        P = min(recent, m, s)
        live.append(h)
        k_top.append(m - P)
        cap.append(min(s - P, C - r - P))
        prot.append(P)
    return s, live, k_top, cap, prot


def ranking_gap(scores, k_top, alpha, cap):
    """Walk the oracle's cross-head ranking and return the score of the last
    slot handed out and of the first token passed over after it (its head
    still under its cap); None where the walk ends without a contest."""
    floors = [math.floor(alpha * k) for k in k_top]
    rank = []
    for h, sc in enumerate(scores):
        order = np.lexsort((np.arange(sc.size), -sc))
        rank += [(-sc[p], h) for p in order[floors[h]:]]
    rank.sort()
    held, left, last = list(floors), sum(k_top) - sum(floors), None
    for neg, h in rank:
        if held[h] >= cap[h]:
            continue
        if left == 0:
            return last, -neg
        held[h] += 1
        left -= 1
        last = -neg
    return None


def check_sequence(wl, x, got, b, alpha, C, recent, full=True, replay_heads=None):
    """Allocation checks for sequence b plus the per-head construction
    checks. Returns the number of certified near-ties."""
    s, live, k_top, cap, prot = heads_of(wl, x, b, C, recent)
    kk_gpu = [int(got["main_len"][b, h]) - P for h, P in zip(live, prot)]
    ties = 0
    if live:
        gs = [got["scores"][b, h, :s - P] for h, P in zip(live, prot)]
        # exact: the oracle's allocation from the GPU's own scores
        assert orc.adakv_allocate(gs, k_top, alpha, cap) == kk_gpu
        assert sum(kk_gpu) == min(sum(k_top), sum(cap))
        if full:
            G = wl.group
            ref = [orc.pool(orc.window_raw_scores(np.asarray(x["K_host"][b, h, :s], np.float64),
                                                  np.asarray(x["q_host"][b, h * G:(h + 1) * G], np.float64)
                                                  )[:s - P], 5) for h, P in zip(live, prot)]
            kk_ref = orc.adakv_allocate(ref, k_top, alpha, cap)
            if kk_ref != kk_gpu:
                gap = ranking_gap(ref, k_top, alpha, cap)
                assert gap is not None and abs(gap[0] - gap[1]) <= 2 * (SCORE_RTOL * gap[0] + SCORE_ATOL), \
                    f"allocation {kk_gpu} != oracle {kk_ref} outside a near-tie"
                ties += 1
    kk = dict(zip(live, kk_gpu))
    for h in range(wl.hkv):
        rep = check_head(wl, x, got, b, h, recent=recent, k_top=kk.get(h), full_oracle=full,
                         replay=replay_heads is None or h in replay_heads)
        ties += rep["near_ties"]
    return ties


def workload(seed, dtype, d, ctx, budget, res, hq, hkv, window=8, n_heavy=4):
    wl = synth.tiny_workload(s=max(ctx), d=d, hq=hq, hkv=hkv, budget=max(budget), res=0, window=window,
                             dtype=dtype, batch=len(ctx), n_heavy=n_heavy)
    wl.ctx = list(ctx)
    wl.budget = list(budget)
    wl.n_heavy = [n_heavy] * len(ctx)
    wl.res = np.asarray(res, np.int64).reshape(1, len(ctx), hkv)
    return wl, host_copies(synth.gen_layer(wl, 0, seed=seed, n_decode=1))


@pytest.mark.parametrize("alpha", [0.0, 0.2, 0.5])
@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128)])
def test_adakv_small(alpha, dtype, d):
    """Two ragged sequences, 4 KV heads (G = 4), residual counts 0..40,
    slot capacity twice the budget so heads can grow."""
    wl, x = workload(11, dtype, d, [700, 451], [96, 64], [[40, 0, 16, 8], [0, 24, 5, 63]], 16, 4)
    C = 192
    got = run_build(wl, x, adakv=alpha, slot_cap=C)
    for b in range(2):
        assert check_sequence(wl, x, got, b, alpha, C, wl.window) <= 1


def test_adakv_moves_budget_between_heads():
    """With safeguard 0.2 the allocation is not the uniform split on these
    inputs (heads differ in how peaked their window attention is), the total
    is conserved and every head keeps its floor."""
    wl, x = workload(12, "bf16", 128, [900], [128], [[16, 0, 32, 8]], 16, 4, n_heavy=6)
    C = 256
    got = run_build(wl, x, adakv=0.2, slot_cap=C)
    check_sequence(wl, x, got, 0, 0.2, C, wl.window)
    s, live, k_top, cap, prot = heads_of(wl, x, 0, C, wl.window)
    kk = [int(got["main_len"][0, h]) - P for h, P in zip(live, prot)]
    assert kk != k_top
    assert sum(kk) == sum(k_top)
    assert all(k >= math.floor(0.2 * t) for k, t in zip(kk, k_top))


def test_adakv_safeguard_one_is_the_uniform_split():
    wl, x = workload(13, "bf16", 128, [600, 333], [80, 48], [[16, 0, 8, 40], [47, 1, 0, 3]], 16, 4)
    a = run_build(wl, x, adakv=1.0, slot_cap=160)
    u = run_build(wl, x, slot_cap=160)
    for k in ("kc", "vc", "logc", "main_idx", "res_len", "main_len", "scores", "assign"):
        np.testing.assert_array_equal(a[k], u[k])


def test_adakv_edge_cases():
    """G = 7; a sequence shorter than some heads' main budgets (those heads
    keep every token and take no part); r larger than the evicted set; a
    slot capacity equal to the budget (every head at its cap: the uniform
    split); a protected window longer than some heads' main budgets."""
    wl, x = workload(14, "bf16", 128, [600, 50, 333], [64, 64, 48], [[16, 0], [8, 30], [47, 1]], 14, 2)
    for C, recent in ((128, 8), (64, 8), (128, 70)):
        got = run_build(wl, x, adakv=0.2, slot_cap=C, recent=recent)
        for b in range(3):
            check_sequence(wl, x, got, b, 0.2, C, recent)
        if C == 64:  # sequences 0 and 1 have budget 64 = C: every head is at its cap
            u = run_build(wl, x, slot_cap=C, recent=recent)
            np.testing.assert_array_equal(got["main_idx"][:2], u["main_idx"][:2])


def test_adakv_cross_head_ties_go_to_lower_heads():
    """Identical keys and queries in every head tie every score across heads:
    the tied slots go to the lower heads first, each up to its cap, with the
    lowest positions inside a head."""
    wl, x = workload(15, "bf16", 64, [200], [40], [[4, 4, 4]], 6, 3)
    x["K"][:] = 1.0
    x["q_obs"][:] = 0.5
    host_copies(x)
    C = 60
    got = run_build(wl, x, adakv=0.0, slot_cap=C)
    check_sequence(wl, x, got, 0, 0.0, C, wl.window)
    s, live, k_top, cap, prot = heads_of(wl, x, 0, C, wl.window)
    kk = [int(got["main_len"][0, h]) - P for h, P in zip(live, prot)]
    # pooling lowers the two ends of the scored range; the interior ties
    assert kk[0] == cap[0] and kk[0] > k_top[0] and kk[2] < k_top[2]


def test_adakv_decode_over_built_cache():
    """Decode over the AdaKV-built cache (main lengths differ per head)."""
    wl, x = workload(16, "bf16", 128, [800, 500], [96, 64], [[24, 0, 8, 40], [5, 16, 0, 31]], 16, 4)
    got = run_build(wl, x, adakv=0.2, slot_cap=192)
    from paper_2607_29591_amd import reskv as rk
    shape = rk.make_shape(wl.batch, wl.hq, wl.hkv, wl.d, wl.dtype, 192, wl.res_cap)
    q = x["q_dec"][0].astype(np.float64)
    out = decode_on_gpu(shape, dict(tau_scalar=0.25, alpha=12.0, g_min=0.0, beta=1.0), q, got["kc"], got["vc"],
                        got["logc"], got["res_len"], got["main_len"], dbg=False)["out"]
    ref, *_ = orc.decode(q, got["kc"], got["vc"], got["logc"], got["res_len"], got["main_len"], 0.25, 12.0, 0.0, 1.0)
    assert rel_err_rows(out, ref).max() <= TOL["bf16"]


def test_adakv_llama_layer():
    """The Llama-3.1-8B-shaped layer (8 KV heads, 32K context, budget 512,
    r per head from {0,16,32,64,128}) with safeguard 0.2 and room for each
    head to double its budget: exact allocation on the GPU's scores, the
    fp64 allocation up to certified near-ties, every head's selection and
    rows; Lloyd replay on two heads."""
    wl = synth.workload(1)
    x = host_copies(synth.gen_layer(wl, 0, n_decode=1))
    C = 1024
    got = run_build(wl, x, adakv=0.2, slot_cap=C, host_cache=False)
    replay = {0, int(np.argmax(wl.res[0, 0]))}
    assert check_sequence(wl, x, got, 0, 0.2, C, wl.window, replay_heads=replay) <= 2


def test_adakv_decode_reserve_keeps_room_for_appends():
    """With a decode reserve of R slots no head grows past C - R at
    construction, so the next R decode steps append on every head (Sec. 3.1):
    main_len grows by one per step everywhere, the appended rows are the
    step's K/V bit for bit, and each step's output matches the oracle's
    decode of the cache it attended. Safeguard 0 (one top-k over the heads of
    a sequence) drives the best-scored heads to their caps."""
    import torch
    from paper_2607_29591_amd import reskv as rk
    wl, x = workload(21, "bf16", 128, [900, 600], [96, 64], [[24, 0, 8, 40], [5, 16, 0, 31]], 16, 4)
    C, R = 128, 8
    wl.steps = R + 1
    x = host_copies(synth.gen_layer(wl, 0, seed=21, n_decode=R + 1))
    got = run_build(wl, x, adakv=0.0, slot_cap=C, reserve=R, keep_device=True)
    for b in range(wl.batch):
        check_sequence(wl, x, got, b, 0.0, C - R, wl.window)
    ml0 = got["main_len"].reshape(-1).astype(np.int64)
    rl = got["res_len"].reshape(-1).astype(np.int64)
    assert (rl + ml0 <= C - R).all() and (rl + ml0 == C - R).any(), "no head reached its cap"
    dev = got["dev"]
    shape = rk.make_shape(wl.batch, wl.hq, wl.hkv, wl.d, wl.dtype, C, wl.res_cap)
    ws = torch.empty(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
    out = torch.empty((wl.batch, wl.hq, wl.d), device="cuda")
    gate = rk.make_gate()
    for t in range(R + 1):
        q = torch.as_tensor(x["q_dec"][t]).to(torch.bfloat16).cuda().contiguous()
        kn = torch.as_tensor(x["k_new"][t]).to(torch.bfloat16).cuda().contiguous()
        vn = torch.as_tensor(x["v_new"][t]).to(torch.bfloat16).cuda().contiguous()
        before = dev["main_len"].cpu().numpy().astype(np.int64)
        rk.reskv_decode_attn(shape, gate, q, dev["kc"], dev["vc"], dev["logc"], dev["res_len"], dev["main_len"],
                             out, ws, k_new=kn, v_new=vn)
        torch.cuda.synchronize()
        after = dev["main_len"].cpu().numpy().astype(np.int64)
        room = rl + before < C
        if t < R:
            assert room.all()
        np.testing.assert_array_equal(after, before + room)
        kc = dev["kc"].float().cpu().numpy().astype(np.float64)
        vc = dev["vc"].float().cpu().numpy().astype(np.float64)
        for bh in np.nonzero(room)[0]:
            b, h = divmod(int(bh), wl.hkv)
            slot = int(rl[bh] + before[bh])
            np.testing.assert_array_equal(kc[b, h, slot], x["k_new"][t, b, h])
            np.testing.assert_array_equal(vc[b, h, slot], x["v_new"][t, b, h])
        ref, *_ = orc.decode(x["q_dec"][t].astype(np.float64), kc, vc, got["logc"], rl.reshape(wl.batch, wl.hkv),
                             after.reshape(wl.batch, wl.hkv), 0.25, 12.0, 0.0, 1.0)
        assert rel_err_rows(out.double().cpu().numpy(), ref).max() <= TOL["bf16"], f"step {t}"
