"""Full-size parity on one GPU, at the sizes of the workloads:

  * Llama-3.1-8B layer (32 q / 8 KV heads, d 128, 32K context, budget 512,
    r per head from {0, 16, 32, 64, 128}): every head built on the GPU and
    checked in full (scores, exact selection, Lloyd replay with the exported
    centres, entries), then all 128 decode queries decoded over the
    GPU-built cache (split-K path) and every (query head, step) compared
    with the oracle, gate and log-sum-exps included;
  * batched decode layer (32 sequences x 8 KV heads, 32K context -> 2048
    slots, r per head from {0, 64, 128, 256, 512}): Lloyd replay on five
    heads including the largest and smallest r, selection on six more, then
    all 256 decode steps with the step's token appended inside the call,
    checked against the oracle at early, middle and last steps (the last
    one fills the 2304-slot capacity);
  * long-context construction layer (4 x 8 KV heads, 128K context, budget
    1024 = 768 + 256, window 64): Lloyd replay on four heads, all 64 decode
    steps with appends, checked at the first, a middle and the last step;
  * ragged GQA-7 layer (64 sequences x 4 KV heads, contexts 4K-64K,
    budgets 256-1024, r fraction in [0, 0.5]): Lloyd replay on four heads
    (shortest and longest context, largest r), all 128 decode steps with
    appends, checked at the first, a middle and the last step.
At every decode step with appends, every head's main_len grows by exactly
one (the caches have room for every step) and the appended slot holds the
step's key and value bit for bit.
"""

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import reskv as rk
from paper_2607_29591_amd import synth
from tests.build_check import HostView, check_head, run_build
from tests.helpers import TOL, gate_atol, rel_err_rows

pytestmark = pytest.mark.gpu


def device_layer(wl, n_decode):
    x = synth.gen_layer_device(wl, 0, torch.device("cuda"), n_decode=n_decode)
    x["K_host"], x["V_host"], x["q_host"] = HostView(x["K"]), HostView(x["V"]), HostView(x["q_obs"])
    return x


def decode_steps(wl, x, got, steps, check_at, samples):
    """Run `steps` decode calls with fused appends on the GPU-built cache.
    Every step: main_len grows by one on every head with room and the
    appended slot holds the step's K/V; at the steps in `check_at` the
    sampled (b, query head) outputs are checked against the oracle run on
    the cache the call attended. Returns the worst relative error."""
    dev = got["dev"]
    B, Hkv, d, C = wl.batch, wl.hkv, wl.d, wl.slot_cap
    BH = B * Hkv
    shape = rk.make_shape(B, wl.hq, Hkv, d, wl.dtype, C, wl.res_cap)
    ws = torch.empty(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
    out = torch.empty((B, wl.hq, d), device="cuda")
    res = got["res_len"]
    rl = dev["res_len"].long()
    rows = torch.arange(BH, device="cuda")
    worst = 0.0
    for t in range(steps):
        tau = x["tau"][t].contiguous()
        gate = rk.make_gate(tau=tau, alpha=wl.alpha, g_min=wl.g_min, beta=wl.beta)
        kn, vn = x["k_new"][t].contiguous(), x["v_new"][t].contiguous()
        before = dev["main_len"].long().clone()
        rk.reskv_decode_attn(shape, gate, x["q_dec"][t].contiguous(), dev["kc"], dev["vc"], dev["logc"],
                             dev["res_len"], dev["main_len"], out, ws, k_new=kn, v_new=vn)
        after = dev["main_len"].long()
        assert bool((rl + before < C).all()), f"step {t}: a cache is full before its last step"
        assert torch.equal(after, before + 1), f"step {t}: main_len did not grow by one on every head"
        slot = rl + before
        assert torch.equal(dev["kc"].view(BH, C, d)[rows, slot], kn.view(BH, d)), f"step {t}: appended keys"
        assert torch.equal(dev["vc"].view(BH, C, d)[rows, slot], vn.view(BH, d)), f"step {t}: appended values"
        if t not in check_at:
            continue
        torch.cuda.synchronize()
        main_len = after.cpu().numpy().reshape(B, Hkv)
        o = out.double().cpu().numpy()
        q = x["q_dec"][t].float().cpu().numpy().astype(np.float64)
        tau_h = tau.cpu().numpy().astype(np.float64)
        for b, h in samples:
            kv = h // wl.group
            r, n = int(res[b, kv]), int(main_len[b, kv])
            kc = dev["kc"][b, kv, :r + n].float().cpu().numpy().astype(np.float64)
            vc = dev["vc"][b, kv, :r + n].float().cpu().numpy().astype(np.float64)
            ref, _ = orc.decode_head(q[b, h], kc[r:], vc[r:], kc[:r], vc[:r], got["logc"][b, kv, :r],
                                     tau_h[b, h], wl.alpha, wl.g_min, wl.beta)
            err = rel_err_rows(o[b, h][None], ref[None]).max()
            worst = max(worst, err)
            assert err <= TOL[wl.dtype], f"step {t} (b={b}, h={h}): rel err {err:.2e}"
    return worst


def test_llama_layer_end_to_end():
    """Every head of the Llama-3.1-8B layer built and checked against the
    oracle, then all 128 decode queries over that cache on every query head."""
    wl = synth.workload(1)
    x = synth.gen_layer(wl, 0)
    x["K_host"], x["V_host"], x["q_host"] = x["K"], x["V"], x["q_obs"]
    got = run_build(wl, x, keep_device=True)
    ties = 0
    for h in range(wl.hkv):
        rep = check_head(wl, x, got, 0, h, lloyd_info=False)
        ties += rep["near_ties"]
    assert ties <= 1
    dev = got["dev"]
    shape = rk.make_shape(wl.batch, wl.hq, wl.hkv, wl.d, wl.dtype, wl.slot_cap, wl.res_cap)
    ws = torch.empty(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
    B, Hq, d = wl.batch, wl.hq, wl.d
    steps = wl.steps
    outs = torch.empty((steps, B, Hq, d), device="cuda")
    dbg = torch.empty((3, steps, B * Hq), device="cuda")
    q_dev = torch.as_tensor(x["q_dec"]).to(torch.bfloat16).cuda().contiguous()
    gate = rk.make_gate(tau_scalar=0.25, alpha=wl.alpha, g_min=wl.g_min, beta=wl.beta)
    for t in range(steps):
        rk.reskv_decode_attn(shape, gate, q_dev[t], dev["kc"], dev["vc"], dev["logc"], dev["res_len"],
                             dev["main_len"], outs[t], ws, dbg[0, t], dbg[1, t], dbg[2, t])
    torch.cuda.synchronize()
    # the cache is static (no appends): the lengths are those of the build
    np.testing.assert_array_equal(dev["main_len"].cpu().numpy().reshape(B, wl.hkv), got["main_len"])
    o = outs.double().cpu().numpy()
    dg = dbg.double().cpu().numpy().reshape(3, steps, B, Hq)
    worst = 0.0
    for t in range(steps):
        ref, lm, lr, g = orc.decode(x["q_dec"][t].astype(np.float64), got["kc"], got["vc"], got["logc"],
                                    got["res_len"], got["main_len"], 0.25, wl.alpha, wl.g_min, wl.beta)
        err = rel_err_rows(o[t], ref).max()
        worst = max(worst, err)
        assert err <= TOL["bf16"], f"step {t}: rel err {err:.2e}"
        qt = x["q_dec"][t].astype(np.float64)
        for h in range(Hq):
            kv = h // wl.group
            r, n = int(got["res_len"][0, kv]), int(got["main_len"][0, kv])
            tol = max(1e-5 * g[0, h], gate_atol(qt[0, h], got["kc"][0, kv, r:r + n], g[0, h], lm[0, h], wl.alpha))
            assert abs(dg[2, t, 0, h] - g[0, h]) <= tol, f"step {t} head {h}: gate {dg[2, t, 0, h]} vs {g[0, h]}"
        np.testing.assert_allclose(dg[0, t], lm, rtol=1e-5, atol=1e-5)
        fin = np.isfinite(lr)
        assert (np.isfinite(dg[1, t]) == fin).all()
        np.testing.assert_allclose(dg[1, t][fin], lr[fin], rtol=1e-5, atol=1e-5)
    print(f"llama layer: 8 heads, {ties} near-ties, 128 x 32 decode rows, worst rel err {worst:.2e}")


@pytest.fixture(scope="module")
def batched_layer():
    wl = synth.workload(2)
    wl.res = wl.res[:1]
    x = device_layer(wl, n_decode=wl.steps)
    got = run_build(wl, x, keep_device=True, host_cache=False)
    return wl, x, got


def test_batched_decode_layer_construction(batched_layer):
    wl, x, got = batched_layer
    r_row = wl.res[0, 0]
    order = np.argsort(r_row, kind="stable")
    nz = [int(h) for h in order if r_row[h] > 0]
    replay = [(0, nz[-1]), (31, nz[0]), (7, nz[len(nz) // 2]), (19, nz[-1]), (12, int(order[0]))]
    for b, h in replay:
        check_head(wl, x, got, b, h, lloyd_info=False)
    rng = np.random.default_rng(0)
    for b, h in [(int(rng.integers(32)), int(rng.integers(8))) for _ in range(6)]:
        check_head(wl, x, got, b, h, full_oracle=False, replay=False)


def test_batched_decode_layer_all_steps(batched_layer):
    wl, x, got = batched_layer
    rng = np.random.default_rng(1)
    samples = [(int(rng.integers(32)), int(rng.integers(32))) for _ in range(12)]
    decode_steps(wl, x, got, wl.steps, {0, 1, 2, 127, 128, 254, 255}, samples)


@pytest.fixture(scope="module")
def long_layer():
    wl = synth.workload(3)
    wl.res = wl.res[:1]
    x = device_layer(wl, n_decode=wl.steps)
    got = run_build(wl, x, keep_device=True, host_cache=False)
    return wl, x, got


def test_long_context_construction(long_layer):
    wl, x, got = long_layer
    for b, h in [(0, 3), (1, 0), (2, 5), (3, 7)]:
        check_head(wl, x, got, b, h, lloyd_info=False)
    for b, h in [(1, 6), (3, 2)]:
        check_head(wl, x, got, b, h, full_oracle=False, replay=False)


def test_long_context_decode_all_steps(long_layer):
    wl, x, got = long_layer
    decode_steps(wl, x, got, wl.steps, {0, 31, 63}, [(0, 13), (3, 31), (2, 0), (1, 17)])


@pytest.fixture(scope="module")
def ragged_layer():
    wl = synth.workload(4)
    wl.res = wl.res[:1]
    x = device_layer(wl, n_decode=wl.steps)
    got = run_build(wl, x, keep_device=True, host_cache=False)
    return wl, x, got


def ragged_heads(wl):
    ctx = np.asarray(wl.ctx)
    r_row = wl.res[0]
    b_short, b_long = int(np.argmin(ctx)), int(np.argmax(ctx))
    b_r, h_r = (int(v) for v in np.unravel_index(int(np.argmax(r_row)), r_row.shape))
    return b_short, b_long, b_r, h_r


def test_ragged_gqa7_construction(ragged_layer):
    wl, x, got = ragged_layer
    b_short, b_long, b_r, h_r = ragged_heads(wl)
    r_row = wl.res[0]
    h_long = int(np.argmax(r_row[b_long]))
    for b, h in [(b_short, 1), (b_r, h_r), (b_long, h_long), (20, 3)]:
        check_head(wl, x, got, b, h, lloyd_info=False)
    check_head(wl, x, got, b_long, (h_long + 1) % 4, full_oracle=False, replay=False)


def test_ragged_gqa7_decode_all_steps(ragged_layer):
    wl, x, got = ragged_layer
    b_short, b_long, b_r, h_r = ragged_heads(wl)
    samples = [(b_short, 3), (b_long, 27), (b_r, 7 * h_r), (b_r, 7 * h_r + 6), (40, 12)]
    decode_steps(wl, x, got, wl.steps, {0, 64, 127}, samples)
