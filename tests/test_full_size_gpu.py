"""Full-size parity on one GPU, sampled: one layer of the batched-decode
(32 x 8 KV heads, 32K context, budget 2048), construction-heavy (4 x 8 KV
heads, 128K context, budget 1024 = 768 + 256, window 64) and ragged GQA-7
(64 x 4 KV heads, contexts 4K-64K, budgets 256-1024) workloads. Every head is
built and decoded on the GPU; sampled heads are checked against the oracle
(construction: scores, exact selection, Lloyd replay, entries; decode: the
oracle run on the GPU-built cache), with this step's token appended in the
decode call."""

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import reskv as rk
from paper_2607_29591_amd import synth
from tests.build_check import HostView, check_head, run_build
from tests.helpers import TOL, rel_err_rows

pytestmark = pytest.mark.gpu


def device_layer(wl, n_decode):
    x = synth.gen_layer_device(wl, 0, torch.device("cuda"), n_decode=n_decode)
    x["K_host"], x["V_host"], x["q_host"] = HostView(x["K"]), HostView(x["V"]), HostView(x["q_obs"])
    return x


def decode_and_check(wl, x, got, steps, samples):
    """Run `steps` decode calls with fused appends on the GPU-built cache;
    check the sampled (b, query head) outputs of every step."""
    dev = got["dev"]
    B, Hkv, d = wl.batch, wl.hkv, wl.d
    shape = rk.make_shape(B, wl.hq, Hkv, d, wl.dtype, wl.slot_cap, wl.res_cap)
    ws = torch.empty(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
    out = torch.empty((B, wl.hq, d), device="cuda")
    res = got["res_len"]
    worst = 0.0
    for t in range(steps):
        tau = x["tau"][t].contiguous()
        gate = rk.make_gate(tau=tau, alpha=wl.alpha, g_min=wl.g_min, beta=wl.beta)
        rk.reskv_decode_attn(shape, gate, x["q_dec"][t].contiguous(), dev["kc"], dev["vc"], dev["logc"],
                             dev["res_len"], dev["main_len"], out, ws, k_new=x["k_new"][t].contiguous(),
                             v_new=x["v_new"][t].contiguous())
        torch.cuda.synchronize()
        main_len = dev["main_len"].cpu().numpy().reshape(B, Hkv)
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


def test_batched_decode_layer():
    wl = synth.workload(2)
    wl.res = wl.res[:1]
    x = device_layer(wl, n_decode=3)
    got = run_build(wl, x, keep_device=True, host_cache=False)
    rng = np.random.default_rng(0)
    r_row = wl.res[0, 0]
    full = [(0, int(np.argmax(r_row))), (31, int(np.argmin(r_row)))]
    for b, h in full:
        check_head(wl, x, got, b, h, full_oracle=True, replay=True)
    for b, h in [(int(rng.integers(32)), int(rng.integers(8))) for _ in range(6)]:
        check_head(wl, x, got, b, h, full_oracle=False, replay=False)
    samples = [(int(rng.integers(32)), int(rng.integers(32))) for _ in range(12)]
    decode_and_check(wl, x, got, 3, samples)


def test_long_context_construction_layer():
    wl = synth.workload(3)
    wl.res = wl.res[:1]
    x = device_layer(wl, n_decode=2)
    got = run_build(wl, x, keep_device=True, host_cache=False)
    check_head(wl, x, got, 0, 3, full_oracle=True, replay=True)
    for b, h in [(1, 0), (2, 5), (3, 7)]:
        check_head(wl, x, got, b, h, full_oracle=False, replay=False)
    decode_and_check(wl, x, got, 2, [(0, 13), (3, 31), (2, 0)])


def test_ragged_gqa7_layer():
    wl = synth.workload(4)
    wl.res = wl.res[:1]
    x = device_layer(wl, n_decode=2)
    got = run_build(wl, x, keep_device=True, host_cache=False)
    ctx = np.asarray(wl.ctx)
    b_short, b_long = int(np.argmin(ctx)), int(np.argmax(ctx))
    r_row = wl.res[0]
    b_r, h_r = np.unravel_index(int(np.argmax(r_row)), r_row.shape)
    check_head(wl, x, got, b_short, 1, full_oracle=True, replay=True)
    check_head(wl, x, got, int(b_r), int(h_r), full_oracle=True, replay=True)
    check_head(wl, x, got, b_long, 2, full_oracle=False, replay=False)
    decode_and_check(wl, x, got, 2, [(b_short, 3), (b_long, 27), (int(b_r), 7 * int(h_r))])
