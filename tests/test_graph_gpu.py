"""The C ABI under HIP graph capture: every entry point enqueues only kernel
launches on the caller's stream (no memsets, copies, allocations or host
synchronisation), and decode reads the cache lengths on the device, so a
decode step with its fused append and a whole construction call can be
captured once and replayed. Each graph is replayed several times, with eager
work (new inputs written, host checks) between the replays, and every replay
is compared bit for bit with the same call run eagerly."""

import numpy as np
import pytest
import torch

from paper_2607_29591_amd import reskv as rk
from paper_2607_29591_amd import synth
from tests.helpers import random_cache, to_dev

pytestmark = pytest.mark.gpu


def decode_state(B, Hkv, G, d, C, Rcap, seed):
    rng = np.random.default_rng(seed)
    res = rng.choice([0, 16, 64], size=(B, Hkv))
    main = rng.integers(1, C - 80, size=(B, Hkv))
    kc, vc, logc = random_cache(rng, B, Hkv, C, Rcap, d, "bf16", res, main)
    dev = dict(kc=to_dev(kc, "bf16"), vc=to_dev(vc, "bf16"),
               logc=torch.as_tensor(logc.astype(np.float32)).cuda(),
               res_len=torch.as_tensor(res.astype(np.int32).reshape(-1)).cuda(),
               main_len=torch.as_tensor(main.astype(np.int32).reshape(-1)).cuda())
    return rng, dev


def clone(state):
    return {k: v.clone() for k, v in state.items()}


@pytest.mark.parametrize("B,Hkv,G,C", [(64, 4, 4, 320), (64, 4, 8, 1500), (2, 2, 7, 320)])
def test_decode_step_graph_replays_match_eager(B, Hkv, G, C):
    """(64, 4, 4, 320): one block per (sequence, KV head) with the append
    fused; (64, 4, 8, 1500): the same kernel on caches long enough for the
    staggered order of the main blocks past the first round; (2, 2, 7, 320):
    the split-K path (partial blocks with the append fused, then the
    combine, which advances the main lengths)."""
    d, Rcap = 128, 64
    shape = rk.make_shape(B, G * Hkv, Hkv, d, "bf16", C, Rcap)
    rng, base = decode_state(B, Hkv, G, d, C, Rcap, 5 + G)
    eager, graphed = clone(base), clone(base)
    q = torch.empty((B, G * Hkv, d), dtype=torch.bfloat16, device="cuda")
    kn = torch.empty((B, Hkv, d), dtype=torch.bfloat16, device="cuda")
    vn = torch.empty_like(kn)
    tau = torch.empty((B * G * Hkv,), device="cuda")
    gate = rk.make_gate(tau=tau)
    ws_e = torch.zeros(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
    ws_g = torch.zeros_like(ws_e)
    out_e = torch.empty((B, G * Hkv, d), device="cuda")
    out_g = torch.empty_like(out_e)

    def call(st, out, ws):
        rk.reskv_decode_attn(shape, gate, q, st["kc"], st["vc"], st["logc"], st["res_len"], st["main_len"], out, ws,
                             k_new=kn, v_new=vn)

    def new_inputs():
        q.copy_(torch.as_tensor(rng.normal(size=q.shape), dtype=torch.float32).to(torch.bfloat16))
        kn.copy_(torch.as_tensor(rng.normal(size=kn.shape), dtype=torch.float32).to(torch.bfloat16))
        vn.copy_(torch.as_tensor(rng.normal(size=vn.shape), dtype=torch.float32).to(torch.bfloat16))
        tau.copy_(torch.as_tensor(rng.normal(0.0, 0.5, size=tau.shape), dtype=torch.float32))

    new_inputs()
    call(clone(base), out_e, ws_e)  # the kernels' first launch happens outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(graphed, out_g, ws_g)
    torch.cuda.synchronize()
    for step in range(4):
        if step:
            new_inputs()
        g.replay()
        torch.cuda.synchronize()
        call(eager, out_e, ws_e)
        torch.cuda.synchronize()
        assert torch.equal(out_g, out_e), f"replay {step}: outputs differ"
        for k in ("kc", "vc", "main_len"):
            assert torch.equal(graphed[k], eager[k]), f"replay {step}: {k} differs"
    # every replay appended one token where there was room
    grew = (eager["main_len"] - base["main_len"]).cpu().numpy()
    full = (base["res_len"] + base["main_len"]).cpu().numpy() >= C
    assert ((grew == 4) | full).all()


def test_build_graph_replays_match_eager():
    """A whole construction call (scores, selection, gather, Lloyd rounds)
    captured once and replayed three times into freshly cleared outputs."""
    wl = synth.tiny_workload(s=900, d=128, hq=16, hkv=4, budget=128, res=0, window=16, dtype="bf16", batch=2,
                             n_heavy=6)
    wl.ctx = [900, 613]
    wl.res = np.array([[[24, 0, 40, 8], [64, 16, 0, 31]]])
    x = synth.gen_layer_device(wl, 0, torch.device("cuda"), n_decode=1)
    B, Hkv, d, C, Rcap, S = wl.batch, wl.hkv, wl.d, wl.slot_cap, wl.res_cap, wl.max_ctx
    shape = rk.make_shape(B, wl.hq, Hkv, d, "bf16", C, Rcap)
    params = rk.BuildParams(S, wl.window, wl.window, wl.lloyd_iters, 0, 0)
    res = x["res"].reshape(-1)
    ws = torch.zeros(rk.reskv_build_workspace_size(shape, params, x["seq_len"], x["budget"], res),
                     dtype=torch.uint8, device="cuda")

    def outputs():
        return dict(kc=torch.zeros((B, Hkv, C, d), dtype=torch.bfloat16, device="cuda"),
                    vc=torch.zeros((B, Hkv, C, d), dtype=torch.bfloat16, device="cuda"),
                    logc=torch.zeros((B, Hkv, Rcap), device="cuda"),
                    main_idx=torch.zeros((B, Hkv, C), dtype=torch.int32, device="cuda"),
                    res_len=torch.zeros((B * Hkv,), dtype=torch.int32, device="cuda"),
                    main_len=torch.zeros((B * Hkv,), dtype=torch.int32, device="cuda"))

    def call(o):
        rk.reskv_build_cache(shape, params, x["K"], x["V"], x["seq_len"], x["q_obs"], x["budget"], res, o["kc"],
                             o["vc"], o["logc"], o["main_idx"], o["res_len"], o["main_len"], ws)

    eager = outputs()
    call(eager)
    torch.cuda.synchronize()
    graphed = outputs()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(graphed)
    torch.cuda.synchronize()
    for rep in range(3):
        for t in graphed.values():
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in eager:
            assert torch.equal(graphed[k], eager[k]), f"replay {rep}: {k} differs"
