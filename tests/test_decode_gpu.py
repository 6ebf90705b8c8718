"""GPU parity of reskv_decode_attn / reskv_append_kv against the fp64 oracle
(Sec. 5.4 shared-softmax decode, Sec. 5.5.2 gate, App. D Algorithm 2).

Bar: per (batch, query head), max|gpu - oracle| / max|oracle| <= 1e-5 for
fp32 caches and <= 2e-3 for bf16 caches; the gate and both log-sum-exps to
1e-5 relative (absolute near zero).
"""

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import reskv as rk
from paper_2607_29591_amd import synth
from tests.helpers import TOL, decode_on_gpu, random_cache, rel_err_rows, to_dev

pytestmark = pytest.mark.gpu

GATE = dict(tau_scalar=0.25, alpha=12.0, g_min=0.0, beta=1.0)


def check(dtype, shape, q, kc, vc, logc, res, main, tau=None, gate=GATE, heads=None, tol=None):
    got = decode_on_gpu(shape, gate, q, kc, vc, logc, res, main, tau=tau)
    t = gate["tau_scalar"] if tau is None else tau
    ref, lm, lr, g = orc.decode(q, kc, vc, logc, np.asarray(res), np.asarray(main), t, gate["alpha"],
                                gate["g_min"], gate["beta"], heads=heads)
    tol = TOL[dtype] if tol is None else tol
    sel = (slice(None),) if heads is None else tuple(np.array(heads).T)
    err = rel_err_rows(got["out"][sel], ref[sel])
    assert np.isfinite(got["out"][sel]).all()
    assert err.max() <= tol, f"max rel err {err.max():.3e} > {tol}"
    np.testing.assert_allclose(got["gate"][sel], g[sel], rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(got["lse_main"][sel], lm[sel], rtol=1e-5, atol=1e-5)
    fin = np.isfinite(lr[sel])
    assert (np.isfinite(got["lse_res"][sel]) == fin).all()
    np.testing.assert_allclose(got["lse_res"][sel][fin], lr[sel][fin], rtol=1e-5, atol=1e-5)
    return err.max()


def cache_case(seed, B, Hq, Hkv, d, dtype, C, Rcap, res, main, **kw):
    rng = np.random.default_rng(seed)
    kc, vc, logc = random_cache(rng, B, Hkv, C, Rcap, d, dtype, res, main, **kw)
    q = rng.normal(size=(B, Hq, d)) * 1.5
    q = np.asarray(torch.as_tensor(q, dtype=torch.float32).to(torch.bfloat16).double()) if dtype == "bf16" else \
        q.astype(np.float32).astype(np.float64)
    shape = rk.make_shape(B, Hq, Hkv, d, dtype, C, Rcap)
    return shape, q, kc, vc, logc


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("G", [1, 2, 4, 7, 8, 16])
def test_decode_ragged_shapes(dtype, d, G):
    """Ragged lengths (tails inside a 16-slot tile, a 64-slot wave and a
    256-slot block), r = 0 heads, empty entries, every supported group size."""
    Hkv = 3
    B = 2
    C, Rcap = 700, 300
    res = [[0, 17, 300], [255, 1, 64]]
    main = [[1, 399, 300], [445, 257, 636]]
    shape, q, kc, vc, logc = cache_case(10 + G + d, B, G * Hkv, Hkv, d, dtype, C, Rcap, res, main)
    check(dtype, shape, q, kc, vc, logc, res, main)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decode_gate_variants(dtype):
    B, Hkv, G, d, C, Rcap = 2, 2, 4, 128, 600, 128
    res = [[128, 40], [0, 100]]
    main = [[300, 472], [600, 20]]
    shape, q, kc, vc, logc = cache_case(3, B, Hkv * G, Hkv, d, dtype, C, Rcap, res, main)
    rng = np.random.default_rng(0)
    tau = rng.normal(0, 0.5, size=(B, Hkv * G)).astype(np.float32)
    check(dtype, shape, q, kc, vc, logc, res, main, tau=tau)
    check(dtype, shape, q, kc, vc, logc, res, main, gate=dict(tau_scalar=0.25, alpha=12.0, g_min=1.0, beta=1.0))
    check(dtype, shape, q, kc, vc, logc, res, main, gate=dict(tau_scalar=0.9, alpha=3.0, g_min=0.2, beta=0.5))
    for gate in GATE_EDGES:
        check(dtype, shape, q, kc, vc, logc, res, main, gate=gate)


# Degenerate gate settings (Sec. 5.5.2; beta weights log c_j in the residual
# logits): no count weighting, a constant gate of 1/2 (alpha = 0), the gate
# pinned at 1 by g_min, a threshold far below every p_max (the sigmoid
# underflows: gate 0 in fp32, ~1e-262 in the fp64 oracle, the residual
# entries switched off either way) and far above it (gate 1).
GATE_EDGES = [dict(tau_scalar=0.25, alpha=12.0, g_min=0.0, beta=0.0),
              dict(tau_scalar=0.25, alpha=0.0, g_min=0.0, beta=1.0),
              dict(tau_scalar=0.25, alpha=0.0, g_min=1.0, beta=0.0),
              dict(tau_scalar=-50.0, alpha=12.0, g_min=0.0, beta=1.0),
              dict(tau_scalar=50.0, alpha=12.0, g_min=0.0, beta=1.0)]


def test_decode_gate_edges_one_block_per_head():
    """The gate edge settings on the one-block-per-head kernel (256 (b, kv
    head) pairs), whose epilogue evaluates the gate and shared denominator."""
    B, Hkv, G, d, C, Rcap = 64, 4, 4, 128, 300, 64
    rng = np.random.default_rng(8)
    res = rng.integers(0, Rcap + 1, size=(B, Hkv))
    main = np.array([[int(rng.integers(1, C - r + 1)) for r in row] for row in res])
    shape, q, kc, vc, logc = cache_case(9, B, Hkv * G, Hkv, d, "bf16", C, Rcap, res, main)
    for gate in GATE_EDGES:
        check("bf16", shape, q, kc, vc, logc, res, main, gate=gate)


def test_decode_all_residual_entries_empty():
    B, Hkv, G, d, C, Rcap = 1, 2, 4, 64, 200, 64
    res, main = [[64, 10]], [[100, 190]]
    shape, q, kc, vc, logc = cache_case(4, B, Hkv * G, Hkv, d, "f32", C, Rcap, res, main)
    logc[:] = -np.inf
    check("f32", shape, q, kc, vc, logc, res, main)


def test_decode_large_logits():
    """Sharp attention (scaled queries) exercises the max shifts."""
    B, Hkv, G, d, C, Rcap = 1, 2, 4, 128, 1100, 200
    res, main = [[200, 33]], [[900, 1000]]
    shape, q, kc, vc, logc = cache_case(5, B, Hkv * G, Hkv, d, "bf16", C, Rcap, res, main, key_scale=3.0)
    q = np.asarray(torch.as_tensor(q * 8, dtype=torch.float32).to(torch.bfloat16).double())
    check("bf16", shape, q, kc, vc, logc, res, main)


def test_decode_is_deterministic_and_workspace_reusable():
    """Bitwise-equal reruns; one workspace serves calls with different
    lengths."""
    B, Hkv, G, d, C, Rcap = 2, 2, 4, 128, 900, 256
    res, main = [[256, 0], [13, 200]], [[600, 900], [700, 3]]
    shape, q, kc, vc, logc = cache_case(6, B, Hkv * G, Hkv, d, "bf16", C, Rcap, res, main)
    ws = torch.zeros(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
    a = decode_on_gpu(shape, GATE, q, kc, vc, logc, res, main, ws=ws)
    b = decode_on_gpu(shape, GATE, q, kc, vc, logc, res, main, ws=ws)
    np.testing.assert_array_equal(a["out"], b["out"])
    main2 = [[100, 300], [1, 3]]
    c = decode_on_gpu(shape, GATE, q, kc, vc, logc, res, main2, ws=ws)
    ref, *_ = orc.decode(q, kc, vc, logc, np.asarray(res), np.asarray(main2), 0.25, 12.0, 0.0, 1.0)
    assert rel_err_rows(c["out"], ref).max() <= TOL["bf16"]
    d2 = decode_on_gpu(shape, GATE, q, kc, vc, logc, res, main, ws=ws)
    np.testing.assert_array_equal(a["out"], d2["out"])


def test_decode_workload0_oracle_built_cache():
    """The fp32 toy workload: cache built by the oracle, 8 decode queries."""
    wl = synth.workload(0)
    x = synth.gen_layer(wl, 0)
    cache = orc.build_cache(x["K"], x["V"], x["q_obs"], x["seq_len"], x["budget"], x["res"], wl.window,
                            wl.lloyd_iters, wl.dtype, wl.slot_cap, wl.res_cap)
    shape = rk.make_shape(wl.batch, wl.hq, wl.hkv, wl.d, wl.dtype, wl.slot_cap, wl.res_cap)
    for step in range(wl.steps):
        check("f32", shape, x["q_dec"][step], cache["kc"], cache["vc"], cache["logc"], cache["res_len"],
              cache["main_len"])


def test_decode_batched_llama_shape_sampled():
    """32 sequences x 8 KV heads x 2048-slot budget + appended room (the
    batched decode workload's per-layer shape); every head decoded on the
    GPU, a sample checked against the oracle."""
    wl = synth.workload(2)
    B, Hkv, G, d = wl.batch, wl.hkv, wl.group, wl.d
    C, Rcap = wl.slot_cap, wl.res_cap
    rng = np.random.default_rng(7)
    res = wl.res[0]
    main = 2048 - res + rng.integers(0, 257, size=res.shape)
    shape, q, kc, vc, logc = cache_case(8, B, Hkv * G, Hkv, d, "bf16", C, Rcap, res, main, empty_frac=0.0)
    tau = (rng.normal(0, 0.5, size=(B, Hkv * G))).astype(np.float32)
    heads = [(int(b), int(h)) for b, h in zip(rng.integers(0, B, 24), rng.integers(0, Hkv * G, 24))]
    check("bf16", shape, q, kc, vc, logc, res, main, tau=tau, heads=heads)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_append_then_decode(dtype):
    B, Hkv, G, d, C, Rcap = 2, 2, 4, 64, 140, 32
    res = np.array([[32, 0], [5, 31]])
    main = np.array([[100, 137], [1, 40]])
    shape, q, kc, vc, logc = cache_case(9, B, Hkv * G, Hkv, d, dtype, C, Rcap, res, main)
    rng = np.random.default_rng(1)
    kcd, vcd = to_dev(kc, dtype), to_dev(vc, dtype)
    rl = torch.as_tensor(res.astype(np.int32).reshape(-1)).cuda()
    ml = torch.as_tensor(main.astype(np.int32).reshape(-1)).cuda()
    kc2, vc2, main2 = kc.copy(), vc.copy(), main.copy()
    for step in range(5):
        kn = rng.normal(size=(B, Hkv, d))
        vn = rng.normal(size=(B, Hkv, d))
        knd, vnd = to_dev(kn, dtype), to_dev(vn, dtype)
        rk.reskv_append_kv(shape, knd, vnd, kcd, vcd, rl, ml)
        for b in range(B):
            for h in range(Hkv):
                slot = res[b, h] + main2[b, h]
                if slot < C:
                    kc2[b, h, slot] = knd[b, h].double().cpu().numpy()
                    vc2[b, h, slot] = vnd[b, h].double().cpu().numpy()
                    main2[b, h] += 1
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ml.cpu().numpy().reshape(B, Hkv), main2)
    np.testing.assert_array_equal(kcd.double().cpu().numpy(), kc2)
    check(dtype, shape, q, kc2, vc2, logc, res, main2)


@pytest.mark.parametrize("dtype,d,G,B,Hkv", [("bf16", 128, 4, 32, 8), ("f32", 64, 2, 64, 4), ("bf16", 64, 1, 16, 16),
                                             ("bf16", 128, 4, 2, 2), ("f32", 128, 7, 2, 2), ("bf16", 128, 7, 64, 4),
                                             ("bf16", 64, 16, 32, 8)])
def test_decode_fused_append(dtype, d, G, B, Hkv):
    """reskv_decode_attn with this step's K/V: the token is appended as main
    slot r + n (cache and main_len written) and attended in the same call.
    B*Hkv >= 256 (bf16, or fp32 rows of 64) takes the one-block-per-head
    kernel, for any group size up to 16; the others the split-K kernels;
    full caches are left unchanged."""
    rng = np.random.default_rng(11 + d + G)
    C, Rcap = 300, 64
    res = rng.choice([0, 16, 64], size=(B, Hkv))
    main = rng.integers(1, C - 64, size=(B, Hkv))
    main[0, 0] = C - res[0, 0]  # full: no append
    shape, q, kc, vc, logc = cache_case(20 + d, B, G * Hkv, Hkv, d, dtype, C, Rcap, res, main)
    kn = rng.normal(size=(B, Hkv, d))
    vn = rng.normal(size=(B, Hkv, d))
    knd, vnd = to_dev(kn, dtype), to_dev(vn, dtype)
    kcd, vcd = to_dev(kc, dtype), to_dev(vc, dtype)
    lcd = torch.as_tensor(logc.astype(np.float32)).cuda()
    rl = torch.as_tensor(res.astype(np.int32).reshape(-1)).cuda()
    ml = torch.as_tensor(main.astype(np.int32).reshape(-1)).cuda()
    qd = to_dev(q, dtype)
    out = torch.empty((B, G * Hkv, d), device="cuda")
    ws = torch.zeros(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
    rk.reskv_decode_attn(shape, rk.make_gate(), qd, kcd, vcd, lcd, rl, ml, out, ws, k_new=knd, v_new=vnd)
    torch.cuda.synchronize()
    kc2, vc2, main2 = kc.copy(), vc.copy(), main.copy()
    for b in range(B):
        for h in range(Hkv):
            slot = res[b, h] + main[b, h]
            if slot < C:
                kc2[b, h, slot] = knd[b, h].double().cpu().numpy()
                vc2[b, h, slot] = vnd[b, h].double().cpu().numpy()
                main2[b, h] += 1
    np.testing.assert_array_equal(ml.cpu().numpy().reshape(B, Hkv), main2)
    np.testing.assert_array_equal(kcd.double().cpu().numpy(), kc2)
    np.testing.assert_array_equal(vcd.double().cpu().numpy(), vc2)
    ref, *_ = orc.decode(q, kc2, vc2, logc, res, main2, 0.25, 12.0, 0.0, 1.0)
    assert rel_err_rows(out.double().cpu().numpy(), ref).max() <= TOL[dtype]


@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 64), ("f32", 128), ("bf16", 128)])
def test_decode_whole_head_path_shapes(dtype, d):
    """256 (b, kv head) pairs (the one-block-per-head kernel; fp32 rows of 128
    take the split kernels), with ragged lengths, r = 0 heads and empty
    entries."""
    B, Hkv, G = 64, 4, 4
    rng = np.random.default_rng(30 + d)
    C, Rcap = 700, 130
    res = rng.choice([0, 1, 63, 130], size=(B, Hkv))
    main = rng.integers(1, C - 130, size=(B, Hkv))
    shape, q, kc, vc, logc = cache_case(40 + d, B, G * Hkv, Hkv, d, dtype, C, Rcap, res, main)
    heads = [(int(b), int(h)) for b, h in zip(rng.integers(0, B, 40), rng.integers(0, G * Hkv, 40))]
    check(dtype, shape, q, kc, vc, logc, res, main, heads=heads)


@pytest.mark.parametrize("dtype,d,G", [("bf16", 128, 7), ("bf16", 128, 8), ("bf16", 64, 16), ("f32", 64, 7),
                                       ("bf16", 128, 16)])
def test_decode_whole_head_wide_groups(dtype, d, G):
    """256 (b, kv head) pairs with more than 4 query heads per KV head (the
    ragged GQA-7 workload's group, 8 and 16): the one-block-per-head kernel,
    whose waves merge the residual states and then the main states through
    one LDS buffer; ragged lengths, r = 0 heads, empty entries, per-query
    thresholds."""
    B, Hkv = 64, 4
    rng = np.random.default_rng(50 + d + G)
    C, Rcap = 640, 130
    res = rng.choice([0, 1, 63, 130], size=(B, Hkv))
    main = rng.integers(1, C - 130, size=(B, Hkv))
    shape, q, kc, vc, logc = cache_case(60 + d + G, B, G * Hkv, Hkv, d, dtype, C, Rcap, res, main)
    heads = [(int(b), int(h)) for b, h in zip(rng.integers(0, B, 48), rng.integers(0, G * Hkv, 48))]
    tau = rng.normal(0.0, 0.5, size=(B, G * Hkv))
    check(dtype, shape, q, kc, vc, logc, res, main, heads=heads, tau=tau)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_decode_whole_head_residual_boundary_inside_a_block(dtype, d):
    """256 (b, kv head) pairs whose residual count r is not a multiple of the
    64-slot unit: the block holding slot r is streamed as its residual part
    and its main part (dealt last), with this step's token appended before,
    at or after the end of that block, and heads short enough that the main
    part is a wave's first unit. Every query head is checked, and the
    appended rows and lengths bit for bit."""
    B, Hkv, G = 64, 4, 4
    rng = np.random.default_rng(70 + d)
    C, Rcap = 640, 200
    res = rng.choice([1, 37, 63, 64, 65, 127, 130, 191], size=(B, Hkv))
    ur = (res + 63) // 64
    # main lengths: inside the boundary block, exactly filling it, or past it
    pick = rng.integers(0, 3, size=(B, Hkv))
    main = np.where(pick == 0, np.maximum(1, 64 * ur - res - 1 - rng.integers(0, 8, size=(B, Hkv))),
                    np.where(pick == 1, np.maximum(1, 64 * ur - res), rng.integers(1, C - 200, size=(B, Hkv))))
    main = np.minimum(main, C - res - 1)
    shape, q, kc, vc, logc = cache_case(80 + d, B, G * Hkv, Hkv, d, dtype, C, Rcap, res, main)
    kn = rng.normal(size=(B, Hkv, d))
    vn = rng.normal(size=(B, Hkv, d))
    knd, vnd = to_dev(kn, dtype), to_dev(vn, dtype)
    kcd, vcd = to_dev(kc, dtype), to_dev(vc, dtype)
    lcd = torch.as_tensor(logc.astype(np.float32)).cuda()
    rl = torch.as_tensor(res.astype(np.int32).reshape(-1)).cuda()
    ml = torch.as_tensor(main.astype(np.int32).reshape(-1)).cuda()
    out = torch.empty((B, G * Hkv, d), device="cuda")
    ws = torch.zeros(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
    rk.reskv_decode_attn(shape, rk.make_gate(), to_dev(q, dtype), kcd, vcd, lcd, rl, ml, out, ws,
                         k_new=knd, v_new=vnd)
    torch.cuda.synchronize()
    kc2, vc2, main2 = kc.copy(), vc.copy(), main + 1
    for b in range(B):
        for h in range(Hkv):
            kc2[b, h, res[b, h] + main[b, h]] = knd[b, h].double().cpu().numpy()
            vc2[b, h, res[b, h] + main[b, h]] = vnd[b, h].double().cpu().numpy()
    np.testing.assert_array_equal(ml.cpu().numpy().reshape(B, Hkv), main2)
    np.testing.assert_array_equal(kcd.double().cpu().numpy(), kc2)
    np.testing.assert_array_equal(vcd.double().cpu().numpy(), vc2)
    ref, *_ = orc.decode(q, kc2, vc2, logc, res, main2, 0.25, 12.0, 0.0, 1.0)
    assert rel_err_rows(out.double().cpu().numpy(), ref).max() <= TOL[dtype]


def test_prepared_decode_call_matches_direct_call():
    """prepare_decode_attn marshals the arguments once; issuing it twice
    (each call appends a token) gives the same caches, lengths and outputs,
    bit for bit, as two reskv_decode_attn calls."""
    B, Hkv, G, d, dtype = 4, 2, 4, 128, "bf16"
    rng = np.random.default_rng(77)
    C, Rcap = 200, 32
    res = rng.choice([0, 16, 32], size=(B, Hkv))
    main = rng.integers(1, C - 40, size=(B, Hkv))
    shape, q, kc, vc, logc = cache_case(77, B, G * Hkv, Hkv, d, dtype, C, Rcap, res, main)
    kn, vn = to_dev(rng.normal(size=(B, Hkv, d)), dtype), to_dev(rng.normal(size=(B, Hkv, d)), dtype)
    qd = to_dev(q, dtype)
    runs = []
    for prepared in (False, True):
        kcd, vcd = to_dev(kc, dtype), to_dev(vc, dtype)
        lcd = torch.as_tensor(logc.astype(np.float32)).cuda()
        rl = torch.as_tensor(res.astype(np.int32).reshape(-1)).cuda()
        ml = torch.as_tensor(main.astype(np.int32).reshape(-1)).cuda()
        out = torch.empty((B, G * Hkv, d), device="cuda")
        ws = torch.zeros(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
        gate = rk.make_gate()
        if prepared:
            call = rk.prepare_decode_attn(shape, gate, qd, kcd, vcd, lcd, rl, ml, out, ws, k_new=kn, v_new=vn)
            call()
            call()
        else:
            for _ in range(2):
                rk.reskv_decode_attn(shape, gate, qd, kcd, vcd, lcd, rl, ml, out, ws, k_new=kn, v_new=vn)
        torch.cuda.synchronize()
        runs.append([t.cpu() for t in (kcd, vcd, ml, out)])
    for a, b in zip(*runs):
        assert torch.equal(a, b)
