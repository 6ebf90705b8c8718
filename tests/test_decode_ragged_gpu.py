"""GPU parity of reskv_decode_attn_ragged (the balanced-range schedule of
the shared-softmax decode, Sec. 5.4, Sec. 5.5.2, App. D Algorithm 2) against
the fp64 oracle, through the C ABI.

Cases cover: fewer units than blocks (every head split over many blocks,
each block one unit or none), more units than 16 per CU (more blocks than
CUs), heads of one unit, r = 0 and empty residual entries, group sizes
1-8, bf16 d 64/128 and fp32 d 64, the fused append (cache rows, main_len)
with full caches left unchanged, per-query tau, and agreement with
reskv_decode_attn on the same inputs."""

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import reskv as rk
from tests.helpers import TOL, gate_atol, random_cache, rel_err_rows, to_dev

pytestmark = pytest.mark.gpu

GATE = dict(tau_scalar=0.25, alpha=12.0, g_min=0.0, beta=1.0)


def ragged_case(seed, B, Hkv, G, d, dtype, C, Rcap, res, main, appends):
    rng = np.random.default_rng(seed)
    kc, vc, logc = random_cache(rng, B, Hkv, C, Rcap, d, dtype, res, main)
    q = rng.normal(size=(B, Hkv * G, d)) * 1.5
    q = np.asarray(torch.as_tensor(q, dtype=torch.float32).to(torch.bfloat16).double()) if dtype == "bf16" else \
        q.astype(np.float32).astype(np.float64)
    tau = rng.normal(0.0, 0.5, size=(B, Hkv * G)).astype(np.float32)
    kn = vn = None
    if appends:
        store = (lambda x: torch.as_tensor(x, dtype=torch.float32).to(torch.bfloat16).double().numpy()) \
            if dtype == "bf16" else (lambda x: np.asarray(x, np.float32).astype(np.float64))
        kn = store(rng.normal(size=(B, Hkv, d)))
        vn = store(rng.normal(size=(B, Hkv, d)))
    return q, kc, vc, logc, tau, kn, vn


def run_ragged(dtype, B, Hkv, G, d, C, Rcap, res, main, seed=0, appends=True, compare_head=False):
    res = np.asarray(res, np.int64)
    main = np.asarray(main, np.int64)
    q, kc, vc, logc, tau, kn, vn = ragged_case(seed, B, Hkv, G, d, dtype, C, Rcap, res, main, appends)
    shape = rk.make_shape(B, Hkv * G, Hkv, d, dtype, C, Rcap)
    nws = rk.reskv_decode_ragged_workspace_size(shape)
    assert nws > 0
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    dev = dict(q=to_dev(q, dtype), kc=to_dev(kc, dtype), vc=to_dev(vc, dtype),
               logc=torch.as_tensor(logc.astype(np.float32)).cuda().contiguous(),
               rl=torch.as_tensor(res.astype(np.int32).reshape(-1)).cuda(),
               ml=torch.as_tensor(main.astype(np.int32).reshape(-1)).cuda(),
               tau=torch.as_tensor(tau.reshape(-1)).cuda())
    kw = {}
    if appends:
        kw = dict(k_new=to_dev(kn, dtype), v_new=to_dev(vn, dtype))
    out = torch.full((B, Hkv * G, d), float("nan"), device="cuda")
    dbg = [torch.full((B * Hkv * G,), float("nan"), device="cuda") for _ in range(3)]
    gate = rk.make_gate(tau=dev["tau"], **{k: v for k, v in GATE.items() if k != "tau_scalar"})
    kc0, vc0, ml0 = dev["kc"].clone(), dev["vc"].clone(), dev["ml"].clone()
    rk.reskv_decode_attn_ragged(shape, gate, dev["q"], dev["kc"], dev["vc"], dev["logc"], dev["rl"], dev["ml"],
                                out, ws, *dbg, **kw)
    torch.cuda.synchronize()
    # the append: row r + n of every head with room, main_len + 1
    kc2, vc2, main2 = kc.copy(), vc.copy(), main.copy()
    if appends:
        for b in range(B):
            for h in range(Hkv):
                slot = res[b, h] + main[b, h]
                if slot < C:
                    kc2[b, h, slot] = kn[b, h]
                    vc2[b, h, slot] = vn[b, h]
                    main2[b, h] += 1
    np.testing.assert_array_equal(dev["ml"].cpu().numpy().reshape(B, Hkv), main2)
    np.testing.assert_array_equal(dev["kc"].double().cpu().numpy(), kc2)
    np.testing.assert_array_equal(dev["vc"].double().cpu().numpy(), vc2)
    ref, lm, lr, g = orc.decode(q, kc2, vc2, logc, res, main2, tau.astype(np.float64), GATE["alpha"],
                                GATE["g_min"], GATE["beta"])
    o = out.double().cpu().numpy()
    assert np.isfinite(o).all()
    err = rel_err_rows(o, ref).max()
    assert err <= TOL[dtype], f"max rel err {err:.3e}"
    dg = [t.double().cpu().numpy().reshape(B, Hkv * G) for t in dbg]
    np.testing.assert_allclose(dg[0], lm, rtol=1e-5, atol=1e-5)
    fin = np.isfinite(lr)
    assert (np.isfinite(dg[1]) == fin).all()
    np.testing.assert_allclose(dg[1][fin], lr[fin], rtol=1e-5, atol=1e-5)
    for b in range(B):
        for h in range(Hkv * G):
            kv = h // G
            K = kc2[b, kv, res[b, kv]:res[b, kv] + main2[b, kv]]
            tol = max(1e-5 * g[b, h], gate_atol(q[b, h], K, g[b, h], lm[b, h], GATE["alpha"]))
            assert abs(dg[2][b, h] - g[b, h]) <= tol
    if compare_head:
        # the same inputs through reskv_decode_attn: equal within rounding
        out2 = torch.empty_like(out)
        ws2 = torch.zeros(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
        rk.reskv_decode_attn(shape, gate, dev["q"], kc0, vc0, dev["logc"], dev["rl"], ml0, out2, ws2, **kw)
        torch.cuda.synchronize()
        assert torch.equal(ml0, dev["ml"]) and torch.equal(kc0, dev["kc"])
        assert rel_err_rows(out2.double().cpu().numpy(), o).max() <= TOL[dtype]
    return err


@pytest.mark.parametrize("dtype,d,G", [("bf16", 128, 7), ("bf16", 128, 4), ("bf16", 64, 8), ("f32", 64, 2),
                                       ("bf16", 128, 1)])
def test_ragged_few_units(dtype, d, G):
    """Fewer units than blocks: long heads are shared by many blocks of one
    unit each."""
    B, Hkv, C, Rcap = 3, 4, 1200, 320
    res = [[0, 300, 16, 64], [257, 0, 1, 128], [0, 0, 64, 5]]
    main = [[1, 850, 1100, 64], [900, 1200, 33, 1000], [65, 640, 1, 700]]
    run_ragged(dtype, B, Hkv, G, d, C, Rcap, res, main, seed=d + G, compare_head=True)


def test_ragged_many_units():
    """More than 16 units per CU: more blocks than the chip's CUs, heads of
    1 to 36 units, ragged over a GQA-7 batch of 384 (sequence, KV head)
    pairs (the one-block-per-head kernel takes the same inputs)."""
    rng = np.random.default_rng(5)
    B, Hkv, G, d, C, Rcap = 96, 4, 7, 128, 2304, 512
    res = rng.choice([0, 16, 64, 256, 512], size=(B, Hkv))
    main = np.minimum(rng.integers(1, 2000, size=(B, Hkv)), C - res)
    main[0, 0] = C - res[0, 0]  # full: no append
    run_ragged("bf16", B, Hkv, G, d, C, Rcap, res, main, seed=7, compare_head=True)


@pytest.mark.parametrize("appends", [False, True])
def test_ragged_gqa7_workload_shape(appends):
    """The ragged GQA-7 layer's shape (64 sequences x 4 KV heads, budgets
    256-1024 with r a fraction of the budget, room for 128 appends)."""
    rng = np.random.default_rng(11)
    B, Hkv, G, d = 64, 4, 7, 128
    budget = rng.choice([256, 512, 1024], size=B)
    frac = rng.uniform(0, 0.5, size=(B, Hkv))
    res = (16 * np.floor(frac * budget[:, None] / 16 + 0.5)).astype(np.int64)
    main = budget[:, None] - res + rng.integers(0, 128, size=(B, Hkv))
    C, Rcap = 1152, int(res.max())
    run_ragged("bf16", B, Hkv, G, d, C, Rcap, res, main, seed=13, appends=appends, compare_head=True)


def test_ragged_is_deterministic():
    B, Hkv, G, d, C, Rcap = 8, 4, 7, 128, 600, 64
    rng = np.random.default_rng(3)
    res = rng.choice([0, 16, 64], size=(B, Hkv))
    main = rng.integers(1, 500, size=(B, Hkv))
    q, kc, vc, logc, tau, _, _ = ragged_case(3, B, Hkv, G, d, "bf16", C, Rcap, res, main, False)
    shape = rk.make_shape(B, Hkv * G, Hkv, d, "bf16", C, Rcap)
    ws = torch.empty(rk.reskv_decode_ragged_workspace_size(shape), dtype=torch.uint8, device="cuda")
    args = [to_dev(q, "bf16"), to_dev(kc, "bf16"), to_dev(vc, "bf16"),
            torch.as_tensor(logc.astype(np.float32)).cuda(), torch.as_tensor(res.astype(np.int32).reshape(-1)).cuda(),
            torch.as_tensor(main.astype(np.int32).reshape(-1)).cuda()]
    outs = []
    for _ in range(2):
        out = torch.empty((B, Hkv * G, d), device="cuda")
        rk.reskv_decode_attn_ragged(shape, rk.make_gate(), *args, out, ws)
        outs.append(out)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


def test_ragged_long_heads():
    """Two 8000-slot heads over a grid of 256 blocks: the plan keeps at least
    two units per block so a head spans no more blocks than the combine
    merges, and each head is shared by about 60 blocks."""
    run_ragged("bf16", 1, 2, 4, 128, 8192, 512, [[0, 512]], [[8000, 7000]], seed=17, compare_head=True)


def test_ragged_skewed_batch():
    """One long head among many short ones (the batch the balanced schedule
    is for): 63 heads of 200-300 slots and one of 8000."""
    rng = np.random.default_rng(19)
    B, Hkv, G, d, C, Rcap = 16, 4, 4, 128, 8100, 64
    res = rng.choice([0, 16, 64], size=(B, Hkv))
    main = rng.integers(200, 300, size=(B, Hkv)) - res
    main[7, 2] = 8000 - res[7, 2]
    run_ragged("bf16", B, Hkv, G, d, C, Rcap, res, main, seed=23, compare_head=True)
