"""GPU parity of reskv_decode_attn on seeded random shapes (Sec. 5.4
shared-softmax decode, Sec. 5.5.2 gate, App. D Algorithm 2).

Each seed draws a cache geometry (group size, head dim, storage type, slot
capacity, residual capacity, per-head residual and main lengths), a gate, a
per-query or scalar threshold, and whether this step's token is appended in
the call; every query head is compared with the oracle decoding the same
cache (after the append), to the bar of the other decode tests. About half
of the seeds have 256 (b, kv head) pairs (the one-block-per-head kernel),
the others a few pairs (the split kernels).
"""

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import reskv as rk
from tests.helpers import TOL, random_cache, rel_err_rows, to_dev

pytestmark = pytest.mark.gpu


def draw_case(seed):
    rng = np.random.default_rng(1000 + seed)
    dtype = ["bf16", "f32"][seed % 2]
    d = [64, 128][(seed // 2) % 2]
    G = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 12, 16]))
    whole = (seed // 4) % 2 == 0 and (dtype == "bf16" or d == 64)
    if whole:
        Hkv = int(rng.choice([1, 2, 4, 8]))
        B = 256 // Hkv
        C = int(rng.integers(8, 360))
        Rcap = int(rng.integers(1, 48))
    else:
        Hkv = int(rng.choice([1, 2, 4]))
        B = int(rng.integers(1, 6))
        C = int(rng.integers(8, 1400))
        Rcap = int(rng.integers(1, 300))
    res = rng.integers(0, min(Rcap, C - 1) + 1, size=(B, Hkv))
    main = np.array([[int(rng.integers(1, C - r + 1)) for r in row] for row in res])
    gate = dict(tau_scalar=float(rng.uniform(0.05, 0.6)), alpha=float(rng.choice([4.0, 12.0])),
                g_min=float(rng.choice([0.0, 0.2])), beta=float(rng.choice([0.5, 1.0])))
    per_query_tau = bool(rng.integers(0, 2))
    append = bool(rng.integers(0, 2))
    return rng, dtype, d, G, B, Hkv, C, Rcap, res, main, gate, per_query_tau, append


@pytest.mark.parametrize("seed", list(range(16)))
def test_decode_random_shape(seed):
    rng, dtype, d, G, B, Hkv, C, Rcap, res, main, gate, per_query_tau, append = draw_case(seed)
    Hq = G * Hkv
    kc, vc, logc = random_cache(rng, B, Hkv, C, Rcap, d, dtype, res, main)
    q = rng.normal(size=(B, Hq, d)) * 1.5
    q = np.asarray(torch.as_tensor(q, dtype=torch.float32).to(torch.bfloat16).double()) if dtype == "bf16" else \
        q.astype(np.float32).astype(np.float64)
    tau = rng.normal(0.3, 0.2, size=(B, Hq)) if per_query_tau else None
    shape = rk.make_shape(B, Hq, Hkv, d, dtype, C, Rcap)

    kcd, vcd = to_dev(kc, dtype), to_dev(vc, dtype)
    lcd = torch.as_tensor(logc.astype(np.float32)).cuda()
    rl = torch.as_tensor(res.astype(np.int32).reshape(-1)).cuda()
    ml = torch.as_tensor(main.astype(np.int32).reshape(-1)).cuda()
    out = torch.full((B, Hq, d), float("nan"), device="cuda")
    lm = torch.empty(B * Hq, device="cuda")
    lr = torch.empty(B * Hq, device="cuda")
    gt = torch.empty(B * Hq, device="cuda")
    taud = None if tau is None else torch.as_tensor(tau.astype(np.float32).reshape(-1)).cuda()
    ws = torch.zeros(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
    kn = vn = knd = vnd = None
    if append:
        kn, vn = rng.normal(size=(B, Hkv, d)), rng.normal(size=(B, Hkv, d))
        knd, vnd = to_dev(kn, dtype), to_dev(vn, dtype)
    rk.reskv_decode_attn(shape, rk.make_gate(tau=taud, **gate), to_dev(q, dtype), kcd, vcd, lcd, rl, ml, out, ws,
                         lm, lr, gt, k_new=knd, v_new=vnd)
    torch.cuda.synchronize()

    main2 = main.copy()
    if append:  # the token becomes main slot r + n wherever the cache has room
        for b in range(B):
            for h in range(Hkv):
                slot = res[b, h] + main[b, h]
                if slot < C:
                    kc[b, h, slot] = knd[b, h].double().cpu().numpy()
                    vc[b, h, slot] = vnd[b, h].double().cpu().numpy()
                    main2[b, h] += 1
        np.testing.assert_array_equal(kcd.double().cpu().numpy(), kc)
        np.testing.assert_array_equal(vcd.double().cpu().numpy(), vc)
    np.testing.assert_array_equal(ml.cpu().numpy().reshape(B, Hkv), main2)

    t = gate["tau_scalar"] if tau is None else tau.astype(np.float32).astype(np.float64)
    ref, lse_m, lse_r, g = orc.decode(q, kc, vc, logc, res, main2, t, gate["alpha"], gate["g_min"], gate["beta"])
    got = out.double().cpu().numpy()
    assert np.isfinite(got).all()
    err = rel_err_rows(got, ref)
    assert err.max() <= TOL[dtype], f"max rel err {err.max():.3e}"
    np.testing.assert_allclose(gt.double().cpu().numpy().reshape(B, Hq), g, rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(lm.double().cpu().numpy().reshape(B, Hq), lse_m, rtol=1e-5, atol=1e-5)
    got_lr = lr.double().cpu().numpy().reshape(B, Hq)
    fin = np.isfinite(lse_r)
    assert (np.isfinite(got_lr) == fin).all()
    np.testing.assert_allclose(got_lr[fin], lse_r[fin], rtol=1e-5, atol=1e-5)
