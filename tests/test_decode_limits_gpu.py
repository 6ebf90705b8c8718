"""GPU parity of the decode entry points at the largest sizes they accept
(Sec. 5.4 shared-softmax decode, Sec. 5.5.2 gate, App. D Algorithm 2):
a 65536-slot cache with 4096 residual entries through the split kernels, the
largest group (16 query heads per KV head) on the one-block-per-head kernel
with 8192-slot caches, and the ragged schedule at its 2048 (b, kv head)
pairs. Sampled query heads against the oracle, to the bar of the other
decode tests; the appended rows and lengths bit for bit.
"""

import numpy as np
import pytest
import torch

from oracle import reskv_oracle as orc
from paper_2607_29591_amd import reskv as rk
from tests.helpers import TOL, random_cache, rel_err_rows, to_dev

pytestmark = pytest.mark.gpu

GATE = dict(tau_scalar=0.25, alpha=12.0, g_min=0.0, beta=1.0)


def run(entry, seed, B, Hkv, G, d, dtype, C, Rcap, res, main, n_heads=48, empty_frac=0.1):
    rng = np.random.default_rng(seed)
    Hq = G * Hkv
    kc, vc, logc = random_cache(rng, B, Hkv, C, Rcap, d, dtype, res, main, empty_frac=empty_frac)
    q = rng.normal(size=(B, Hq, d)) * 1.5
    q = np.asarray(torch.as_tensor(q, dtype=torch.float32).to(torch.bfloat16).double()) if dtype == "bf16" else \
        q.astype(np.float32).astype(np.float64)
    kn, vn = rng.normal(size=(B, Hkv, d)), rng.normal(size=(B, Hkv, d))
    shape = rk.make_shape(B, Hq, Hkv, d, dtype, C, Rcap)
    kcd, vcd = to_dev(kc, dtype), to_dev(vc, dtype)
    knd, vnd = to_dev(kn, dtype), to_dev(vn, dtype)
    lcd = torch.as_tensor(logc.astype(np.float32)).cuda()
    rl = torch.as_tensor(res.astype(np.int32).reshape(-1)).cuda()
    ml = torch.as_tensor(main.astype(np.int32).reshape(-1)).cuda()
    out = torch.full((B, Hq, d), float("nan"), device="cuda")
    args = (shape, rk.make_gate(**GATE), to_dev(q, dtype), kcd, vcd, lcd, rl, ml, out)
    if entry == "ragged":
        ws = torch.zeros(rk.reskv_decode_ragged_workspace_size(shape), dtype=torch.uint8, device="cuda")
        rk.reskv_decode_attn_ragged(*args, ws, k_new=knd, v_new=vnd)
    else:
        ws = torch.zeros(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
        rk.reskv_decode_attn(*args, ws, k_new=knd, v_new=vnd)
    torch.cuda.synchronize()
    main2 = main.copy()
    knr, vnr = knd.double().cpu().numpy(), vnd.double().cpu().numpy()
    got_k, got_v = kcd.double().cpu().numpy(), vcd.double().cpu().numpy()
    for b in range(B):
        for h in range(Hkv):
            slot = res[b, h] + main[b, h]
            if slot < C:
                kc[b, h, slot], vc[b, h, slot] = knr[b, h], vnr[b, h]
                main2[b, h] += 1
    np.testing.assert_array_equal(ml.cpu().numpy().reshape(B, Hkv), main2)
    np.testing.assert_array_equal(got_k, kc)
    np.testing.assert_array_equal(got_v, vc)
    sel = rng.choice(B * Hq, size=min(n_heads, B * Hq), replace=False)
    heads = [(int(i) // Hq, int(i) % Hq) for i in sel]
    ref, *_ = orc.decode(q, kc, vc, logc, res, main2, GATE["tau_scalar"], GATE["alpha"], GATE["g_min"],
                         GATE["beta"], heads=heads)
    got = out.double().cpu().numpy()
    bi, hi = np.array(heads).T
    assert np.isfinite(got[bi, hi]).all()
    err = rel_err_rows(got[bi, hi], ref[bi, hi])
    assert err.max() <= TOL[dtype], f"max rel err {err.max():.3e}"


def test_split_path_65536_slots():
    """Two (b, kv head) pairs of 65536 slots: 4096 residual entries and a
    main cache filling the rest, and one residual entry with a 60000-slot
    main cache; 16 query heads per KV head; the split kernels (256 records
    per head)."""
    res = np.array([[4096, 1]])
    main = np.array([[65536 - 4096, 60000]])
    run("workspace", 1, 1, 2, 16, 128, "bf16", 65536, 4096, res, main, n_heads=32, empty_frac=0.02)


def test_whole_head_largest_group_8192_slots():
    """256 pairs of 8192-slot caches with 16 query heads each (the one-block-
    per-head kernel at its widest group), residual counts up to 512."""
    B, Hkv = 64, 4
    rng = np.random.default_rng(2)
    res = rng.integers(0, 513, size=(B, Hkv))
    main = np.array([[int(rng.integers(1, 8192 - r)) for r in row] for row in res])
    run("workspace", 2, B, Hkv, 16, 128, "bf16", 8192, 512, res, main)


def test_ragged_schedule_2048_pairs():
    """The ragged schedule at its largest batch: 2048 (b, kv head) pairs,
    8 query heads each, ragged lengths in 512-slot caches."""
    B, Hkv = 512, 4
    rng = np.random.default_rng(3)
    res = rng.integers(0, 65, size=(B, Hkv))
    main = np.array([[int(rng.integers(1, 512 - r)) for r in row] for row in res])
    run("ragged", 3, B, Hkv, 8, 64, "bf16", 512, 64, res, main)
