"""reskv_decode_attn_static (no workspace: split-K records in the library's
static device scratch) against reskv_decode_attn with a caller workspace,
through the C ABI: two calls in a row, the second on a smaller input, each
bit for bit equal to the workspace entry point on identical copies of the
cache (outputs, debug outputs, appended rows and lengths)."""

import numpy as np
import pytest
import torch

from paper_2607_29591_amd import reskv as rk
from tests.helpers import random_cache, to_dev

pytestmark = pytest.mark.gpu


def case(seed, B, Hq, Hkv, d, C, Rcap, res, main):
    rng = np.random.default_rng(seed)
    kc, vc, logc = random_cache(rng, B, Hkv, C, Rcap, d, "bf16", res, main)
    q = rng.normal(size=(B, Hq, d)) * 1.5
    kn = rng.normal(size=(B, Hkv, d))
    vn = rng.normal(size=(B, Hkv, d))
    shape = rk.make_shape(B, Hq, Hkv, d, "bf16", C, Rcap)
    dev = dict(q=to_dev(q, "bf16"), kc=to_dev(kc, "bf16"), vc=to_dev(vc, "bf16"),
               logc=torch.as_tensor(np.asarray(logc, np.float32)).cuda().contiguous(),
               rl=torch.as_tensor(np.asarray(res, np.int32).reshape(-1)).cuda(),
               ml=torch.as_tensor(np.asarray(main, np.int32).reshape(-1)).cuda(),
               kn=to_dev(kn, "bf16"), vn=to_dev(vn, "bf16"))
    return shape, dev


def run(shape, dev, static):
    B, Hq, d = dev["q"].shape
    kc, vc, ml = dev["kc"].clone(), dev["vc"].clone(), dev["ml"].clone()
    out = torch.full((B, Hq, d), float("nan"), device="cuda")
    dbg = [torch.full((B * Hq,), float("nan"), device="cuda") for _ in range(3)]
    gate = rk.make_gate()
    if static:
        rk.reskv_decode_attn_static(shape, gate, dev["q"], kc, vc, dev["logc"], dev["rl"], ml, out, *dbg,
                                    k_new=dev["kn"], v_new=dev["vn"])
    else:
        ws = torch.empty(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device="cuda")
        rk.reskv_decode_attn(shape, gate, dev["q"], kc, vc, dev["logc"], dev["rl"], ml, out, ws, *dbg,
                             k_new=dev["kn"], v_new=dev["vn"])
    torch.cuda.synchronize()
    return [out, *dbg, kc, vc, ml]


def same(a, b):
    for x, y in zip(a, b):
        assert torch.equal(x.nan_to_num(123.0), y.nan_to_num(123.0))
    assert torch.isfinite(a[0]).all()


def test_static_scratch_matches_workspace_two_calls():
    # first call: split-K path (6 (sequence, KV head) pairs), GQA 7, ragged
    # lengths over several 256-slot blocks, one cache full (no append)
    res1 = [[300, 0], [17, 256], [0, 64]]
    main1 = [[700, 1100], [1, 800], [513, 1036]]
    s1, d1 = case(3, 3, 14, 2, 128, 1100, 300, res1, main1)
    assert rk.reskv_decode_workspace_size(s1) > 0
    same(run(s1, d1, True), run(s1, d1, False))
    # second call, smaller: fewer pairs, shorter caches, d = 64, G = 4
    res2 = [[3, 40]]
    main2 = [[60, 300]]
    s2, d2 = case(4, 1, 8, 2, 64, 400, 64, res2, main2)
    assert rk.reskv_decode_workspace_size(s2) < rk.reskv_decode_workspace_size(s1)
    same(run(s2, d2, True), run(s2, d2, False))
