"""Host-side checks of the C ABI: the library loads, exports every entry
point declared in include/reskv.h, sizes workspaces, and rejects bad
arguments before launching anything (no GPU needed)."""

import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_29591_amd import reskv as rk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(rk.LIB_PATH):
        from paper_2607_29591_amd import build_lib
        build_lib.build()
    return rk.lib()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "reskv.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(reskv_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert {"reskv_build_cache", "reskv_decode_attn", "reskv_append_kv"} <= set(names)
    for n in names:
        assert hasattr(L, n), n
    assert set(rk._SIG) == set(names)


def test_status_strings(L):
    assert rk.status_string(0) == "ok"
    assert "workspace" in rk.status_string(3)


def shape(**kw):
    d = dict(batch=2, num_q_heads=8, num_kv_heads=2, head_dim=128, dtype="bf16", slot_cap=640, res_cap=64)
    d.update(kw)
    return rk.make_shape(**d)


def test_decode_workspace_size(L):
    s = shape()
    n = rk.reskv_decode_workspace_size(s)
    # 1 residual chunk + 3 main chunks of 256 slots, 4 heads, d + 2 floats each
    assert n >= 2 * 2 * 4 * 4 * (128 + 2) * 4
    assert rk.reskv_decode_workspace_size(shape(head_dim=96)) == 0
    assert rk.reskv_decode_workspace_size(shape(num_q_heads=7)) == 0


class FakeTensor:
    """Stands in for a device tensor: a non-null pointer that is never
    dereferenced because validation fails first."""

    def __init__(self, nbytes=16):
        self._n = nbytes

    def is_contiguous(self):
        return True

    def data_ptr(self):
        return 0x1000

    def numel(self):
        return self._n

    def element_size(self):
        return 1


@pytest.mark.parametrize("bad,code", [
    (dict(head_dim=96), 2), (dict(num_q_heads=7), 1), (dict(num_q_heads=34), 2),
    (dict(batch=0), 1), (dict(slot_cap=0), 1), (dict(dtype=5), 2)])
def test_decode_rejects_bad_shapes(L, bad, code):
    t = FakeTensor()
    with pytest.raises(rk.ReskvError) as ei:
        rk.reskv_decode_attn(shape(**bad), rk.make_gate(), t, t, t, t, t, t, t, t, stream=FakeStream())
    assert ei.value.status == code
    assert rk.last_error()


class FakeStream:
    cuda_stream = 0


def test_decode_rejects_small_workspace_and_bad_gate(L):
    t = FakeTensor()
    with pytest.raises(rk.ReskvError) as ei:
        rk.reskv_decode_attn(shape(), rk.make_gate(), t, t, t, t, t, t, t, FakeTensor(8), stream=FakeStream())
    assert ei.value.status == 3
    with pytest.raises(rk.ReskvError) as ei:
        rk.reskv_decode_attn(shape(), rk.make_gate(g_min=1.5), t, t, t, t, t, t, t, t, stream=FakeStream())
    assert ei.value.status == 1
    with pytest.raises(rk.ReskvError) as ei:
        rk.reskv_decode_attn(shape(), rk.make_gate(), None, t, t, t, t, t, t, t, stream=FakeStream())
    assert ei.value.status == 1
