"""Python binding of the ResKV C ABI (include/reskv.h).

Argument marshalling only: every step of construction and decode runs in the
HIP kernels of libreskv.so. Torch tensors supply device memory and the
current stream; this module passes their raw pointers through ctypes. If the
library is missing or fails to load, every entry point raises.
"""

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libreskv.so")

RESKV_F32 = 0
RESKV_BF16 = 1

STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported configuration",
          3: "workspace missing or too small", 4: "HIP runtime error"}


class ReskvError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("slot_cap", ctypes.c_int32),
                ("res_cap", ctypes.c_int32)]


class BuildParams(ctypes.Structure):
    _fields_ = [("max_seq_len", ctypes.c_int32), ("obs_window", ctypes.c_int32),
                ("recent_window", ctypes.c_int32), ("lloyd_iters", ctypes.c_int32),
                ("fit_rows", ctypes.c_int32), ("pool_kernel", ctypes.c_int32)]


class ProxyParams(ctypes.Structure):
    _fields_ = [("grid_host", ctypes.POINTER(ctypes.c_double)), ("n_grid", ctypes.c_int32),
                ("val_rows", ctypes.c_int32), ("delta", ctypes.c_float)]


class Gate(ctypes.Structure):
    _fields_ = [("tau", ctypes.c_void_p), ("tau_scalar", ctypes.c_float),
                ("alpha", ctypes.c_float), ("g_min", ctypes.c_float), ("beta", ctypes.c_float)]


_lib = None

_P = ctypes.c_void_p
_SIG = {
    "reskv_build_cache": (ctypes.c_int, [ctypes.POINTER(Shape), ctypes.POINTER(BuildParams), _P, _P, _P, _P,
                                         _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "reskv_build_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(Shape), ctypes.POINTER(BuildParams),
                                                     _P, _P, _P]),
    "reskv_build_cache_adakv": (ctypes.c_int, [ctypes.POINTER(Shape), ctypes.POINTER(BuildParams), ctypes.c_double,
                                               ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                               _P, _P, _P, ctypes.c_size_t, _P]),
    "reskv_build_adakv_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(Shape), ctypes.POINTER(BuildParams),
                                                           ctypes.c_double, ctypes.c_int32, _P, _P, _P]),
    "reskv_build_cache_proxy": (ctypes.c_int, [ctypes.POINTER(Shape), ctypes.POINTER(BuildParams),
                                               ctypes.POINTER(ProxyParams), ctypes.POINTER(Gate), _P, _P, _P, _P,
                                               _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "reskv_build_proxy_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(Shape), ctypes.POINTER(BuildParams),
                                                           ctypes.POINTER(ProxyParams), _P, _P]),
    "reskv_decode_attn": (ctypes.c_int, [ctypes.POINTER(Shape), ctypes.POINTER(Gate), _P, _P, _P, _P, _P, _P,
                                         _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "reskv_decode_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(Shape)]),
    "reskv_decode_attn_ragged": (ctypes.c_int, [ctypes.POINTER(Shape), ctypes.POINTER(Gate), _P, _P, _P, _P, _P,
                                                _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "reskv_decode_ragged_workspace_size": (ctypes.c_size_t, [ctypes.POINTER(Shape)]),
    "reskv_decode_attn_static": (ctypes.c_int, [ctypes.POINTER(Shape), ctypes.POINTER(Gate), _P, _P, _P, _P, _P,
                                                _P, _P, _P, _P, _P, _P, _P, _P]),
    "reskv_decode_branches": (ctypes.c_int, [ctypes.POINTER(Shape), ctypes.POINTER(Gate), _P, _P, _P, _P, _P, _P,
                                             _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "reskv_merge_branches": (ctypes.c_int, [ctypes.POINTER(Shape), ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P]),
    "reskv_append_kv": (ctypes.c_int, [ctypes.POINTER(Shape), _P, _P, _P, _P, _P, _P, _P]),
    "reskv_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "reskv_last_error": (ctypes.c_char_p, []),
}


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_29591_amd.build_lib` (or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIG.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status):
    if status != 0:
        raise ReskvError(status, lib().reskv_last_error().decode())


def _ptr(t):
    """Raw device pointer of a contiguous tensor (None -> NULL)."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the ResKV library must be contiguous")
    return t.data_ptr()


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def make_shape(batch, num_q_heads, num_kv_heads, head_dim, dtype, slot_cap, res_cap):
    dt = {"f32": RESKV_F32, "bf16": RESKV_BF16}.get(dtype, dtype)
    return Shape(batch, num_q_heads, num_kv_heads, head_dim, dt, slot_cap, res_cap)


def make_gate(tau=None, tau_scalar=0.25, alpha=12.0, g_min=0.0, beta=1.0):
    return Gate(_ptr(tau), tau_scalar, alpha, g_min, beta)


def _host_i32(x):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.int32).reshape(-1))
    return a, a.ctypes.data_as(ctypes.c_void_p)


def reskv_build_workspace_size(shape, params, seq_len, budget, res_count):
    sl, slp = _host_i32(seq_len)
    bu, bup = _host_i32(budget)
    rc, rcp = _host_i32(res_count)
    return lib().reskv_build_workspace_size(ctypes.byref(shape), ctypes.byref(params), slp, bup, rcp)


def reskv_build_cache(shape, params, k, v, seq_len, q_obs, budget, res_count, kc, vc, logc, main_idx,
                      res_len, main_len, workspace, dbg_scores=None, dbg_assign=None, dbg_centers=None,
                      stream=None):
    sl, slp = _host_i32(seq_len)
    bu, bup = _host_i32(budget)
    rc, rcp = _host_i32(res_count)
    _check(lib().reskv_build_cache(ctypes.byref(shape), ctypes.byref(params), _ptr(k), _ptr(v), slp,
                                   _ptr(q_obs), bup, rcp, _ptr(kc), _ptr(vc), _ptr(logc), _ptr(main_idx),
                                   _ptr(res_len), _ptr(main_len), _ptr(dbg_scores), _ptr(dbg_assign),
                                   _ptr(dbg_centers), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                   _stream(stream)))


def reskv_build_adakv_workspace_size(shape, params, safeguard, decode_reserve, seq_len, budget, res_count):
    sl, slp = _host_i32(seq_len)
    bu, bup = _host_i32(budget)
    rc, rcp = _host_i32(res_count)
    return lib().reskv_build_adakv_workspace_size(ctypes.byref(shape), ctypes.byref(params), float(safeguard),
                                                  int(decode_reserve), slp, bup, rcp)


def reskv_build_cache_adakv(shape, params, safeguard, decode_reserve, k, v, seq_len, q_obs, budget, res_count, kc,
                            vc, logc, main_idx, res_len, main_len, workspace, dbg_scores=None, dbg_assign=None,
                            dbg_centers=None, stream=None):
    sl, slp = _host_i32(seq_len)
    bu, bup = _host_i32(budget)
    rc, rcp = _host_i32(res_count)
    _check(lib().reskv_build_cache_adakv(ctypes.byref(shape), ctypes.byref(params), float(safeguard),
                                         int(decode_reserve), _ptr(k), _ptr(v), slp, _ptr(q_obs), bup, rcp, _ptr(kc),
                                         _ptr(vc), _ptr(logc), _ptr(main_idx), _ptr(res_len), _ptr(main_len),
                                         _ptr(dbg_scores), _ptr(dbg_assign), _ptr(dbg_centers), _ptr(workspace),
                                         workspace.numel() * workspace.element_size(), _stream(stream)))


def make_proxy(grid=(0.0, 0.05, 0.10, 0.15, 0.20), val_rows=8, delta=0.01):
    """Proxy parameters; the grid array lives on the returned object."""
    g = (ctypes.c_double * len(grid))(*[float(f) for f in grid])
    x = ProxyParams(ctypes.cast(g, ctypes.POINTER(ctypes.c_double)), len(grid), val_rows, delta)
    x._grid = g  # keep the host array alive with the struct
    return x


def reskv_build_proxy_workspace_size(shape, params, proxy, seq_len, budget):
    sl, slp = _host_i32(seq_len)
    bu, bup = _host_i32(budget)
    return lib().reskv_build_proxy_workspace_size(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(proxy),
                                                  slp, bup)


def reskv_build_cache_proxy(shape, params, proxy, gate, k, v, seq_len, q_obs, budget, kc, vc, logc, main_idx,
                            res_len, main_len, workspace, val_loss=None, stream=None):
    sl, slp = _host_i32(seq_len)
    bu, bup = _host_i32(budget)
    _check(lib().reskv_build_cache_proxy(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(proxy),
                                         ctypes.byref(gate), _ptr(k), _ptr(v), slp, _ptr(q_obs), bup, _ptr(kc),
                                         _ptr(vc), _ptr(logc), _ptr(main_idx), _ptr(res_len), _ptr(main_len),
                                         _ptr(val_loss), _ptr(workspace),
                                         workspace.numel() * workspace.element_size(), _stream(stream)))


def reskv_decode_workspace_size(shape):
    return lib().reskv_decode_workspace_size(ctypes.byref(shape))


def reskv_decode_attn(shape, gate, q, kc, vc, logc, res_len, main_len, out, workspace,
                      dbg_lse_main=None, dbg_lse_res=None, dbg_gate=None, k_new=None, v_new=None, stream=None):
    _check(lib().reskv_decode_attn(ctypes.byref(shape), ctypes.byref(gate), _ptr(q), _ptr(kc), _ptr(vc),
                                   _ptr(logc), _ptr(res_len), _ptr(main_len), _ptr(k_new), _ptr(v_new), _ptr(out),
                                   _ptr(dbg_lse_main), _ptr(dbg_lse_res), _ptr(dbg_gate), _ptr(workspace),
                                   workspace.numel() * workspace.element_size(), _stream(stream)))


def reskv_decode_ragged_workspace_size(shape):
    return lib().reskv_decode_ragged_workspace_size(ctypes.byref(shape))


def reskv_decode_attn_ragged(shape, gate, q, kc, vc, logc, res_len, main_len, out, workspace, dbg_lse_main=None,
                             dbg_lse_res=None, dbg_gate=None, k_new=None, v_new=None, stream=None):
    _check(lib().reskv_decode_attn_ragged(ctypes.byref(shape), ctypes.byref(gate), _ptr(q), _ptr(kc), _ptr(vc),
                                          _ptr(logc), _ptr(res_len), _ptr(main_len), _ptr(k_new), _ptr(v_new),
                                          _ptr(out), _ptr(dbg_lse_main), _ptr(dbg_lse_res), _ptr(dbg_gate),
                                          _ptr(workspace), workspace.numel() * workspace.element_size(),
                                          _stream(stream)))


def prepare_decode_attn_ragged(shape, gate, q, kc, vc, logc, res_len, main_len, out, workspace,
                               dbg_lse_main=None, dbg_lse_res=None, dbg_gate=None, k_new=None, v_new=None,
                               stream=None):
    """As prepare_decode_attn, for reskv_decode_attn_ragged."""
    fn = lib().reskv_decode_attn_ragged
    args = (ctypes.byref(shape), ctypes.byref(gate), _ptr(q), _ptr(kc), _ptr(vc), _ptr(logc), _ptr(res_len),
            _ptr(main_len), _ptr(k_new), _ptr(v_new), _ptr(out), _ptr(dbg_lse_main), _ptr(dbg_lse_res),
            _ptr(dbg_gate), _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream))
    keep = (shape, gate)

    def call():
        status = fn(*args)
        if status != 0:
            _check(status)

    call.keep = keep
    return call


def reskv_decode_attn_static(shape, gate, q, kc, vc, logc, res_len, main_len, out, dbg_lse_main=None,
                             dbg_lse_res=None, dbg_gate=None, k_new=None, v_new=None, stream=None):
    _check(lib().reskv_decode_attn_static(ctypes.byref(shape), ctypes.byref(gate), _ptr(q), _ptr(kc), _ptr(vc),
                                          _ptr(logc), _ptr(res_len), _ptr(main_len), _ptr(k_new), _ptr(v_new),
                                          _ptr(out), _ptr(dbg_lse_main), _ptr(dbg_lse_res), _ptr(dbg_gate),
                                          _stream(stream)))


def prepare_decode_attn(shape, gate, q, kc, vc, logc, res_len, main_len, out, workspace,
                        dbg_lse_main=None, dbg_lse_res=None, dbg_gate=None, k_new=None, v_new=None, stream=None):
    """Marshal the arguments of one reskv_decode_attn call once and return a
    function that issues it (for loops that launch the same calls many
    times). The caller keeps the tensors alive and unchanged in place."""
    fn = lib().reskv_decode_attn
    args = (ctypes.byref(shape), ctypes.byref(gate), _ptr(q), _ptr(kc), _ptr(vc), _ptr(logc), _ptr(res_len),
            _ptr(main_len), _ptr(k_new), _ptr(v_new), _ptr(out), _ptr(dbg_lse_main), _ptr(dbg_lse_res),
            _ptr(dbg_gate), _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream))
    keep = (shape, gate)

    def call():
        status = fn(*args)
        if status != 0:
            _check(status)

    call.keep = keep
    return call


RESKV_MERGE_SHARED, RESKV_MERGE_SEPARATE = 0, 1


def reskv_decode_branches(shape, gate, q, kc, vc, logc, res_len, main_len, out_main, lse_main, out_res, lse_res,
                          gate_out, workspace, stream=None):
    _check(lib().reskv_decode_branches(ctypes.byref(shape), ctypes.byref(gate), _ptr(q), _ptr(kc), _ptr(vc),
                                       _ptr(logc), _ptr(res_len), _ptr(main_len), _ptr(out_main), _ptr(lse_main),
                                       _ptr(out_res), _ptr(lse_res), _ptr(gate_out), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _stream(stream)))


def reskv_merge_branches(shape, mode, out_main, lse_main, out_res, lse_res, gate, out, stream=None):
    _check(lib().reskv_merge_branches(ctypes.byref(shape), int(mode), _ptr(out_main), _ptr(lse_main), _ptr(out_res),
                                      _ptr(lse_res), _ptr(gate), _ptr(out), _stream(stream)))


def reskv_append_kv(shape, k_new, v_new, kc, vc, res_len, main_len, stream=None):
    _check(lib().reskv_append_kv(ctypes.byref(shape), _ptr(k_new), _ptr(v_new), _ptr(kc), _ptr(vc),
                                 _ptr(res_len), _ptr(main_len), _stream(stream)))


def status_string(status):
    return lib().reskv_status_string(status).decode()


def last_error():
    return lib().reskv_last_error().decode()
