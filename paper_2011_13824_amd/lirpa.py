"""Thin ctypes binding of ``liblirpa.so`` (the C ABI declared in include/lirpa.h).

The functions below carry the C names and only marshal arguments: torch CUDA tensors become
device pointers and the current torch stream becomes the ``hipStream_t``.  Every step of the
bound computation runs in the HIP library; there is no fallback.  ``Network`` is a small
convenience owner of device weights, a net handle and a workspace.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liblirpa.so")

LIRPA_OK, LIRPA_EINVAL, LIRPA_ENOMEM, LIRPA_EDEVICE, LIRPA_EUNSUPPORTED, LIRPA_EDATA = \
    0, -1, -2, -3, -4, -5
LINEAR, CONV2D = 0, 1


class lirpa_layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("in_c", ctypes.c_int), ("in_h", ctypes.c_int),
                ("in_w", ctypes.c_int), ("out_c", ctypes.c_int), ("out_h", ctypes.c_int),
                ("out_w", ctypes.c_int), ("k", ctypes.c_int), ("stride", ctypes.c_int),
                ("pad", ctypes.c_int), ("W", ctypes.c_void_p), ("b", ctypes.c_void_p)]


class lirpa_opt_params(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int), ("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps_adam", ctypes.c_float), ("t0", ctypes.c_int),
                ("fresh", ctypes.c_int)]


class lirpa_bab_params(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int), ("max_domains", ctypes.c_int),
                ("max_iters", ctypes.c_int), ("root_steps", ctypes.c_int),
                ("steps", ctypes.c_int), ("lr", ctypes.c_float), ("beta1", ctypes.c_float),
                ("beta2", ctypes.c_float), ("eps_adam", ctypes.c_float)]


class lirpa_bab_result(ctypes.Structure):
    _fields_ = [("status", ctypes.c_int), ("f_lo", ctypes.c_float), ("f_hi", ctypes.c_float),
                ("iterations", ctypes.c_int), ("domains_bounded", ctypes.c_int64),
                ("domains_left", ctypes.c_int)]


BAB_VERIFIED, BAB_VIOLATED, BAB_UNKNOWN_STUCK, BAB_UNKNOWN_LIMIT = 1, 2, 3, 4


class lirpa_kernel_time(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("total_ms", ctypes.c_double),
                ("launches", ctypes.c_int64)]


SYMBOLS = ("lirpa_net_create", "lirpa_net_destroy", "lirpa_net_num_relu",
           "lirpa_workspace_bytes", "lirpa_bound", "lirpa_bound_child", "lirpa_bound_noalloc",
           "lirpa_bound_ul",
           "lirpa_bound_grad", "lirpa_optimize", "lirpa_optimize_ul",
           "lirpa_bab_workspace_bytes", "lirpa_bab",
           "lirpa_timing_begin", "lirpa_timing_end", "lirpa_last_error")

_lib = None


def load() -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built (no CPU fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -c 'import __graft_entry__ as g; g.build()'`")
    L = ctypes.CDLL(LIB_PATH)
    P, i, f, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    L.lirpa_net_create.argtypes = [ctypes.POINTER(lirpa_layer), i, ctypes.POINTER(P)]
    L.lirpa_net_create.restype = i
    L.lirpa_net_destroy.argtypes = [P]
    L.lirpa_net_destroy.restype = None
    L.lirpa_net_num_relu.argtypes = [P]
    L.lirpa_net_num_relu.restype = ctypes.c_int64
    L.lirpa_workspace_bytes.argtypes = [P, i, i, i]
    L.lirpa_workspace_bytes.restype = sz
    L.lirpa_bound.argtypes = [P, P, f, P, i, i, P, P, P, P, P, P, P, sz, P]
    L.lirpa_bound.restype = i
    L.lirpa_bound_child.argtypes = [P, P, f, P, i, i, P, P, P, P, P, P, P, P, P, sz, P]
    L.lirpa_bound_child.restype = i
    L.lirpa_bound_noalloc.argtypes = [P, P, f, P, i, i, P, P, P, P, P, P, P]
    L.lirpa_bound_noalloc.restype = i
    L.lirpa_bound_ul.argtypes = [P, P, f, P, i, i, P, P, P, P, P, P, P, P, sz, P]
    L.lirpa_bound_ul.restype = i
    L.lirpa_optimize_ul.argtypes = [P, P, f, P, i, i, P, P, P, P, P, P, P,
                                    ctypes.POINTER(lirpa_opt_params), P, P, P, sz, P]
    L.lirpa_optimize_ul.restype = i
    L.lirpa_bab_workspace_bytes.argtypes = [P, ctypes.POINTER(lirpa_bab_params)]
    L.lirpa_bab_workspace_bytes.restype = sz
    L.lirpa_bab.argtypes = [P, P, f, P, ctypes.POINTER(lirpa_bab_params),
                            ctypes.POINTER(lirpa_bab_result), P, sz, P]
    L.lirpa_bab.restype = i
    L.lirpa_bound_grad.argtypes = [P, P, f, P, i, i, P, P, i, P, P, P, sz, P]
    L.lirpa_bound_grad.restype = i
    L.lirpa_optimize.argtypes = [P, P, f, P, i, i, P, P, P, P, ctypes.POINTER(lirpa_opt_params),
                                 P, P, P, sz, P]
    L.lirpa_optimize.restype = i
    L.lirpa_timing_begin.argtypes = []
    L.lirpa_timing_begin.restype = i
    L.lirpa_timing_end.argtypes = [ctypes.POINTER(lirpa_kernel_time), i, ctypes.POINTER(i)]
    L.lirpa_timing_end.restype = i
    L.lirpa_last_error.argtypes = []
    L.lirpa_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


class LirpaError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"lirpa error {code}: {msg}")
        self.code = code


def _check(rc):
    if rc != LIRPA_OK:
        raise LirpaError(rc, load().lirpa_last_error().decode())


def _dev(t, dtype=None, what="tensor"):
    """Device pointer of a contiguous CUDA tensor (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{what} must be a CUDA tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{what} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def lirpa_last_error() -> str:
    return load().lirpa_last_error().decode()


def lirpa_timing_begin():
    _check(load().lirpa_timing_begin())


def lirpa_timing_end(max_entries=256):
    """{kernel class: (total_ms, launches)} of the kernels enqueued since lirpa_timing_begin."""
    arr = (lirpa_kernel_time * max_entries)()
    n = ctypes.c_int(0)
    _check(load().lirpa_timing_end(arr, max_entries, ctypes.byref(n)))
    return {arr[i].name.decode(): (arr[i].total_ms, int(arr[i].launches))
            for i in range(min(n.value, max_entries))}


def lirpa_net_create(layers):
    """layers: list of dicts with the layer fields and device tensors ``W``, ``b``."""
    arr = (lirpa_layer * len(layers))()
    for i, t in enumerate(layers):
        arr[i] = lirpa_layer(t["kind"], t["in_c"], t["in_h"], t["in_w"], t["out_c"], t["out_h"],
                             t["out_w"], t.get("k", 0), t.get("stride", 1), t.get("pad", 0),
                             _dev(t["W"], torch.float32, "W"), _dev(t["b"], torch.float32, "b"))
    h = ctypes.c_void_p()
    _check(load().lirpa_net_create(arr, len(layers), ctypes.byref(h)))
    return h


def lirpa_net_destroy(net):
    load().lirpa_net_destroy(net)


def lirpa_net_num_relu(net) -> int:
    return int(load().lirpa_net_num_relu(net))


def lirpa_workspace_bytes(net, S, B_chunk, mode=0) -> int:
    return int(load().lirpa_workspace_bytes(net, S, B_chunk, mode))


def lirpa_bound(net, x0, eps, C, S, B, split, alpha, lb, l_out, u_out, code_out, ws,
                ws_bytes, stream=None):
    _check(load().lirpa_bound(net, _dev(x0, torch.float32, "x0"), float(eps),
                              _dev(C, torch.float32, "C"), int(S), int(B),
                              _dev(split, torch.int8, "split"),
                              _dev(alpha, torch.float32, "alpha"),
                              _dev(lb, torch.float32, "lb"), _dev(l_out, torch.float32, "l_out"),
                              _dev(u_out, torch.float32, "u_out"),
                              _dev(code_out, torch.int8, "code_out"), _dev(ws, None, "ws"),
                              int(ws_bytes), _stream(stream)))


def lirpa_bound_child(net, x0, eps, C, S, B, split, alpha, l_parent, u_parent, lb, l_out, u_out,
                      code_out, ws, ws_bytes, stream=None):
    f32 = torch.float32
    _check(load().lirpa_bound_child(net, _dev(x0, f32, "x0"), float(eps), _dev(C, f32, "C"),
                                    int(S), int(B), _dev(split, torch.int8, "split"),
                                    _dev(alpha, f32, "alpha"), _dev(l_parent, f32, "l_parent"),
                                    _dev(u_parent, f32, "u_parent"), _dev(lb, f32, "lb"),
                                    _dev(l_out, f32, "l_out"), _dev(u_out, f32, "u_out"),
                                    _dev(code_out, torch.int8, "code_out"), _dev(ws, None, "ws"),
                                    int(ws_bytes), _stream(stream)))


def lirpa_bound_noalloc(net, x0, eps, C, S, B, split, alpha, lb, l_out, u_out, code_out,
                        stream=None):
    _check(load().lirpa_bound_noalloc(net, _dev(x0, torch.float32, "x0"), float(eps),
                                      _dev(C, torch.float32, "C"), int(S), int(B),
                                      _dev(split, torch.int8, "split"),
                                      _dev(alpha, torch.float32, "alpha"),
                                      _dev(lb, torch.float32, "lb"),
                                      _dev(l_out, torch.float32, "l_out"),
                                      _dev(u_out, torch.float32, "u_out"),
                                      _dev(code_out, torch.int8, "code_out"), _stream(stream)))


def lirpa_bound_ul(net, x0, eps, C, S, B, split, alpha, lb, ub, l_out, u_out, code_out, ws,
                   ws_bytes, stream=None):
    _check(load().lirpa_bound_ul(net, _dev(x0, torch.float32, "x0"), float(eps),
                                 _dev(C, torch.float32, "C"), int(S), int(B),
                                 _dev(split, torch.int8, "split"),
                                 _dev(alpha, torch.float32, "alpha"),
                                 _dev(lb, torch.float32, "lb"), _dev(ub, torch.float32, "ub"),
                                 _dev(l_out, torch.float32, "l_out"),
                                 _dev(u_out, torch.float32, "u_out"),
                                 _dev(code_out, torch.int8, "code_out"), _dev(ws, None, "ws"),
                                 int(ws_bytes), _stream(stream)))


def lirpa_optimize_ul(net, x0, eps, C, S, B, split, alpha_lo, m_lo, v_lo, alpha_up, m_up, v_up,
                      params, lb_best, ub_best, ws, ws_bytes, stream=None):
    p = params if isinstance(params, lirpa_opt_params) else lirpa_opt_params(**params)
    f32 = torch.float32
    _check(load().lirpa_optimize_ul(net, _dev(x0, f32, "x0"), float(eps), _dev(C, f32, "C"),
                                    int(S), int(B), _dev(split, torch.int8, "split"),
                                    _dev(alpha_lo, f32, "alpha_lo"), _dev(m_lo, f32, "m_lo"),
                                    _dev(v_lo, f32, "v_lo"), _dev(alpha_up, f32, "alpha_up"),
                                    _dev(m_up, f32, "m_up"), _dev(v_up, f32, "v_up"),
                                    ctypes.byref(p), _dev(lb_best, f32, "lb_best"),
                                    _dev(ub_best, f32, "ub_best"), _dev(ws, None, "ws"),
                                    int(ws_bytes), _stream(stream)))


def lirpa_bab_workspace_bytes(net, params) -> int:
    return int(load().lirpa_bab_workspace_bytes(net, ctypes.byref(params)))


def lirpa_bab(net, x0, eps, c, params, ws, ws_bytes, stream=None):
    """Runs the search (the call synchronises the stream); returns the lirpa_bab_result."""
    res = lirpa_bab_result()
    _check(load().lirpa_bab(net, _dev(x0, torch.float32, "x0"), float(eps),
                            _dev(c, torch.float32, "c"), ctypes.byref(params),
                            ctypes.byref(res), _dev(ws, None, "ws"), int(ws_bytes),
                            _stream(stream)))
    return res


def lirpa_bound_grad(net, x0, eps, C, S, B, split, alpha, full, lb, grad, ws, ws_bytes,
                     stream=None):
    _check(load().lirpa_bound_grad(net, _dev(x0, torch.float32, "x0"), float(eps),
                                   _dev(C, torch.float32, "C"), int(S), int(B),
                                   _dev(split, torch.int8, "split"),
                                   _dev(alpha, torch.float32, "alpha"), int(full),
                                   _dev(lb, torch.float32, "lb"),
                                   _dev(grad, torch.float32, "grad"), _dev(ws, None, "ws"),
                                   int(ws_bytes), _stream(stream)))


def lirpa_optimize(net, x0, eps, C, S, B, split, alpha, adam_m, adam_v, params, lb_best,
                   lb_trace, ws, ws_bytes, stream=None):
    p = params if isinstance(params, lirpa_opt_params) else lirpa_opt_params(**params)
    _check(load().lirpa_optimize(net, _dev(x0, torch.float32, "x0"), float(eps),
                                 _dev(C, torch.float32, "C"), int(S), int(B),
                                 _dev(split, torch.int8, "split"),
                                 _dev(alpha, torch.float32, "alpha"),
                                 _dev(adam_m, torch.float32, "adam_m"),
                                 _dev(adam_v, torch.float32, "adam_v"), ctypes.byref(p),
                                 _dev(lb_best, torch.float32, "lb_best"),
                                 _dev(lb_trace, torch.float32, "lb_trace"), _dev(ws, None, "ws"),
                                 int(ws_bytes), _stream(stream)))


class Network:
    """Device copy of a network (layer dicts with numpy W, b), its handle and a workspace."""

    def __init__(self, layers, device="cuda"):
        self.layers = []
        for t in layers:
            d = dict(t)
            d["W"] = torch.as_tensor(np.ascontiguousarray(t["W"], dtype=np.float32)).to(device)
            d["b"] = torch.as_tensor(np.ascontiguousarray(t["b"], dtype=np.float32)).to(device)
            self.layers.append(d)
        self.device = device
        self.handle = lirpa_net_create(self.layers)
        self.n_relu = lirpa_net_num_relu(self.handle)
        self._ws = None

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and _lib is not None:
            lirpa_net_destroy(h)
            self.handle = None

    def workspace(self, S, B, mode=0, max_bytes=None):
        """A workspace for up to B sub-domains per chunk (capped at max_bytes), reused."""
        need = lirpa_workspace_bytes(self.handle, S, B, mode)
        if max_bytes is not None and need > max_bytes:
            need = max_bytes
        if self._ws is None or self._ws.numel() < need:
            self._ws = None
            self._ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        return self._ws, need

    def bound(self, x0, eps, C, split=None, alpha=None, B=None, want_lu=False, ws=None,
              ws_bytes=None, max_ws_bytes=16 << 30, want_codes=False):
        S = C.shape[0]
        if B is None:
            B = split.shape[0] if split is not None else (alpha.shape[0] if alpha is not None
                                                            else 1)
        lb = torch.empty((B, S), dtype=torch.float32, device=self.device)
        l = u = code = None
        if want_lu:
            l = torch.empty((B, self.n_relu), dtype=torch.float32, device=self.device)
            u = torch.empty_like(l)
        if want_codes:
            code = torch.empty((B, self.n_relu), dtype=torch.int8, device=self.device)
        if ws is None:
            ws, ws_bytes = self.workspace(S, B, 0, max_ws_bytes)
        lirpa_bound(self.handle, x0, eps, C, S, B, split, alpha, lb, l, u, code, ws, ws_bytes)
        out = (lb, l, u) if want_lu else (lb,)
        if want_codes:
            out = out + (code,)
        return out if len(out) > 1 else lb

    def bound_child(self, x0, eps, C, split, alpha, l_parent, u_parent, max_ws_bytes=16 << 30):
        """(lb, l, u, codes) with every layer's bounds intersected with the parent's."""
        S, B = C.shape[0], l_parent.shape[0]
        lb = torch.empty((B, S), dtype=torch.float32, device=self.device)
        l = torch.empty((B, self.n_relu), dtype=torch.float32, device=self.device)
        u = torch.empty_like(l)
        code = torch.empty((B, self.n_relu), dtype=torch.int8, device=self.device)
        ws, ws_bytes = self.workspace(S, B, 0, max_ws_bytes)
        lirpa_bound_child(self.handle, x0, eps, C, S, B, split, alpha, l_parent, u_parent, lb, l,
                          u, code, ws, ws_bytes)
        return lb, l, u, code

    def bound_ul(self, x0, eps, C, split=None, alpha=None, B=None, max_ws_bytes=16 << 30):
        """(lb, ub) [B, S] of the spec rows: Eq. 8's lower and upper bounds in one call."""
        S = C.shape[0]
        if B is None:
            B = split.shape[0] if split is not None else (alpha.shape[0] if alpha is not None
                                                            else 1)
        lb = torch.empty((B, S), dtype=torch.float32, device=self.device)
        ub = torch.empty_like(lb)
        ws, ws_bytes = self.workspace(S, B, 2, max_ws_bytes)
        lirpa_bound_ul(self.handle, x0, eps, C, S, B, split, alpha, lb, ub, None, None, None, ws,
                       ws_bytes)
        return lb, ub

    def optimize_ul(self, x0, eps, C, split, B=None, steps=20, lr=0.1, beta1=0.9, beta2=0.999,
                    eps_adam=1e-8, max_ws_bytes=16 << 30, state=None):
        """Optimised (lb_best, ub_best) from a fresh start (state None) or from the state dict a
        previous call returned (alpha, m, v of both sides, t0); returns (lb, ub, state)."""
        S = C.shape[0]
        B = split.shape[0] if B is None else B
        fresh = state is None
        if fresh:
            state = {k: torch.empty((B, self.n_relu), dtype=torch.float32, device=self.device)
                     for k in ("alpha_lo", "m_lo", "v_lo", "alpha_up", "m_up", "v_up")}
            state["t0"] = 0
        lb = torch.empty((B, S), dtype=torch.float32, device=self.device)
        ub = torch.empty_like(lb)
        ws, ws_bytes = self.workspace(S, B, 3, max_ws_bytes)
        lirpa_optimize_ul(self.handle, x0, eps, C, S, B, split, state["alpha_lo"], state["m_lo"],
                          state["v_lo"], state["alpha_up"], state["m_up"], state["v_up"],
                          lirpa_opt_params(steps, lr, beta1, beta2, eps_adam, state["t0"],
                                           int(fresh)), lb, ub, ws, ws_bytes)
        state = dict(state, t0=state["t0"] + steps)
        return lb, ub, state

    def bab(self, x0, eps, c, batch=64, max_domains=4000, max_iters=30, root_steps=0, steps=0,
            lr=0.1, beta1=0.9, beta2=0.999, eps_adam=1e-8):
        """Branch and bound on c^T f(x) >= 0; returns a dict of the lirpa_bab_result fields."""
        p = lirpa_bab_params(batch, max_domains, max_iters, root_steps, steps, lr, beta1, beta2,
                             eps_adam)
        need = lirpa_bab_workspace_bytes(self.handle, p)
        ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        r = lirpa_bab(self.handle, x0, eps, c, p, ws, need)
        return {k: getattr(r, k) for k, _ in lirpa_bab_result._fields_}

    def bound_grad(self, x0, eps, C, split, alpha, full=True, max_ws_bytes=16 << 30):
        S, B = C.shape[0], alpha.shape[0]
        lb = torch.empty((B, S), dtype=torch.float32, device=self.device)
        grad = torch.empty((B, self.n_relu), dtype=torch.float32, device=self.device)
        ws, ws_bytes = self.workspace(S, B, 1, max_ws_bytes)
        lirpa_bound_grad(self.handle, x0, eps, C, S, B, split, alpha, int(full), lb, grad, ws,
                         ws_bytes)
        return lb, grad

    def optimize(self, x0, eps, C, split, alpha, adam_m=None, adam_v=None, steps=20, lr=0.1,
                 beta1=0.9, beta2=0.999, eps_adam=1e-8, t0=0, trace=False, fresh=False,
                 max_ws_bytes=16 << 30):
        """In place on alpha (and adam_m, adam_v); returns lb_best (and the lb trace)."""
        S, B = C.shape[0], alpha.shape[0]
        if adam_m is None:
            adam_m = torch.zeros_like(alpha)
        if adam_v is None:
            adam_v = torch.zeros_like(alpha)
        best = torch.empty((B, S), dtype=torch.float32, device=self.device)
        tr = torch.empty((steps + 1, B, S), dtype=torch.float32, device=self.device) \
            if trace else None
        ws, ws_bytes = self.workspace(S, B, 1, max_ws_bytes)
        lirpa_optimize(self.handle, x0, eps, C, S, B, split, alpha, adam_m, adam_v,
                       lirpa_opt_params(steps, lr, beta1, beta2, eps_adam, t0, int(fresh)),
                       best, tr, ws,
                       ws_bytes)
        return (best, tr) if trace else best
