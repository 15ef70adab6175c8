"""ctypes wrapper of the CHAOS oracle -- TEST INFRASTRUCTURE ONLY.

Only tests/, the smoke check and the benchmark's CPU-baseline leg may import
this module.  It never imports the HIP library or its binding; the two sides
meet only through the seeded inputs of paper_1506_09067_amd.workloads.

Every function mirrors one in chaos_oracle.c (see the header there for the
passages of the paper each step follows).  Arrays are numpy; parameters are
converted to double before the call.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "chaos_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

CONV, MAXPOOL, FC = 1, 2, 3
ACT_TANH, ACT_IDENTITY = 0, 1


def build(force: bool = False) -> str:
    """Compile chaos_oracle.c into liboracle.so with gcc (plain C, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
                        "-fno-fast-math", _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        i32, i64, f64 = ctypes.c_int, ctypes.c_longlong, ctypes.c_double
        P = ctypes.c_void_p
        L.orc_shape.argtypes = [i32, i32, P, i32, P, P]
        L.orc_activation.argtypes = [i32, f64, P, P]
        L.orc_activation.restype = None
        L.orc_conv_forward.argtypes = [P, i32, i32, i32, P, P, i32, i32, P]
        L.orc_conv_forward.restype = None
        L.orc_conv_wgrad.argtypes = [P, i32, i32, i32, P, i32, i32, P, P]
        L.orc_conv_wgrad.restype = None
        L.orc_conv_backdata.argtypes = [P, i32, i32, P, i32, i32, i32, P]
        L.orc_conv_backdata.restype = None
        L.orc_forward_backward.argtypes = [i32, i32, P, i32, i32, P, i64, P, i32, P, P, P, P]
        L.orc_train_sequential.argtypes = [i32, i32, P, i32, i32, P, i64, i32, P, P, i64, f64, P, P]
        L.orc_grad_sum.argtypes = [i32, i32, P, i32, i32, P, i64, P, P, i64, P, P, P]
        L.orc_evaluate.argtypes = [i32, i32, P, i32, i32, P, i64, P, P, i64, P, P]
        for name in ("orc_shape", "orc_forward_backward", "orc_train_sequential",
                     "orc_grad_sum", "orc_evaluate"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _layers(layers):
    return np.ascontiguousarray(np.array(layers, dtype=np.int32).reshape(-1))


def _check(rc, what):
    if rc != 0:
        raise OracleError(f"{what} failed with status {rc}")


def shape(layers, in_h=29, in_w=29):
    """Per-layer (cin, hin, win, cout, hout, wout, n_weights_incl_bias), n_params."""
    ly = _layers(layers)
    n = len(ly) // 3
    dims = np.zeros((n, 7), dtype=np.int64)
    npar = ctypes.c_longlong(0)
    rc = lib().orc_shape(in_h, in_w, _ptr(ly), n, _ptr(dims), ctypes.byref(npar))
    return rc, dims, npar.value


def n_params(layers, in_h=29, in_w=29):
    rc, _, n = shape(layers, in_h, in_w)
    _check(rc, "shape")
    return n


def activation(z, act=ACT_TANH):
    f, df = ctypes.c_double(), ctypes.c_double()
    lib().orc_activation(act, float(z), ctypes.byref(f), ctypes.byref(df))
    return f.value, df.value


def conv_forward(inp, w, b, K):
    inp = np.ascontiguousarray(inp, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    C, H, W = inp.shape
    O = w.shape[0]
    out = np.zeros((O, H - K + 1, W - K + 1))
    bb = None if b is None else np.ascontiguousarray(b, dtype=np.float64)
    lib().orc_conv_forward(_ptr(inp), C, H, W, _ptr(w), _ptr(bb), O, K, _ptr(out))
    return out


def conv_wgrad(inp, d, K):
    inp = np.ascontiguousarray(inp, dtype=np.float64)
    d = np.ascontiguousarray(d, dtype=np.float64)
    C, H, W = inp.shape
    O = d.shape[0]
    gw = np.zeros((O, C, K, K))
    gb = np.zeros(O)
    lib().orc_conv_wgrad(_ptr(inp), C, H, W, _ptr(d), O, K, _ptr(gw), _ptr(gb))
    return gw, gb


def conv_backdata(d, w, H, W):
    d = np.ascontiguousarray(d, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    O, C, K, _ = w.shape
    e = np.zeros((C, H, W))
    lib().orc_conv_backdata(_ptr(d), O, K, _ptr(w), C, H, W, _ptr(e))
    return e


def _params(p):
    return np.ascontiguousarray(p, dtype=np.float64)


def forward_backward(layers, params, x, label, act=ACT_TANH, in_h=29, in_w=29, grad=True):
    """One sample at fixed weights -> dict(out, loss, grad, min_gap)."""
    ly = _layers(layers)
    p = _params(params)
    x = np.ascontiguousarray(x, dtype=np.float32).reshape(-1)
    rc, dims, npar = shape(layers, in_h, in_w)
    _check(rc, "shape")
    n_out = int(dims[-1, 3] * dims[-1, 4] * dims[-1, 5])
    out = np.zeros(n_out)
    loss = ctypes.c_double()
    gap = ctypes.c_double()
    g = np.zeros(npar) if grad else None
    rc = lib().orc_forward_backward(in_h, in_w, _ptr(ly), len(ly) // 3, act, _ptr(p), npar,
                                    _ptr(x), int(label), _ptr(out), ctypes.byref(loss),
                                    _ptr(g), ctypes.byref(gap))
    _check(rc, "forward_backward")
    return {"out": out, "loss": loss.value, "grad": g, "min_gap": gap.value}


def train_sequential(layers, params, x, labels, lr, act=ACT_TANH, store_f32=True,
                     in_h=29, in_w=29, with_gaps=False):
    """Per-sample SGD in index order -> (params after, per-sample losses[, gaps])."""
    ly = _layers(layers)
    p = _params(params).copy()
    x = np.ascontiguousarray(x, dtype=np.float32)
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    n = len(labels)
    losses = np.zeros(n)
    gaps = np.zeros(n)
    rc = lib().orc_train_sequential(in_h, in_w, _ptr(ly), len(ly) // 3, act, _ptr(p), p.size,
                                    int(store_f32), _ptr(x), _ptr(labels), n, float(lr),
                                    _ptr(losses), _ptr(gaps))
    _check(rc, "train_sequential")
    return (p, losses, gaps) if with_gaps else (p, losses)


def grad_sum(layers, params, x, labels, act=ACT_TANH, in_h=29, in_w=29, with_gaps=False):
    """sum_i grad E_i(W) at fixed W (double) -> (G, per-sample losses[, per-sample
    smallest relative max-pool gaps])."""
    ly = _layers(layers)
    p = _params(params)
    x = np.ascontiguousarray(x, dtype=np.float32)
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    n = len(labels)
    g = np.zeros(p.size)
    losses = np.zeros(n)
    gaps = np.zeros(n) if with_gaps else None
    rc = lib().orc_grad_sum(in_h, in_w, _ptr(ly), len(ly) // 3, act, _ptr(p), p.size, _ptr(x),
                            _ptr(labels), n, _ptr(g), _ptr(losses), _ptr(gaps))
    _check(rc, "grad_sum")
    return (g, losses, gaps) if with_gaps else (g, losses)


def evaluate(layers, params, x, labels, act=ACT_TANH, in_h=29, in_w=29):
    """Forward only -> (outputs [n][n_out], number of wrong predictions)."""
    ly = _layers(layers)
    p = _params(params)
    x = np.ascontiguousarray(x, dtype=np.float32)
    labels = np.ascontiguousarray(labels, dtype=np.int32)
    n = len(labels)
    rc, dims, npar = shape(layers, in_h, in_w)
    _check(rc, "shape")
    n_out = int(dims[-1, 3] * dims[-1, 4] * dims[-1, 5])
    out = np.zeros((n, n_out))
    wrong = ctypes.c_longlong()
    rc = lib().orc_evaluate(in_h, in_w, _ptr(ly), len(ly) // 3, act, _ptr(p), p.size, _ptr(x),
                            _ptr(labels), n, _ptr(out), ctypes.byref(wrong))
    _check(rc, "evaluate")
    return out, wrong.value
