"""Thin ctypes binding of libchaos.so (include/chaos.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  Tensors are torch CUDA tensors (PyTorch provides device memory and
streams); calls are asynchronous on the current torch stream.

The binding fails loudly when libchaos.so has not been built: there is no
CPU fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch  # loads the HIP runtime that libchaos.so binds to

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libchaos.so")

CONV, MAXPOOL, FC = 1, 2, 3
SEQUENTIAL, HOGWILD_ATOMIC, HOGWILD_RACY = 0, 1, 2

OK, EINVAL, ESHAPE, ENOMEM, EDEVICE, EUNSUPPORTED = 0, -1, -2, -3, -4, -5
_CODES = {EINVAL: "EINVAL", ESHAPE: "ESHAPE", ENOMEM: "ENOMEM", EDEVICE: "EDEVICE",
          EUNSUPPORTED: "EUNSUPPORTED"}


class ChaosError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{_CODES.get(code, code)}: {msg}")
        self.code = code


class chaos_layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("maps", ctypes.c_int32), ("kernel", ctypes.c_int32)]


_lib = None


def lib():
    """Load libchaos.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it first "
                               "(python -c 'import __graft_entry__ as g; g.build()')")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        sig = {
            "chaos_create_net": ([i32, i32, P, i32, P, i64, P], ctypes.c_int),
            "chaos_destroy_net": ([P], ctypes.c_int),
            "chaos_num_params": ([P], ctypes.c_int64),
            "chaos_num_outputs": ([P], ctypes.c_int32),
            "chaos_get_params": ([P, P, P], ctypes.c_int),
            "chaos_set_params": ([P, P, P], ctypes.c_int),
            "chaos_forward_backward": ([P, P, P, i64, P, P, P, P, P], ctypes.c_int),
            "chaos_forward_backward_noalloc": ([P, P, P, i64, P, P, P, P, P], ctypes.c_int),
            "chaos_apply_update": ([P, P, f32, P], ctypes.c_int),
            "chaos_train_epoch": ([P, P, P, i64, f32, i32, i32, P, P], ctypes.c_int),
            "chaos_evaluate": ([P, P, P, i64, P, P, P], ctypes.c_int),
            "chaos_train_session": ([P, P, P, i64, P, P, i64, i32, f32, f32, i32, i32, P, P, P],
                                    ctypes.c_int),
            "chaos_max_workers": ([P], ctypes.c_int32),
            "chaos_default_workers": ([P], ctypes.c_int32),
            "chaos_worker_limit": ([P], ctypes.c_int32),
            "chaos_set_claim_counter": ([P, P], ctypes.c_int),
            "chaos_set_push_delay": ([P, i32], ctypes.c_int),
            "chaos_set_replicas": ([P, i32, i32], ctypes.c_int),
            "chaos_last_error": ([], ctypes.c_char_p),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def last_error() -> str:
    return lib().chaos_last_error().decode()


def _check(rc):
    if rc != OK:
        raise ChaosError(rc, last_error())
    return rc


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, dtype, name, numel=None, optional=False):
    """Device pointer of a contiguous CUDA tensor (or None if optional and absent)."""
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs {numel}")
    return ctypes.c_void_p(t.data_ptr())


class Net:
    """A CHAOS net: architecture + shared fp32 weights on the current device."""

    def __init__(self, layers, init_params, in_h: int = 29, in_w: int = 29):
        import numpy as np
        arr = (chaos_layer * len(layers))(*[chaos_layer(*map(int, l)) for l in layers])
        p = np.ascontiguousarray(np.asarray(init_params, dtype=np.float32).reshape(-1))
        h = ctypes.c_void_p()
        _check(lib().chaos_create_net(in_h, in_w, arr, len(layers),
                                      p.ctypes.data_as(ctypes.c_void_p), p.size,
                                      ctypes.byref(h)))
        self._h = h
        self.layers = [tuple(l) for l in layers]
        self.n_params = int(lib().chaos_num_params(h))
        self.n_out = int(lib().chaos_num_outputs(h))
        self.in_size = in_h * in_w

    def close(self):
        if getattr(self, "_h", None):
            lib().chaos_destroy_net(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    @property
    def max_workers(self) -> int:
        return int(lib().chaos_max_workers(self._h))

    @property
    def default_workers(self) -> int:
        """Workers of a Hogwild epoch called with workers=0 (one per compute unit)."""
        return int(lib().chaos_default_workers(self._h))

    @property
    def worker_limit(self) -> int:
        return int(lib().chaos_worker_limit(self._h))

    def get_params(self, out=None):
        if out is None:
            out = torch.empty(self.n_params, dtype=torch.float32, device="cuda")
        _check(lib().chaos_get_params(self._h, _dev(out, torch.float32, "out", self.n_params),
                                      _stream()))
        return out

    def set_params(self, src):
        _check(lib().chaos_set_params(self._h, _dev(src, torch.float32, "src", self.n_params),
                                      _stream()))

    def apply_update(self, grad, lr: float):
        _check(lib().chaos_apply_update(self._h, _dev(grad, torch.float32, "grad", self.n_params),
                                        float(lr), _stream()))

    def _xy(self, x, labels):
        n = labels.numel()
        return (_dev(x, torch.float32, "x", n * self.in_size),
                _dev(labels, torch.int32, "labels", n), n)

    def forward_backward(self, x, labels, out=None, loss=None, grad_sum=None, grad_each=None):
        px, py, n = self._xy(x, labels)
        _check(lib().chaos_forward_backward(
            self._h, px, py, n,
            _dev(out, torch.float32, "out", n * self.n_out, True),
            _dev(loss, torch.float32, "loss", n, True),
            _dev(grad_sum, torch.float32, "grad_sum", self.n_params, True),
            _dev(grad_each, torch.float32, "grad_each", n * self.n_params, True),
            _stream()))

    def forward_backward_noalloc(self, x, labels, out=None, loss=None, grad_sum=None,
                                 grad_each=None):
        """chaos_forward_backward_noalloc: as forward_backward, allocating no
        device memory (partial sums in the library's fixed scratch array)."""
        px, py, n = self._xy(x, labels)
        _check(lib().chaos_forward_backward_noalloc(
            self._h, px, py, n,
            _dev(out, torch.float32, "out", n * self.n_out, True),
            _dev(loss, torch.float32, "loss", n, True),
            _dev(grad_sum, torch.float32, "grad_sum", self.n_params, True),
            _dev(grad_each, torch.float32, "grad_each", n * self.n_params, True),
            _stream()))

    def train_epoch(self, x, labels, lr: float, mode: int = HOGWILD_ATOMIC, workers: int = 0,
                    loss=None):
        px, py, n = self._xy(x, labels)
        _check(lib().chaos_train_epoch(self._h, px, py, n, float(lr), int(mode), int(workers),
                                       _dev(loss, torch.float32, "loss", n, True), _stream()))

    def train_session(self, x, labels, x_test, labels_test, epochs: int, lr0: float,
                      decay: float = 1.0, mode: int = HOGWILD_ATOMIC, workers: int = 0,
                      checkpoints=None):
        """Training + Validation + Testing per epoch; returns stats [epochs][5] on
        the device: mean training loss, wrong on the training set, wrong on the
        test set, mean test loss, divergence flag (1.0 when the epoch's loss is
        above the loss at the starting weights).  checkpoints: optional float32 CUDA tensor
        [epochs][n_params] that receives the weights after each epoch's
        Training (canonical layout)."""
        px, py, n = self._xy(x, labels)
        pxt, pyt, nt = self._xy(x_test, labels_test)
        stats = torch.empty(max(epochs, 1), 5, dtype=torch.float32, device="cuda")
        ck = _dev(checkpoints, torch.float32, "checkpoints", max(epochs, 0) * self.n_params, True)
        _check(lib().chaos_train_session(self._h, px, py, n, pxt, pyt, nt, int(epochs),
                                         float(lr0), float(decay), int(mode), int(workers),
                                         ctypes.c_void_p(stats.data_ptr()), ck, _stream()))
        return stats[:epochs]

    def evaluate(self, x, labels, out=None, n_wrong=None):
        px, py, n = self._xy(x, labels)
        if n_wrong is None:
            n_wrong = torch.empty(1, dtype=torch.int32, device="cuda")
        _check(lib().chaos_evaluate(self._h, px, py, n,
                                    _dev(out, torch.float32, "out", n * self.n_out, True),
                                    _dev(n_wrong, torch.int32, "n_wrong", 1), _stream()))
        return n_wrong

    def set_claim_counter(self, claims):
        _check(lib().chaos_set_claim_counter(
            self._h, _dev(claims, torch.int32, "claims", optional=True)))

    def set_replicas(self, r: int, m: int = 4):
        """Atomic Hogwild workers read r replicas of the weights, each copied
        from the shared weights after every m-th sample completed on it
        (r = 1: off)."""
        _check(lib().chaos_set_replicas(self._h, int(r), int(m)))

    def set_push_delay(self, k: int):
        """Samples between a worker's pushes in atomic Hogwild epochs (1 = per layer)."""
        _check(lib().chaos_set_push_delay(self._h, int(k)))
