"""The C-ABI library: it loads, exports every declared entry point, and its
host-side argument checks return the documented codes.  No GPU needed: the
calls below are rejected on the host before any device work."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "chaos.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(chaos_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_1506_09067_amd import chaos
    if not os.path.exists(chaos.LIB_PATH):
        from paper_1506_09067_amd import build
        build.build_library()
    return chaos.lib()


def test_header_declares_the_boundary():
    names = _declared()
    for required in ("chaos_create_net", "chaos_forward_backward", "chaos_apply_update",
                     "chaos_train_epoch", "chaos_evaluate", "chaos_destroy_net",
                     "chaos_get_params", "chaos_set_params", "chaos_num_params",
                     "chaos_max_workers", "chaos_last_error"):
        assert required in names


def test_library_exports_every_declared_symbol(lib):
    for name in _declared():
        assert hasattr(lib, name), name


def _create(lib, layers, n_params, params=None, in_hw=29):
    from paper_1506_09067_amd import chaos
    arr = (chaos.chaos_layer * len(layers))(*[chaos.chaos_layer(*l) for l in layers])
    p = np.zeros(max(n_params, 1), dtype=np.float32) if params is None else params
    h = ctypes.c_void_p()
    rc = lib.chaos_create_net(in_hw, in_hw, arr, len(layers), p.ctypes.data_as(ctypes.c_void_p),
                              n_params, ctypes.byref(h))
    return rc, h


@pytest.mark.parametrize("layers,n_params,code", [
    ([(1, 2, 30)], 0, -2),                     # kernel larger than the 29x29 map
    ([(1, 5, 4), (2, 0, 3)], 85, -2),          # 26 not divisible by 3
    ([(9, 5, 4)], 85, -1),                     # unknown kind
    ([(3, 0, 0)], 0, -1),                      # FC without neurons
    ([(1, 0, 4)], 0, -1),                      # conv without maps
    ([(1, 5, 4), (2, 0, 2), (3, 10, 0)], 123, -2),  # n_params mismatch
    ([(1, 1 << 22, 1)], 0, -5),                # 2^22 maps of 29x29: outputs beyond 2^31
    ([(1, 1 << 20, 1), (3, 4, 0)], 0, -5),     # FC over 2^20 x 841 inputs
])
def test_create_rejects_bad_architectures(lib, layers, n_params, code):
    rc, h = _create(lib, layers, n_params)
    assert rc == code
    assert not h.value
    assert lib.chaos_last_error()  # a message is set


def test_null_and_range_arguments(lib):
    from paper_1506_09067_amd import chaos
    P = ctypes.c_void_p
    assert lib.chaos_create_net(29, 29, None, 1, None, 0, ctypes.byref(P())) == -1
    arr = (chaos.chaos_layer * 1)(chaos.chaos_layer(3, 10, 0))
    assert lib.chaos_create_net(29, 29, arr, 1, None, 8420, None) == -1
    assert lib.chaos_create_net(29, 29, arr, 0, None, 8420, ctypes.byref(P())) == -1
    assert lib.chaos_create_net(29, 29, arr, 99, None, 8420, ctypes.byref(P())) == -1
    assert lib.chaos_create_net(0, 29, arr, 1, None, 8420, ctypes.byref(P())) == -1
    # calls on a NULL net
    assert lib.chaos_num_params(None) == -1
    assert lib.chaos_max_workers(None) == -1
    assert lib.chaos_default_workers(None) == -1
    assert lib.chaos_train_epoch(None, None, None, 0, 0.0, 0, 0, None, None) == -1
    assert lib.chaos_forward_backward(None, None, None, 0, None, None, None, None, None) == -1
    assert lib.chaos_evaluate(None, None, None, 0, None, None, None) == -1
    assert lib.chaos_apply_update(None, None, 0.0, None) == -1
    assert lib.chaos_train_session(None, None, None, 0, None, None, 0, 1, 0.0, 1.0, 0, 0, None,
                                   None, None) == -1
    assert lib.chaos_set_push_delay(None, 2) == -1
    assert lib.chaos_destroy_net(None) == 0
