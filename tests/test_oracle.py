"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: values
printed in Table I, closed forms, a hand-worked example, library routines
(scipy, torch CPU autograd), finite differences, and special cases that reduce
to a textbook result.  No GPU needed.
"""
import math
import os

import numpy as np
import pytest

from oracle import oracle as orc
from paper_1506_09067_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
A, B = 1.7159, 2.0 / 3.0


# --------------------------------------------------------------------------
# Table I: maps, map sizes, neurons and weight counts of the three nets.
def _table1():
    rows = {}
    with open(os.path.join(GOLDEN, "table1_architectures.txt")) as f:
        for line in f:
            line = line.split("#")[0].split()
            if not line:
                continue
            net, typ, maps, mh, mw, neurons, k, weights = line
            rows.setdefault(net, []).append((typ, int(maps), int(mh), int(mw), int(neurons),
                                             int(k), int(weights)))
    return rows


@pytest.mark.parametrize("net", ["small", "medium", "large_table1"])
def test_table1_shapes_and_weight_counts(net):
    table = _table1()[net]
    rc, dims, npar = orc.shape(wl.NETS[net])
    assert rc == 0
    assert table[0][1:5] == (1, 29, 29, 841)
    for (typ, maps, mh, mw, neurons, k, weights), d, layer in zip(table[1:], dims, wl.NETS[net]):
        cin, hin, win, cout, hout, wout, nw = (int(v) for v in d)
        if typ in ("full", "output"):
            assert layer[0] == orc.FC and cout == maps == neurons
        else:
            assert cout == maps and (hout, wout) == (mh, mw)
            assert cout * hout * wout == neurons
            assert layer[2] == k
        assert nw == weights
    assert npar == sum(r[6] for r in table)


def test_param_totals_of_all_nets():
    # Table I sums (small, medium, large) and the conv60-k3 large net.
    assert orc.n_params(wl.NETS["small"]) == 85 + 1260 + 4550 + 510 == 6405
    assert orc.n_params(wl.NETS["medium"]) == 340 + 20040 + 54150 + 1510 == 76040
    assert orc.n_params(wl.NETS["large_table1"]) == 340 + 30060 + 216100 + 135150 + 1510
    # conv20 k4 (340) + conv60 k3 on 20 maps (60*(180+1)) + conv100 k6 on 60 maps
    # + FC 900->150 + FC 150->10
    assert orc.n_params(wl.NETS["large"]) == 340 + 10860 + 216100 + 135150 + 1510 == 363960
    for name in wl.NETS:  # the input generator's bookkeeping agrees
        assert wl.init_params(wl.NETS[name]).size == orc.n_params(wl.NETS[name])


@pytest.mark.parametrize("layers,code", [
    ([(orc.CONV, 2, 30)], -2),                    # kernel larger than the map
    ([(orc.CONV, 2, 4), (orc.MAXPOOL, 0, 3)], -2),  # 26 not divisible by 3
    ([(7, 2, 4)], -1),                            # unknown kind
    ([(orc.FC, 0, 0)], -1),                       # empty FC
])
def test_shape_errors(layers, code):
    rc, _, _ = orc.shape(layers)
    assert rc == code


# --------------------------------------------------------------------------
# Activation: scaled tanh f(z) = A tanh(B z), chosen so that f(+-1) ~= +-1.
def test_activation_closed_form():
    f1, _ = orc.activation(1.0)
    assert abs(f1 - 1.0) < 1e-5            # LeCun's constants make f(1) ~= 1
    f0, d0 = orc.activation(0.0)
    assert f0 == 0.0
    assert abs(d0 - 1.1439333333333333) < 1e-12   # A*B
    fm, _ = orc.activation(-1.0)
    assert fm == -f1                       # odd
    big, dbig = orc.activation(40.0)
    assert abs(big - A) < 1e-12 and dbig < 1e-20  # saturates at A
    for z in (-2.3, -0.4, 0.0, 0.7, 1.0, 3.1):    # f' against central differences of f
        h = 1e-6
        fd = (orc.activation(z + h)[0] - orc.activation(z - h)[0]) / (2 * h)
        assert abs(orc.activation(z)[1] - fd) < 1e-8
    f, d = orc.activation(0.37, orc.ACT_IDENTITY)
    assert (f, d) == (0.37, 1.0)


# --------------------------------------------------------------------------
# Hand-worked 3x3 example: input [[1,2,3],[4,5,6],[7,8,9]], kernel [[1,2],[3,4]].
IN3 = np.arange(1, 10, dtype=np.float64).reshape(1, 3, 3)
K2 = np.array([[1, 2], [3, 4]], dtype=np.float64).reshape(1, 1, 2, 2)


def test_hand_worked_conv_forward_is_cross_correlation():
    out = orc.conv_forward(IN3, K2, np.zeros(1), 2)
    # 1*1+2*2+3*4+4*5 = 37 ... ; a flipped kernel would give 23 at (0,0)
    assert out[0].tolist() == [[37, 47], [67, 77]]
    out_b = orc.conv_forward(IN3, K2, np.array([0.5]), 2)
    assert out_b[0].tolist() == [[37.5, 47.5], [67.5, 77.5]]


def test_hand_worked_conv_gradients():
    d = np.array([[[1, 0], [0, 0]]], dtype=np.float64)
    gw, gb = orc.conv_wgrad(IN3, d, 2)
    assert gw[0, 0].tolist() == [[1, 2], [4, 5]] and gb.tolist() == [1]
    e = orc.conv_backdata(d, K2, 3, 3)
    assert e[0].tolist() == [[1, 2, 0], [3, 4, 0], [0, 0, 0]]
    d = np.array([[[0, 0], [0, 1]]], dtype=np.float64)
    gw, gb = orc.conv_wgrad(IN3, d, 2)
    assert gw[0, 0].tolist() == [[5, 6], [8, 9]] and gb.tolist() == [1]
    e = orc.conv_backdata(d, K2, 3, 3)
    assert e[0].tolist() == [[0, 0, 0], [0, 1, 2], [0, 3, 4]]


# --------------------------------------------------------------------------
# Library routines: scipy's 2-D correlation / convolution, multi-map.
def test_conv_primitives_against_scipy():
    from scipy.signal import convolve2d, correlate2d
    rng = np.random.default_rng(11)
    C, H, W, O, K = 3, 9, 8, 4, 3
    x = rng.standard_normal((C, H, W))
    w = rng.standard_normal((O, C, K, K))
    b = rng.standard_normal(O)
    d = rng.standard_normal((O, H - K + 1, W - K + 1))
    out = orc.conv_forward(x, w, b, K)
    ref = np.stack([b[o] + sum(correlate2d(x[c], w[o, c], "valid") for c in range(C))
                    for o in range(O)])
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
    gw, gb = orc.conv_wgrad(x, d, K)
    ref_gw = np.stack([[correlate2d(x[c], d[o], "valid") for c in range(C)] for o in range(O)])
    np.testing.assert_allclose(gw, ref_gw, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(gb, d.sum(axis=(1, 2)), rtol=1e-12)
    e = orc.conv_backdata(d, w, H, W)
    ref_e = np.stack([sum(convolve2d(d[o], w[o, c], "full") for o in range(O)) for c in range(C)])
    np.testing.assert_allclose(e, ref_e, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------
# Whole-net back-propagation.
TINY_NETS = {
    "conv_pool_fc": (8, [(orc.CONV, 2, 3), (orc.MAXPOOL, 0, 2), (orc.FC, 4, 0)]),
    "two_convs": (8, [(orc.CONV, 2, 2), (orc.CONV, 3, 3), (orc.FC, 3, 0)]),
    "pool_first": (6, [(orc.MAXPOOL, 0, 2), (orc.CONV, 2, 2), (orc.FC, 5, 0)]),
    "pool_k1": (7, [(orc.CONV, 2, 2), (orc.MAXPOOL, 0, 1), (orc.CONV, 1, 2), (orc.FC, 3, 0)]),
    "fc_fc": (5, [(orc.FC, 6, 0), (orc.FC, 4, 0)]),
    "conv_conv_pool": (9, [(orc.CONV, 2, 2), (orc.CONV, 2, 3), (orc.MAXPOOL, 0, 3), (orc.FC, 3, 0)]),
}


def _rand_params(layers, hw, rng, scale=0.6):
    n = orc.n_params(layers, hw, hw)
    return rng.uniform(-scale, scale, n)


@pytest.mark.parametrize("name", sorted(TINY_NETS))
@pytest.mark.parametrize("act", [orc.ACT_TANH, orc.ACT_IDENTITY])
def test_gradient_matches_finite_differences(name, act):
    hw, layers = TINY_NETS[name]
    rng = np.random.default_rng(sum(map(ord, name)) * 7 + act)
    params = _rand_params(layers, hw, rng)
    x = rng.uniform(0.05, 1.0, hw * hw).astype(np.float32)  # no zeros: pooling ties impossible
    n_out = orc.shape(layers, hw, hw)[1][-1, 3]
    label = int(rng.integers(0, n_out))
    res = orc.forward_backward(layers, params, x, label, act=act, in_h=hw, in_w=hw)
    g = res["grad"]
    h = 1e-6
    fd = np.zeros_like(params)
    for i in range(params.size):
        p1, p2 = params.copy(), params.copy()
        p1[i] += h
        p2[i] -= h
        e1 = orc.forward_backward(layers, p1, x, label, act=act, in_h=hw, in_w=hw, grad=False)
        e2 = orc.forward_backward(layers, p2, x, label, act=act, in_h=hw, in_w=hw, grad=False)
        fd[i] = (e1["loss"] - e2["loss"]) / (2 * h)
    assert np.max(np.abs(g - fd)) <= 1e-6 * max(1.0, np.max(np.abs(fd)))
    assert res["min_gap"] > 1e-9


def _torch_net_loss(layers, params, x, label, hw):
    """Same net written with torch CPU ops in float64 (conv2d is cross-correlation)."""
    import torch
    import torch.nn.functional as F
    p = torch.tensor(params, dtype=torch.float64, requires_grad=True)
    a = torch.tensor(x, dtype=torch.float64).reshape(1, 1, hw, hw)
    off = 0
    _, dims, _ = orc.shape(layers, hw, hw)
    for (kind, maps, k), d in zip(layers, dims):
        cin = int(d[0])
        if kind == orc.CONV:
            nw = maps * cin * k * k
            w = p[off:off + nw].reshape(maps, cin, k, k)
            b = p[off + nw:off + nw + maps]
            off += nw + maps
            a = A * torch.tanh(B * F.conv2d(a, w, b))
        elif kind == orc.MAXPOOL:
            a = F.max_pool2d(a, k, k)
        else:
            a = a.reshape(1, -1)
            nw = maps * cin
            w = p[off:off + nw].reshape(maps, cin)
            b = p[off + nw:off + nw + maps]
            off += nw + maps
            a = A * torch.tanh(B * F.linear(a, w, b))
    y = a.reshape(-1)
    t = torch.zeros_like(y)
    t[label] = 1.0
    E = 0.5 * ((y - t) ** 2).sum()
    E.backward()
    return y.detach().numpy(), E.item(), p.grad.numpy()


def test_torch_max_pool_tie_rule_is_first_maximum():
    # The torch cross-check below relies on torch's CPU max-pool picking the
    # first maximum in row-major order on exact ties, as the oracle does.
    import torch
    import torch.nn.functional as F
    a = torch.zeros(1, 1, 2, 2, dtype=torch.float64, requires_grad=True)
    F.max_pool2d(a, 2, 2).sum().backward()
    assert a.grad.reshape(-1).tolist() == [1.0, 0.0, 0.0, 0.0]


@pytest.mark.parametrize("net", ["small", "medium", "large"])
def test_whole_net_gradient_against_torch_autograd(net):
    layers = wl.NETS[net]
    params = wl.init_params(layers).astype(np.float64)
    x, y = wl.train_set(3)
    for i in range(2):
        res = orc.forward_backward(layers, params, x[i], int(y[i]))
        out_t, loss_t, grad_t = _torch_net_loss(layers, params, x[i], int(y[i]), 29)
        np.testing.assert_allclose(res["out"], out_t, rtol=1e-12, atol=1e-14)
        assert abs(res["loss"] - loss_t) <= 1e-12 * abs(loss_t)
        np.testing.assert_allclose(res["grad"], grad_t, rtol=1e-9, atol=1e-13)


# --------------------------------------------------------------------------
# Special cases that reduce to textbook results.
def test_pool_k1_is_identity():
    rng = np.random.default_rng(3)
    a = [(orc.CONV, 2, 3), (orc.CONV, 2, 2), (orc.FC, 3, 0)]
    b = [(orc.CONV, 2, 3), (orc.MAXPOOL, 0, 1), (orc.CONV, 2, 2), (orc.FC, 3, 0)]
    p = _rand_params(a, 8, rng)
    x = rng.random(64).astype(np.float32)
    ra = orc.forward_backward(a, p, x, 1, in_h=8, in_w=8)
    rb = orc.forward_backward(b, p, x, 1, in_h=8, in_w=8)
    assert np.array_equal(ra["out"], rb["out"]) and np.array_equal(ra["grad"], rb["grad"])


def test_conv_with_kernel_equal_to_map_is_fc():
    # conv(O maps, k = H) on C x H x W has the weight layout W[o][c][u][v], which
    # is exactly an FC layer's W[j][i] over the map-major flattened input.
    rng = np.random.default_rng(4)
    a = [(orc.CONV, 3, 2), (orc.CONV, 4, 6), (orc.FC, 3, 0)]
    b = [(orc.CONV, 3, 2), (orc.FC, 4, 0), (orc.FC, 3, 0)]
    p = _rand_params(a, 7, rng)
    assert p.size == orc.n_params(b, 7, 7)
    x = rng.random(49).astype(np.float32)
    ra = orc.forward_backward(a, p, x, 2, in_h=7, in_w=7)
    rb = orc.forward_backward(b, p, x, 2, in_h=7, in_w=7)
    np.testing.assert_allclose(ra["out"], rb["out"], rtol=1e-14)
    np.testing.assert_allclose(ra["grad"], rb["grad"], rtol=1e-12, atol=1e-15)


def test_identity_fc_gradient_is_least_squares():
    # One FC layer, identity activation: E = 1/2 |Wx + b - t|^2,
    # dE/dW = (Wx + b - t) x^T, dE/db = Wx + b - t.
    rng = np.random.default_rng(5)
    layers = [(orc.FC, 4, 0)]
    W = rng.standard_normal((4, 9))
    b = rng.standard_normal(4)
    x = rng.random(9).astype(np.float32)
    p = np.concatenate([W.ravel(), b])
    res = orc.forward_backward(layers, p, x, 3, act=orc.ACT_IDENTITY, in_h=3, in_w=3)
    t = np.eye(4)[3]
    r = W @ x.astype(np.float64) + b - t
    np.testing.assert_allclose(res["out"], W @ x.astype(np.float64) + b, rtol=1e-14)
    np.testing.assert_allclose(res["grad"], np.concatenate([np.outer(r, x).ravel(), r]),
                               rtol=1e-13, atol=1e-15)
    assert abs(res["loss"] - 0.5 * r @ r) < 1e-13


def test_lr_zero_leaves_weights_unchanged():
    layers = wl.NETS["small"]
    p0 = wl.init_params(layers).astype(np.float64)
    x, y = wl.tiny_set(20)
    p1, losses = orc.train_sequential(layers, p0, x, y, 0.0)
    assert np.array_equal(p0, p1)
    # with frozen weights every per-sample loss equals the fixed-weight loss
    for i in (0, 7, 19):
        assert losses[i] == orc.forward_backward(layers, p0, x[i], int(y[i]), grad=False)["loss"]


def test_one_sgd_step_is_w_minus_lr_g():
    layers = wl.NETS["small"]
    p0 = wl.init_params(layers).astype(np.float64)
    x, y = wl.tiny_set(1)
    g = orc.forward_backward(layers, p0, x[0], int(y[0]))["grad"]
    lr = 0.05
    p1, _ = orc.train_sequential(layers, p0, x, y, lr, store_f32=False)
    np.testing.assert_allclose(p1, p0 - lr * g, rtol=0, atol=1e-15)
    p1f, _ = orc.train_sequential(layers, p0, x, y, lr, store_f32=True)
    assert np.array_equal(p1f, (p0 - lr * g).astype(np.float32).astype(np.float64))


def test_two_sgd_steps_use_the_updated_weights():
    layers = wl.NETS["small"]
    p0 = wl.init_params(layers).astype(np.float64)
    x, y = wl.tiny_set(2)
    lr = 0.05
    g0 = orc.forward_backward(layers, p0, x[0], int(y[0]))["grad"]
    p1 = p0 - lr * g0
    g1 = orc.forward_backward(layers, p1, x[1], int(y[1]))["grad"]
    p2, _ = orc.train_sequential(layers, p0, x, y, lr, store_f32=False)
    np.testing.assert_allclose(p2, p1 - lr * g1, rtol=0, atol=1e-14)


def test_grad_sum_and_evaluate_consistency():
    layers = wl.NETS["small"]
    p = wl.init_params(layers).astype(np.float64)
    x, y = wl.tiny_set(12)
    G, losses = orc.grad_sum(layers, p, x, y)
    ref = sum(orc.forward_backward(layers, p, x[i], int(y[i]))["grad"] for i in range(12))
    np.testing.assert_allclose(G, ref, rtol=1e-13, atol=1e-15)
    out, wrong = orc.evaluate(layers, p, x, y)
    assert wrong == int(np.sum(np.argmax(out, axis=1) != y))  # numpy: first maximum
    assert wrong == sum(int(np.argmax(orc.forward_backward(layers, p, x[i], 0, grad=False)["out"]) != y[i])
                        for i in range(12))


def test_exact_pool_ties_pick_first_maximum():
    # An all-zero image: every conv output of a map equals f(b_o), so every
    # pooling window is an exact tie; the first element must receive the error.
    layers = [(orc.CONV, 1, 2), (orc.MAXPOOL, 0, 2), (orc.FC, 2, 0)]
    conv = [0.1, -0.2, 0.3, 0.4, 0.25]          # W[0][0][2][2], b[0]
    p = np.concatenate([conv, np.full(2 * 16, 0.3), [0.1, -0.1]])
    x = np.zeros(81, dtype=np.float32)
    res = orc.forward_backward(layers, p, x, 0, in_h=9, in_w=9)
    # conv weight grad = sum over argmax positions of delta * input = 0 (input is 0),
    # bias grad = sum of deltas routed to the 16 first-elements.
    assert np.all(res["grad"][:4] == 0.0)
    assert res["grad"][4] != 0.0
    # the bias gradient equals the sum over windows of the routed error times
    # f'(b) -- each window routes to exactly one element
    fb, dfb = orc.activation(0.25)
    y_pool = np.full(16, fb)
    z_fc = 0.3 * y_pool.sum() + np.array([0.1, -0.1])
    out = A * np.tanh(B * z_fc)
    e_out = out - np.array([1.0, 0.0])
    delta_fc = e_out * A * B * (1 - np.tanh(B * z_fc) ** 2)
    e_pool = 0.3 * delta_fc.sum()
    assert abs(res["grad"][4] - 16 * e_pool * dfb) < 1e-12


# --------------------------------------------------------------------------
# Learning: per-sample SGD on the learnable synthetic task improves accuracy.
@pytest.mark.slow
def test_small_net_learns_projection_labels():
    layers = wl.NETS["small"]
    p0 = wl.init_params(layers).astype(np.float64)
    x, y = wl.train_set(6000)
    xt, yt = wl.test_set(1000)
    _, wrong0 = orc.evaluate(layers, p0, xt, yt)
    p1, losses = orc.train_sequential(layers, p0, x, y, 0.01)
    _, wrong1 = orc.evaluate(layers, p1, xt, yt)
    assert losses[-1000:].mean() < 0.92 * losses[:1000].mean()
    assert wrong1 < 0.85 * wrong0


# --------------------------------------------------------------------------
# Prediction ties (reading: lowest index among equal maxima; Table II counts
# depend on it).  All-zero output-layer weights and biases make every output
# exactly f(0) = 0, so every prediction is class 0.
def test_prediction_ties_go_to_the_lowest_index():
    layers = wl.NETS["small"]
    p = wl.init_params(layers).astype(np.float64)
    n_fc2 = 10 * 50 + 10
    p[-n_fc2:] = 0.0
    x, y = wl.train_set(200)
    out, wrong = orc.evaluate(layers, p, x, y)
    assert np.all(out == 0.0)
    assert wrong == int(np.sum(y != 0)) and 0 < wrong < 200
    # a tie between two classes above the rest: outputs 3 and 7 share the
    # largest bias, so every prediction is 3
    p[-10:] = [0.1, 0.0, 0.2, 0.5, -0.3, 0.1, 0.0, 0.5, 0.2, -0.1]
    out, wrong = orc.evaluate(layers, p, x, y)
    assert np.all(out[:, 3] == out[:, 7]) and np.all(out[:, 3] > out[:, [0, 1, 2, 4, 5, 6, 8, 9]].T)
    assert wrong == int(np.sum(y != 3))


# --------------------------------------------------------------------------
# The max-pool gap diagnostic (smallest positive relative distance between a
# window's maximum and its runner-up) decides which fp32/fp64 mismatches the
# GPU comparisons may forgive, so it is pinned on hand-built windows: a
# pooling layer directly on the image makes each window's values the pixels.
def _gap_net_and_images():
    layers = [(orc.MAXPOOL, 0, 2), (orc.FC, 2, 0)]
    a = np.array([[0.5, 0.4, 0.9, 0.45],     # window (0,0): 0.5 / 0.4   -> 0.2
                  [0.2, 0.1, 0.3, 0.2],      # window (0,1): 0.9 / 0.45  -> 0.5
                  [0.3, 0.2, 0.6, 0.6],      # window (1,0): 0.3 / 0.297 -> 0.01
                  [0.297, 0.0, 0.6, 0.6]],   # window (1,1): exact tie   -> left out
                 dtype=np.float32)
    b = np.array([[-0.3, -0.5, 0.7, 0.7],    # window (0,0): -0.3 / -0.5 -> 2/3
                  [-0.6, -0.9, 0.7, 0.7],    # the other three windows are exact ties
                  [0.1, 0.1, 0.2, 0.2],
                  [0.1, 0.1, 0.2, 0.2]], dtype=np.float32)
    c = np.full((4, 4), 0.25, dtype=np.float32)  # every window an exact tie
    return layers, np.stack([a.ravel(), b.ravel(), c.ravel()])


def test_min_gap_on_hand_built_windows():
    layers, x = _gap_net_and_images()
    p = np.linspace(-0.5, 0.5, orc.n_params(layers, 4, 4))
    f32 = lambda v: float(np.float32(v))  # the image holds fp32 pixels
    expect = [(f32(0.3) - f32(0.297)) / f32(0.3),
              (f32(-0.3) - f32(-0.5)) / abs(f32(-0.3)),
              math.inf]
    y = np.array([0, 1, 0], dtype=np.int32)
    for i in range(3):
        g = orc.forward_backward(layers, p, x[i], int(y[i]), in_h=4, in_w=4)["min_gap"]
        assert g == pytest.approx(expect[i], rel=1e-12) if math.isfinite(expect[i]) else g == math.inf
    assert abs(expect[0] - 0.01) < 1e-6 and abs(expect[1] - 2.0 / 3.0) < 1e-7
    # the training and gradient-sum paths report the same per-sample gaps
    _, _, gaps = orc.train_sequential(layers, p, x, y, 0.0, in_h=4, in_w=4, with_gaps=True)
    _, _, gaps2 = orc.grad_sum(layers, p, x, y, in_h=4, in_w=4, with_gaps=True)
    for gg in (gaps, gaps2):
        assert gg[0] == pytest.approx(expect[0], rel=1e-12)
        assert gg[1] == pytest.approx(expect[1], rel=1e-12)
        assert gg[2] == math.inf
