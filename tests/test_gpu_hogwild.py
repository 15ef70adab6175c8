"""Hogwild acceptance on MI355X: training with many concurrent lock-free
workers ends within 1% of sequential per-sample SGD on the same seeded data.

Hogwild results are not deterministic (Section IV-B attributes the spread in
Table II to the non-deterministic weight updates), so they are compared with
the sequential run statistically: final test-set loss within 1% (relative)
and accuracy within 1 percentage point.  Sequential SGD itself is checked
against the oracle in test_gpu_parity.py.
"""
import os

import numpy as np
import pytest

from paper_1506_09067_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1506_09067_amd import chaos
    chaos.lib()
    return torch, chaos


def _train_and_test(torch, chaos, name, x, y, xt, yt, epochs, lr, decay, mode, workers):
    layers = wl.NETS[name]
    net = chaos.Net(layers, wl.init_params(layers))
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    for ep in range(epochs):
        net.train_epoch(xd, yd, lr * decay ** ep, mode=mode, workers=workers)
        if epochs > 5:  # long runs report their progress
            torch.cuda.synchronize()
            print(f"  {name} mode {mode} epoch {ep + 1}/{epochs} done", flush=True)
    xtd, ytd = torch.from_numpy(xt).cuda(), torch.from_numpy(yt).cuda()
    loss = torch.empty(len(yt), device="cuda")
    net.forward_backward(xtd, ytd, loss=loss)
    wrong = net.evaluate(xtd, ytd)
    w = net.get_params()
    torch.cuda.synchronize()
    assert torch.isfinite(w).all()
    return float(loss.double().mean()), int(wrong.item()), net.default_workers


# (net, training samples, epochs, lr, lr decay per epoch, Hogwild workers;
# 0 = the library's default: one worker per compute unit, 256).  That is the
# benchmark's configuration; the workers of an epoch join as its first
# samples complete, so their first gradients are not all computed at the same
# weights.  The small net has only 6,405 weights, each touched by every
# sample: at 512 or 768 concurrent workers (its kernel holds 768) its loss
# spikes early in the first epoch and a few runs in a hundred saturate and do
# not recover (a delayed-gradient instability: staleness x lr x the curvature
# of the output layer's common direction), while at 256 no run has spiked.
CASES = [
    ("small", 60000, 5, 1e-3, 0.9, 0),     # the small net's schedule
    ("medium", 60000, 3, 1e-3, 0.9, 0),
    ("large", 60000, 1, 1e-3, 0.9, 0),
    ("large", 60000, 1, 1e-3, 0.9, 64),
    ("large_table1", 30000, 1, 1e-3, 0.9, 0),
]

# The medium and large nets' full configurations (constant lr 1e-3, 5 and 15
# epochs of 60,000 samples, the default 256 workers).  The sequential reference
# of the large net takes about four minutes of one-worker training, so these
# run only with CHAOS_SLOW=1.
SLOW_CASES = [
    ("medium", 60000, 5, 1e-3, 1.0, 0),
    ("large", 60000, 15, 1e-3, 1.0, 0),
]


@pytest.mark.parametrize("name,n,epochs,lr,decay,workers", CASES)
def test_hogwild_matches_sequential_sgd(env, name, n, epochs, lr, decay, workers):
    _accept(env, name, n, epochs, lr, decay, workers)


@pytest.mark.slow
@pytest.mark.skipif(os.environ.get("CHAOS_SLOW") != "1",
                    reason="full-length acceptance runs (minutes of sequential training): CHAOS_SLOW=1")
@pytest.mark.parametrize("name,n,epochs,lr,decay,workers", SLOW_CASES)
def test_hogwild_matches_sequential_sgd_full_length(env, name, n, epochs, lr, decay, workers):
    _accept(env, name, n, epochs, lr, decay, workers)


def _accept(env, name, n, epochs, lr, decay, workers):
    torch, chaos = env
    x, y = wl.train_set(n)
    xt, yt = wl.test_set(10000)
    seq = _train_and_test(torch, chaos, name, x, y, xt, yt, epochs, lr, decay, chaos.SEQUENTIAL, 0)
    hog = _train_and_test(torch, chaos, name, x, y, xt, yt, epochs, lr, decay,
                          chaos.HOGWILD_ATOMIC, workers)
    # the sequential run learned something, so the comparison is not vacuous
    init = _train_and_test(torch, chaos, name, x[:0], y[:0], xt, yt, 1, lr, decay,
                           chaos.SEQUENTIAL, 0)
    assert seq[0] < init[0]
    nt = len(yt)
    msg = (f"{name}: sequential loss {seq[0]:.5f} wrong {seq[1]}/{nt}; Hogwild with "
           f"{workers or hog[2]} workers loss {hog[0]:.5f} wrong {hog[1]}/{nt}; "
           f"untrained loss {init[0]:.5f}")
    print(msg, flush=True)
    assert abs(hog[0] - seq[0]) <= 0.01 * seq[0], msg
    # accuracy within one percentage point, counted in whole test images
    assert 100 * abs(hog[1] - seq[1]) <= nt, msg
