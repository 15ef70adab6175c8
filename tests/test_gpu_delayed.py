"""Delayed pushes on MI355X (chaos_set_push_delay): every worker sums its
per-layer gradients privately and pushes the sum every k samples.

With one worker nothing else updates the weights, so an epoch is mini-batch
SGD over k consecutive samples: each batch's per-sample gradients are taken at
the weights left by the previous batch and their sum is applied at once.  The
expected values come from the oracle's frozen-weight gradient sums
(grad_sum, pinned in test_oracle.py) applied batch by batch.
"""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_1506_09067_amd import workloads as wl

from ._compare import assert_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1506_09067_amd import chaos
    chaos.lib()
    return torch, chaos


def _dev(torch, a, dtype):
    return torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def _minibatch_sgd(layers, p, x, y, lr, k):
    """Batches of k consecutive samples (the last one may be shorter): the
    gradient sum at the current weights, then w <- w - lr * sum, stored as
    fp32 like the shared weights."""
    w = np.asarray(p, dtype=np.float32).copy()
    losses = []
    for b in range(0, len(y), k):
        g, l = orc.grad_sum(layers, w, x[b:b + k], y[b:b + k])
        losses.append(l)
        w = (w.astype(np.float64) - lr * g).astype(np.float32)
    return w, np.concatenate(losses)


@pytest.mark.parametrize("k,n", [(4, 64), (5, 63)])
def test_one_worker_is_minibatch_sgd(env, k, n):
    torch, chaos = env
    layers = wl.NETS["small"]
    p = wl.init_params(layers)
    x, y = wl.tiny_set(n)
    net = chaos.Net(layers, p)
    net.set_push_delay(k)
    loss = torch.empty(n, device="cuda")
    net.train_epoch(_dev(torch, x, torch.float32), _dev(torch, y, torch.int32), 1e-2,
                    mode=chaos.HOGWILD_ATOMIC, workers=1, loss=loss)
    w = net.get_params().cpu().numpy()
    w_ref, l_ref = _minibatch_sgd(layers, p, x, y, 1e-2, k)
    assert_close(loss.cpu().numpy(), l_ref, what=f"per-sample losses, batches of {k}")
    assert_close(w - p, w_ref - p, tol=1e-3, what="total weight change")
    assert_close(w, w_ref, what=f"weights after {n} samples in batches of {k}")


def test_every_worker_lr_zero_claims_once(env):
    torch, chaos = env
    layers = wl.NETS["small"]
    p = wl.init_params(layers)
    net = chaos.Net(layers, p)
    plain = net.max_workers
    net.set_push_delay(8)
    wmax = net.max_workers  # the delayed kernel's capacity
    assert 0 < wmax < plain
    n = 20000
    x, y = wl.train_set(n)
    xd, yd = _dev(torch, x, torch.float32), _dev(torch, y, torch.int32)
    claims = torch.zeros(n, dtype=torch.int32, device="cuda")
    net.set_claim_counter(claims)
    loss = torch.empty(n, device="cuda")
    net.train_epoch(xd, yd, 0.0, mode=chaos.HOGWILD_ATOMIC, workers=wmax, loss=loss)
    net.set_claim_counter(None)
    torch.cuda.synchronize()
    assert torch.all(claims == 1)
    assert torch.equal(net.get_params().cpu(), torch.from_numpy(p))
    ref = np.array([orc.forward_backward(layers, p, x[i], int(y[i]), grad=False)["loss"]
                    for i in range(0, n, n // 16)])
    assert_close(loss.cpu().numpy()[::n // 16], ref, what="losses at lr 0")
    # and a real epoch stays finite and changes the weights
    net.train_epoch(xd, yd, 1e-3, mode=chaos.HOGWILD_ATOMIC, workers=wmax)
    w = net.get_params()
    torch.cuda.synchronize()
    assert torch.isfinite(w).all() and not torch.equal(w.cpu(), torch.from_numpy(p))


def test_push_delay_arguments(env):
    torch, chaos = env
    small = chaos.Net(wl.NETS["small"], wl.init_params(wl.NETS["small"]))
    with pytest.raises(chaos.ChaosError) as e:
        small.set_push_delay(0)
    assert e.value.code == chaos.EINVAL
    small.set_push_delay(4)
    x, y = wl.tiny_set(8)
    with pytest.raises(chaos.ChaosError) as e:
        small.train_epoch(_dev(torch, x, torch.float32), _dev(torch, y, torch.int32), 1e-3,
                          mode=chaos.HOGWILD_ATOMIC, workers=small.max_workers + 1)
    assert e.value.code == chaos.EINVAL
    small.set_push_delay(1)  # back to the per-layer push and the net's own capacity
    assert small.max_workers > 0
    medium = chaos.Net(wl.NETS["medium"], wl.init_params(wl.NETS["medium"]))
    with pytest.raises(chaos.ChaosError) as e:
        medium.set_push_delay(2)
    assert e.value.code == chaos.EUNSUPPORTED
    medium.set_push_delay(1)
