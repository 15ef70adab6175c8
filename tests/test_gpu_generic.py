"""Parity of the generic kernel (any layer list the shape walk accepts) with
the oracle, on MI355X.

The four nets of the evaluation have fused kernels of their own; every other
architecture runs on the generic worker kernel (per-worker state in HBM,
scalar loops over runtime shapes).  These nets are none of the four: two of
the oracle's finite-difference nets on 8x8 and 9x9 inputs and a 29x29 net
with a 5x5 pooling layer.  Covered: per-sample outputs, losses and gradients
when every worker processes several samples in a row, the gradient sum,
short per-sample SGD runs (which need each worker to see its own updates of
the previous sample, Section III-A.2), Hogwild with one worker equal to
sequential SGD bit for bit, and lr = 0 with every resident worker.
"""
import numpy as np
import pytest

from oracle import oracle as orc
from paper_1506_09067_amd import workloads as wl

from . import _oracle_par as par
from ._compare import assert_close, close_report

pytestmark = pytest.mark.gpu

NEAR_TIE = 1e-5
AMBIGUOUS = 2e-6

# name: (input side, layer list)
GENERIC = {
    "conv_pool_fc": (8, [(orc.CONV, 2, 3), (orc.MAXPOOL, 0, 2), (orc.FC, 4, 0)]),
    "conv_conv_pool": (9, [(orc.CONV, 2, 2), (orc.CONV, 2, 3), (orc.MAXPOOL, 0, 3), (orc.FC, 3, 0)]),
    "conv_pool5_fc_fc": (29, [(orc.CONV, 6, 5), (orc.MAXPOOL, 0, 5), (orc.FC, 20, 0), (orc.FC, 10, 0)]),
}


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.fixture(scope="module")
def chaos(torch_cuda):
    from paper_1506_09067_amd import chaos as c
    c.lib()
    return c


def _dev(torch, a, dtype):
    return torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def _setup(name, n, seed=7):
    hw, layers = GENERIC[name]
    p = wl.init_params(layers, seed=wl.SEED_INIT, in_h=hw, in_w=hw)
    n_out = int(np.prod(orc.shape(layers, hw, hw)[1][-1, 3:6]))
    x = wl.images(n, seed, hw * hw)
    y = (wl.uniform_labels(n, seed) % n_out).astype(np.int32)
    return hw, layers, p, x, y


def _fb(name, layers, p, x, y, hw, idx, grad=True):
    return par.forward_backward(layers, p, x, y, idx, in_h=hw, in_w=hw, grad=grad)


@pytest.mark.parametrize("name", sorted(GENERIC))
def test_generic_per_sample_and_sum(chaos, torch_cuda, name):
    torch = torch_cuda
    hw0, layers0 = GENERIC[name]
    probe = chaos.Net(layers0, wl.init_params(layers0, in_h=hw0, in_w=hw0), in_h=hw0, in_w=hw0)
    n = 2 * probe.max_workers + 7  # every worker two or three samples in a row
    hw, layers, p, x, y = _setup(name, n)
    net = chaos.Net(layers, p, in_h=hw, in_w=hw)
    xd, yd = _dev(torch, x, torch.float32), _dev(torch, y, torch.int32)
    each = torch.empty(n, net.n_params, device="cuda")
    out = torch.empty(n, net.n_out, device="cuda")
    loss = torch.empty(n, device="cuda")
    net.forward_backward(xd, yd, out=out, loss=loss, grad_each=each)
    gsum = torch.empty(net.n_params, device="cuda")
    net.forward_backward(xd, yd, grad_sum=gsum)
    torch.cuda.synchronize()
    out, loss, each = out.cpu().numpy(), loss.cpu().numpy(), each.cpu().double().numpy()
    refs = _fb(name, layers, p, x, y, hw, range(n))
    skipped = []
    for i, r in enumerate(refs):
        assert_close(out[i], r["out"], what=f"{name} out[{i}]")
        assert_close([loss[i]], [r["loss"]], what=f"{name} loss[{i}]")
        ok, msg = close_report(each[i], r["grad"])
        if not ok and r["min_gap"] < NEAR_TIE:
            skipped.append(i)
            continue
        assert ok, f"{name} grad[{i}]: {msg}"
    assert len(skipped) <= 2, skipped
    keep = [i for i in range(n) if i not in skipped]
    G = np.sum([refs[i]["grad"] for i in keep], axis=0)
    assert_close(gsum.cpu().double().numpy() - each[skipped].sum(0), G,
                 what=f"{name} gradient sum over {n} samples")


@pytest.mark.parametrize("name", sorted(GENERIC))
def test_generic_sequential_sgd(chaos, torch_cuda, name):
    """Per-sample SGD, lr 1e-2, index order, against the oracle up to the
    first ambiguous max-pool tie (losses over the whole run)."""
    torch = torch_cuda
    n = 300
    hw, layers, p, x, y = _setup(name, n, seed=8)
    _, L_ref, gaps = orc.train_sequential(layers, p, x, y, 1e-2, in_h=hw, in_w=hw, with_gaps=True)
    amb = np.where(gaps < AMBIGUOUS)[0]
    n_cut = int(amb[0]) if amb.size else n
    assert n_cut >= 50
    net = chaos.Net(layers, p, in_h=hw, in_w=hw)
    loss = torch.empty(n_cut, device="cuda")
    net.train_epoch(_dev(torch, x[:n_cut], torch.float32), _dev(torch, y[:n_cut], torch.int32), 1e-2,
                    mode=chaos.SEQUENTIAL, loss=loss)
    w = net.get_params().cpu().numpy()
    p_ref, L_cut = orc.train_sequential(layers, p, x[:n_cut], y[:n_cut], 1e-2, in_h=hw, in_w=hw)
    assert_close(loss.cpu().numpy(), L_cut, what=f"{name} per-sample losses, {n_cut} samples")
    assert_close(w, p_ref, what=f"{name} weights after {n_cut} samples")
    assert_close(w - p, p_ref - p, tol=1e-3, what=f"{name} total weight change")


@pytest.mark.parametrize("name", sorted(GENERIC))
def test_generic_hogwild_one_worker_is_sequential(chaos, torch_cuda, name):
    torch = torch_cuda
    n = 400
    hw, layers, p, x, y = _setup(name, n, seed=9)
    xd, yd = _dev(torch, x, torch.float32), _dev(torch, y, torch.int32)
    res = []
    for mode, workers in ((chaos.SEQUENTIAL, 0), (chaos.HOGWILD_ATOMIC, 1), (chaos.HOGWILD_RACY, 1)):
        net = chaos.Net(layers, p, in_h=hw, in_w=hw)
        loss = torch.empty(n, device="cuda")
        net.train_epoch(xd, yd, 1e-2, mode=mode, workers=workers, loss=loss)
        res.append((net.get_params().cpu(), loss.cpu()))
    for what, (w, l) in zip(("atomic", "racy"), res[1:]):
        assert torch.equal(w, res[0][0]) and torch.equal(l, res[0][1]), what


@pytest.mark.parametrize("name", sorted(GENERIC))
def test_generic_every_worker_lr_zero_claims_once(chaos, torch_cuda, name):
    torch = torch_cuda
    hw0, layers0 = GENERIC[name]
    probe = chaos.Net(layers0, wl.init_params(layers0, in_h=hw0, in_w=hw0), in_h=hw0, in_w=hw0)
    n = 3 * probe.max_workers + 11
    hw, layers, p, x, y = _setup(name, n, seed=10)
    net = chaos.Net(layers, p, in_h=hw, in_w=hw)
    xd, yd = _dev(torch, x, torch.float32), _dev(torch, y, torch.int32)
    claims = torch.zeros(n, dtype=torch.int32, device="cuda")
    net.set_claim_counter(claims)
    loss = torch.empty(n, device="cuda")
    net.train_epoch(xd, yd, 0.0, mode=chaos.HOGWILD_ATOMIC, workers=net.max_workers, loss=loss)
    net.set_claim_counter(None)
    torch.cuda.synchronize()
    assert torch.all(claims == 1)
    assert torch.equal(net.get_params().cpu(), torch.from_numpy(p))
    idx = list(range(0, n, max(1, n // 16)))
    ref = np.array([r["loss"] for r in _fb(name, layers, p, x, y, hw, idx, grad=False)])
    assert_close(loss.cpu().numpy()[idx], ref, what=f"{name} losses at lr 0")
