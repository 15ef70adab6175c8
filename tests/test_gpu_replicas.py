"""Weight replicas on MI355X (chaos_set_replicas): atomic Hogwild workers read
one of r copies of the small net's weights, push every update to the shared
weights and to their copy, and each copy is refreshed from the shared weights
after every m-th sample completed on it.

With one worker nothing else updates the weights, so an epoch must equal
sequential per-sample SGD bit for bit; with every resident worker at lr 0
every sample is claimed once at the initial weights; over a training run the
result must stay within the Hogwild acceptance bound of sequential SGD
(Section IV-B; reading 17).
"""
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


def _dev(torch, a, dtype):
    return torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


@pytest.mark.parametrize("r,m", [(8, 1), (8, 4), (3, 5)])
def test_one_worker_with_replicas_is_sequential(env, r, m):
    torch, chaos = env
    layers = wl.NETS["small"]
    p = wl.init_params(layers)
    x, y = wl.train_set(400)
    xd, yd = _dev(torch, x, torch.float32), _dev(torch, y, torch.int32)
    seq = chaos.Net(layers, p)
    l_seq = torch.empty(400, device="cuda")
    seq.train_epoch(xd, yd, 1e-2, mode=chaos.SEQUENTIAL, loss=l_seq)
    net = chaos.Net(layers, p)
    net.set_replicas(r, m)
    l_rep = torch.empty(400, device="cuda")
    net.train_epoch(xd, yd, 1e-2, mode=chaos.HOGWILD_ATOMIC, workers=1, loss=l_rep)
    # a second epoch starts from replicas copied again from the shared weights
    net.train_epoch(xd, yd, 1e-2, mode=chaos.HOGWILD_ATOMIC, workers=1)
    seq.train_epoch(xd, yd, 1e-2, mode=chaos.SEQUENTIAL)
    torch.cuda.synchronize()
    assert torch.equal(l_rep, l_seq)
    assert torch.equal(net.get_params(), seq.get_params())


def test_every_worker_with_replicas_lr_zero_claims_once(env):
    torch, chaos = env
    layers = wl.NETS["small"]
    p = wl.init_params(layers)
    net = chaos.Net(layers, p)
    net.set_replicas(8, 2)
    n = 20011
    x, y = wl.train_set(n)
    xd, yd = _dev(torch, x, torch.float32), _dev(torch, y, torch.int32)
    claims = torch.zeros(n, dtype=torch.int32, device="cuda")
    net.set_claim_counter(claims)
    loss = torch.empty(n, device="cuda")
    net.train_epoch(xd, yd, 0.0, mode=chaos.HOGWILD_ATOMIC, workers=net.max_workers, loss=loss)
    net.set_claim_counter(None)
    ref = torch.empty(n, device="cuda")
    net.forward_backward(xd, yd, loss=ref)
    torch.cuda.synchronize()
    assert torch.all(claims == 1)
    assert torch.equal(net.get_params().cpu(), torch.from_numpy(p))
    assert torch.equal(loss, ref)


def test_replica_arguments(env):
    torch, chaos = env
    small = chaos.Net(wl.NETS["small"], wl.init_params(wl.NETS["small"]))
    for r, m in ((0, 4), (65, 4), (8, 0)):
        with pytest.raises(chaos.ChaosError) as e:
            small.set_replicas(r, m)
        assert e.value.code == chaos.EINVAL
    small.set_replicas(8, 4)
    with pytest.raises(chaos.ChaosError) as e:
        small.set_push_delay(2)
    assert e.value.code == chaos.EINVAL
    small.set_replicas(1, 1)
    small.set_push_delay(2)
    with pytest.raises(chaos.ChaosError) as e:
        small.set_replicas(8, 4)
    assert e.value.code == chaos.EINVAL
    small.set_push_delay(1)
    medium = chaos.Net(wl.NETS["medium"], wl.init_params(wl.NETS["medium"]))
    with pytest.raises(chaos.ChaosError) as e:
        medium.set_replicas(8, 4)
    assert e.value.code == chaos.EUNSUPPORTED
    medium.set_replicas(1, 1)  # off is always accepted


def test_replicas_match_sequential_sgd(env):
    """The small net's schedule (60,000 samples x 5 epochs, lr 1e-3 x 0.9 per
    epoch) with the default 256 workers on 8 replicas refreshed every 8
    samples: final test loss within 1 % and accuracy within one percentage
    point of sequential SGD."""
    torch, chaos = env
    layers = wl.NETS["small"]
    p = wl.init_params(layers)
    x, y = wl.train_set(60000)
    xt, yt = wl.test_set(10000)
    xd, yd = _dev(torch, x, torch.float32), _dev(torch, y, torch.int32)
    xtd, ytd = _dev(torch, xt, torch.float32), _dev(torch, yt, torch.int32)

    def run(mode, replicas):
        net = chaos.Net(layers, p)
        if replicas:
            net.set_replicas(8, 8)
        for ep in range(5):
            net.train_epoch(xd, yd, 1e-3 * 0.9 ** ep, mode=mode)
        loss = torch.empty(10000, device="cuda")
        net.forward_backward(xtd, ytd, loss=loss)
        wrong = net.evaluate(xtd, ytd)
        torch.cuda.synchronize()
        return float(loss.double().mean()), int(wrong.item())

    seq = run(chaos.SEQUENTIAL, False)
    rep = run(chaos.HOGWILD_ATOMIC, True)
    msg = f"sequential {seq}, 8 replicas every 8 samples {rep}"
    print(msg, flush=True)
    assert abs(rep[0] - seq[0]) <= 0.01 * seq[0], msg
    assert 100 * abs(rep[1] - seq[1]) <= 10000, msg
