"""chaos_forward_backward_noalloc against chaos_forward_backward, on MI355X.

The variant allocates nothing: a gradient sum's per-worker partial sums live
in a fixed array of device memory that every call on the device shares.  Its
outputs and losses must equal the allocating entry point's bit for bit (the
per-sample forward pass does not depend on the worker), its gradient sum must
meet the allocating one's at 1e-4 (the same sum in another fixed order: fewer
workers, and for the large net per-sample pushes instead of the batched
contractions).  Two calls in a row, the second with fewer samples, check that
the array left by the first call does not leak into the second.
"""
import numpy as np
import pytest

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


@pytest.mark.parametrize("name,sizes", [("small", (1500, 311)), ("medium", (700, 123)),
                                        ("large", (300, 77)), ("large_table1", (200, 45))])
def test_noalloc_matches_forward_backward(env, name, sizes):
    torch, chaos = env
    layers = wl.NETS[name]
    net = chaos.Net(layers, wl.init_params(layers))
    x, y = wl.batch_set(max(sizes))
    xd, yd = _dev(torch, x, torch.float32), _dev(torch, y, torch.int32)
    for n in sizes:
        print(f"noalloc {name} n={n}", flush=True)
        ref = {k: torch.empty(s, device="cuda") for k, s in
               (("out", (n, net.n_out)), ("loss", (n,)), ("g", (net.n_params,)))}
        new = {k: torch.full_like(v, float("nan")) for k, v in ref.items()}
        net.forward_backward(xd[:n], yd[:n], out=ref["out"], loss=ref["loss"], grad_sum=ref["g"])
        net.forward_backward_noalloc(xd[:n], yd[:n], out=new["out"], loss=new["loss"],
                                     grad_sum=new["g"])
        again = torch.empty(net.n_params, device="cuda")
        net.forward_backward_noalloc(xd[:n], yd[:n], grad_sum=again)
        torch.cuda.synchronize()
        assert torch.equal(new["out"], ref["out"]) and torch.equal(new["loss"], ref["loss"])
        assert torch.equal(again, new["g"])  # reproducible bit for bit
        assert_close(new["g"].cpu().numpy(), ref["g"].cpu().double().numpy(),
                     what=f"{name} gradient sum over {n} samples")


def test_noalloc_empty_input_and_rejected_sizes(env):
    torch, chaos = env
    layers = wl.NETS["small"]
    net = chaos.Net(layers, wl.init_params(layers))
    g = torch.full((net.n_params,), 3.0, device="cuda")
    net.forward_backward_noalloc(torch.empty(0, 841, device="cuda"),
                                 torch.empty(0, dtype=torch.int32, device="cuda"), grad_sum=g)
    torch.cuda.synchronize()
    assert torch.all(g == 0)
    # one partial-sum row of a net with more weights than the fixed array holds
    big = [(chaos.FC, 9980, 0), (chaos.FC, 10, 0)]
    rng = np.random.default_rng(1)
    nb = 9980 * 842 + 10 * 9981
    assert nb > 32 * 2**20 // 4
    bnet = chaos.Net(big, rng.uniform(-0.03, 0.03, nb).astype(np.float32))
    x, y = wl.batch_set(3)
    xd, yd = _dev(torch, x, torch.float32), _dev(torch, y, torch.int32)
    with pytest.raises(chaos.ChaosError) as e:
        bnet.forward_backward_noalloc(xd, yd, grad_sum=torch.empty(nb, device="cuda"))
    assert e.value.code == chaos.EUNSUPPORTED
    # without a gradient sum the same call needs no scratch
    out_a = torch.empty(3, 10, device="cuda")
    out_b = torch.empty(3, 10, device="cuda")
    bnet.forward_backward(xd, yd, out=out_a)
    bnet.forward_backward_noalloc(xd, yd, out=out_b)
    torch.cuda.synchronize()
    assert torch.equal(out_a, out_b)
