"""Benchmark of the CHAOS hot path on one MI355X.

One step = one Training epoch of the large net (conv20 k4 -> max2 -> conv60 k3
-> conv100 k6 -> max2 -> FC150 -> FC10) over the 60,000-sample synthetic set,
Hogwild with the maximum number of resident workers, lr 1e-3: every sample is
claimed, forward-propagated, back-propagated and pushed to the shared weights
layer by layer.  Inputs are resident in HBM before the timed region.

Prints one JSON line.  Extra fields:
  roofline      the training kernel's algorithmic FLOP rate (dense count of
                forward, backward-data, weight-gradient and update
                multiply-adds, x2) over its average launch time, against the
                MI355X FP32 peak
  update_stream the training kernel's shared-weight update stream (one fp32
                atomic add per parameter per sample, performed at the memory
                side) in adds/s, next to a plain atomic kernel timed on the
                same footprint (torch's index_add_)
  cpu_baseline  the CPU oracle (sequential per-sample SGD, one core) on a
                bounded sample of the same workload
  rows          training throughput of the small and medium nets and of
                Table I's large net on the same set (default workers, with
                the FP32-peak fraction and the oracle's sequential rate on a
                short prefix), of the small net on 8 weight replicas, and the
                throughput of the frozen-weight 16,384-sample batch gradient
                and of the 10,000-sample test forward pass of the large net
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "training samples/sec (fwd+bwd+update) and % FP32 peak, large net"
PEAK_FP32_TFLOPS = 157.3
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "traffic.json")


def train_flops_per_sample(layers, in_hw=29):
    """Dense algorithmic FLOPs of one training sample: 2 x (forward MACs +
    backward-data MACs of every layer above the input + weight-gradient MACs
    incl. the bias sums + one multiply-add per parameter for the update)."""
    c, h, w = 1, in_hw, in_hw
    fwd = bwd = wgrad = params = 0
    for i, (kind, maps, k) in enumerate(layers):
        if kind == 1:
            ho, wo = h - k + 1, w - k + 1
            mac = maps * ho * wo * c * k * k
            fwd += mac
            if i > 0:
                bwd += mac
            wgrad += mac + maps * ho * wo
            params += maps * (c * k * k + 1)
            c, h, w = maps, ho, wo
        elif kind == 2:
            h, w = h // k, w // k
        else:
            s = c * h * w
            fwd += maps * s
            if i > 0:
                bwd += maps * s
            wgrad += maps * s + maps
            params += maps * (s + 1)
            c, h, w = maps, 1, 1
    return 2 * (fwd + bwd + wgrad + params), 2 * fwd


def kernel_source_hash():
    import hashlib
    csrc = os.path.join(ROOT, "paper_1506_09067_amd", "csrc")
    return hashlib.sha256(b"".join(open(os.path.join(csrc, f), "rb").read()
                                   for f in ("fused_large.hip", "device_common.h"))).hexdigest()


def measured_traffic(net, workers, samples):
    """Calibrated HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE
    counter runs, or None when they were taken on another configuration or
    before the kernel source last changed."""
    if not os.path.exists(PROFILE_TRAFFIC):
        return None
    with open(PROFILE_TRAFFIC) as f:
        t = json.load(f)
    if (t.get("net"), t.get("workers"), t.get("samples_per_launch")) != (net, workers, samples):
        return None
    if t.get("source_sha256") != kernel_source_hash():
        return None
    return t.get("bytes_per_launch")


def update_stream(torch, n_params, samples_per_s, sweeps=256):
    """Atomic adds per second of the Hogwild update stream (every sample adds
    one fp32 value to each of the n_params shared weights, Section III-A.2),
    and the rate of torch's index_add_ adding `sweeps` full sweeps of ones
    into a vector of n_params floats: a plain atomic scatter kernel on the
    same footprint, timed here."""
    acc = torch.zeros(n_params, device="cuda")
    idx = torch.arange(n_params, device="cuda").repeat(sweeps)
    src = torch.ones(n_params * sweeps, device="cuda")
    acc.index_add_(0, idx, src)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(3):
        acc.index_add_(0, idx, src)
    b.record()
    torch.cuda.synchronize()
    ref = 3 * n_params * sweeps / (a.elapsed_time(b) / 1e3)
    adds = samples_per_s * n_params
    del acc, idx, src
    return {"adds_per_s": adds, "reference_adds_per_s": ref,
            "reference": f"torch index_add_, {sweeps} sweeps over {n_params} floats",
            "frac_of_reference": adds / ref}


def cpu_baseline(layers, p0, x, y, budget_s=15.0):
    """The oracle, as it stands, on the first samples of the same set."""
    from oracle import oracle as orc
    n = 8
    t0 = time.perf_counter()
    orc.train_sequential(layers, p0, x[:n], y[:n], 1e-3)
    per = (time.perf_counter() - t0) / n
    n = max(8, min(len(y), int(budget_s / max(per, 1e-6))))
    t0 = time.perf_counter()
    orc.train_sequential(layers, p0, x[:n], y[:n], 1e-3)
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "training samples/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n} samples of the 60,000-sample training set, sequential "
                      f"per-sample SGD (fp64 oracle, one thread), {dt:.1f} s"}


def cpu_batch_baseline(layers, p0, x, y, budget_s=3.0):
    """The oracle's frozen-weight gradient sum on every host core the process
    may use (at most 16): contiguous chunks of a prefix of the batch, one
    thread each (the oracle's C call releases the interpreter lock), partial
    sums added in chunk order."""
    import threading
    import numpy as np
    from oracle import oracle as orc
    cores = max(1, min(len(os.sched_getaffinity(0)), int(os.environ.get("OMP_NUM_THREADS", 16)), 16))
    t0 = time.perf_counter()
    orc.grad_sum(layers, p0, x[:2], y[:2])
    per = (time.perf_counter() - t0) / 2
    k = max(1, min(len(y) // cores, int(budget_s / max(per, 1e-6))))
    n = k * cores
    parts = [None] * cores

    def work(t):
        parts[t] = orc.grad_sum(layers, p0, x[t * k:(t + 1) * k], y[t * k:(t + 1) * k])[0]

    threads = [threading.Thread(target=work, args=(t,)) for t in range(cores)]
    t0 = time.perf_counter()
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    g = np.zeros_like(parts[0])
    for q in parts:
        g += q
    dt = time.perf_counter() - t0
    return {"value": n / dt, "unit": "samples/s", "cores": cores, "kind": "oracle",
            "sample": f"first {n} samples of the 16,384-sample batch, frozen-weight gradient "
                      f"sum (fp64 oracle, {cores} threads of {k} samples, partial sums added "
                      f"in order), {dt:.1f} s"}


def mean_test_loss(net, torch, xtd, ytd):
    """Mean loss over the test set at the net's current weights."""
    loss = torch.empty(ytd.numel(), device="cuda")
    net.forward_backward(xtd, ytd, loss=loss)
    torch.cuda.synchronize()
    return float(loss.double().mean())


def row_quality(initial, final):
    """The row's training converged: finite and below the loss at the initial
    weights (a saturated Hogwild run ends far above it)."""
    return {"test_loss_initial": initial, "test_loss_final": final,
            "converging": bool(final == final and final < initial)}


def train_row(chaos, wl, torch, name, xd, yd, x, y, xtd, ytd, steps, with_cpu, replicas=None):
    """Training throughput of one net over the resident training set (atomic
    pushes, lr 1e-3, the library's default worker count: one worker per
    compute unit), and the test loss before and after.  replicas = (r, m):
    the workers read r weight replicas refreshed every m samples
    (chaos_set_replicas)."""
    layers = wl.NETS[name]
    p0 = wl.init_params(layers)
    net = chaos.Net(layers, p0)
    if replicas:
        net.set_replicas(*replicas)
    workers = net.default_workers
    flops, _ = train_flops_per_sample(layers)
    n = yd.numel()
    initial = mean_test_loss(net, torch, xtd, ytd)
    net.train_epoch(xd, yd, 1e-3, mode=chaos.HOGWILD_ATOMIC, workers=workers)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(steps):
        net.train_epoch(xd, yd, 1e-3, mode=chaos.HOGWILD_ATOMIC, workers=workers)
    b.record(stream)
    torch.cuda.synchronize()
    sps = n * steps / (a.elapsed_time(b) / 1e3)
    tflops = sps * flops / 1e12
    row = {"samples_per_s": sps, "workers": workers, "resident_workers": net.max_workers,
           "train_flop_per_sample": flops,
           "tflops": tflops, "frac_fp32_peak": tflops / PEAK_FP32_TFLOPS,
           "ms_per_epoch": a.elapsed_time(b) / steps,
           "quality": row_quality(initial, mean_test_loss(net, torch, xtd, ytd))}
    if replicas:
        row["replicas"] = {"copies": replicas[0], "refresh_every": replicas[1]}
    if with_cpu:
        row["cpu_oracle"] = cpu_baseline(layers, p0, x, y, budget_s=3.0)
    return row


def worker_sweep(chaos, wl, torch):
    """Training samples/s against the number of concurrent Hogwild workers
    (atomic pushes, lr 1e-3), one timed epoch per point after one warm-up
    epoch; small worker counts run on a prefix of the training set."""
    x, y = wl.train_set(60000)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    out = {}
    for name in ("small", "medium", "large"):
        layers = wl.NETS[name]
        net = chaos.Net(layers, wl.init_params(layers))
        flops, _ = train_flops_per_sample(layers)
        counts, p = [], 1
        while p < net.worker_limit:
            counts.append(p)
            p *= 2
        counts = sorted(set(counts + [net.max_workers, net.worker_limit]))
        rows = []
        for w in counts:
            n = min(60000, max(2000, 500 * w))
            for _ in range(2):
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                net.train_epoch(xd[:n], yd[:n], 1e-3, mode=chaos.HOGWILD_ATOMIC, workers=w)
                b.record()
                torch.cuda.synchronize()
            sps = n / (a.elapsed_time(b) / 1e3)
            rows.append({"workers": w, "samples": n, "samples_per_s": sps,
                         "tflops": sps * flops / 1e12,
                         "kernel": "fused" if w <= net.max_workers else "one-wavefront generic"})
            print(f"sweep {name}: {w} workers, {sps:,.0f} samples/s", file=sys.stderr, flush=True)
        out[name] = {"max_workers": net.max_workers, "worker_limit": net.worker_limit,
                     "train_flop_per_sample": flops, "points": rows}
    return {"sweep": "Hogwild training throughput vs concurrent workers", "nets": out}


def model_fit(chaos, wl, torch, name):
    """Fit the performance model of Section III-C (paper_1506_09067_amd.perfmodel)
    to this GPU: Training epochs timed at 1, 2, 4, ... workers, the forward
    rate from the 10,000-sample test set, then MemoryContention(p).  The
    accuracy alpha is measured three ways: worker counts left out of the fit
    (every other power of two below the largest), extrapolation (a fit on the
    counts up to a quarter of the resident workers predicting the larger
    ones), and a whole Training + Validation + Testing session of two epochs
    at every resident worker.  The what-if table is the Table III analog, in
    seconds, at the resident worker count and at twice that; twice is beyond
    what the fused kernel holds, so that column is the model's answer for a
    kernel that could, and the epochs the library actually runs there (one-
    wavefront generic workers) are measured beside it."""
    from paper_1506_09067_amd import perfmodel as pm
    layers = wl.NETS[name]
    p0 = wl.init_params(layers)
    x, y = wl.train_set(60000)
    xt, yt = wl.test_set(10000)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    xtd, ytd = torch.from_numpy(xt).cuda(), torch.from_numpy(yt).cuda()
    flops, fwd = train_flops_per_sample(layers)
    net = chaos.Net(layers, p0)
    pmax = net.max_workers

    def timed(fn, reps=1):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / 1e3 / reps

    epochs = {}
    p = 1
    while p <= pmax:
        n = min(60000, max(2000, 500 * p))
        net.set_params(torch.from_numpy(p0).cuda())
        secs = timed(lambda: net.train_epoch(xd[:n], yd[:n], 1e-3, workers=p))
        epochs[p] = (n, secs)
        p *= 2
    t_fwd_one = timed(lambda: net.evaluate(xtd, ytd), 3) / 10000 * pmax
    n1, s1 = epochs[1]
    ps = sorted(epochs)
    held = [q for k, q in enumerate(ps) if k % 2 == 1 and q != ps[-1]]  # interior points
    fit_part = pm.fit(fwd, flops - fwd, s1 / n1, t_fwd_one,
                      {q: v for q, v in epochs.items() if q not in held})
    loo = {q: pm.accuracy(epochs[q][1], fit_part.predict_training(epochs[q][0], 1, q))
           for q in held}
    # extrapolation: fit on p <= pmax / 4 only, predict the two largest counts
    low = {q: v for q, v in epochs.items() if q <= pmax // 4}
    fit_low = pm.fit(fwd, flops - fwd, s1 / n1, t_fwd_one, low)
    extrap = {q: {"measured_s": epochs[q][1],
                  "predicted_s": fit_low.predict_training(epochs[q][0], 1, q),
                  "alpha_pct": pm.accuracy(epochs[q][1], fit_low.predict_training(epochs[q][0], 1, q))}
              for q in sorted(epochs) if q > pmax // 4}
    model = pm.fit(fwd, flops - fwd, s1 / n1, t_fwd_one, epochs)
    # beyond residency the library runs one-wavefront generic workers, a
    # different kernel: measured here next to the fused-kernel model
    beyond = {}
    for q in (2 * pmax, 4 * pmax):
        if q <= net.worker_limit:
            net.set_params(torch.from_numpy(p0).cuda())
            secs = timed(lambda: net.train_epoch(xd, yd, 1e-3, workers=q))
            beyond[str(q)] = {"measured_s": secs, "model_s": model.predict_training(60000, 1, q),
                              "kernel": "one-wavefront generic"}
    # a whole session: Training + Validation + Testing, two epochs
    net.set_params(torch.from_numpy(p0).cuda())
    sess = timed(lambda: net.train_session(xd, yd, xtd, ytd, 2, 1e-3, 1.0))
    sess_pred = model.predict(60000, 10000, 2, pmax)
    table = {}
    for p in (pmax, 2 * pmax):
        table[str(p)] = {f"{i // 1000}k/{it // 1000}k": {str(ep): model.predict(i, it, ep, p)
                                                         for ep in (70, 140, 280, 560)}
                         for i, it in ((60000, 10000), (120000, 20000), (240000, 40000))}
    return {
        "model": "Section III-C, refitted on MI355X", "net": name, "resident_workers": pmax,
        "FProp": fwd, "BProp": flops - fwd, "s_flop_per_s": pm.PEAK_FP32_PER_CU,
        "penalty_train": model.penalty_train, "penalty_fwd": model.penalty_fwd,
        "t_train_one_worker_s": model.t_train(), "t_fwd_one_worker_s": model.t_fwd(),
        "memory_contention_s": {str(q): v for q, v in model.contention.items()},
        "measured_training_epochs": {str(q): {"samples": n, "seconds": t} for q, (n, t) in epochs.items()},
        "alpha_left_out_pct": {str(q): v for q, v in loo.items()},
        "extrapolation_from_quarter_residency": {str(q): v for q, v in extrap.items()},
        "beyond_residency_measured_epoch": beyond,
        "sequential_ops_s": model.t_seq(60000, 10000, 1),
        "session_2_epochs": {"measured_s": sess, "predicted_s": sess_pred,
                             "alpha_pct": pm.accuracy(sess, sess_pred)},
        "what_if_seconds": table,
    }


def training_session(chaos, wl, torch, name, epochs, lr, decay, seq_epochs):
    """A whole training session (Section III-A.1): per epoch Training over the
    60,000-sample set, Validation on it and Testing on the 10,000-sample set,
    with every resident worker (Hogwild, atomic pushes), timed as one call;
    then the same session with one worker (sequential per-sample SGD) for
    `seq_epochs` epochs, for the per-epoch comparison and the speed-up."""
    layers = wl.NETS[name]
    p0 = wl.init_params(layers)
    x, y = wl.train_set(60000)
    xt, yt = wl.test_set(10000)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    xtd, ytd = torch.from_numpy(xt).cuda(), torch.from_numpy(yt).cuda()

    def run(mode, n_epochs):
        net = chaos.Net(layers, p0)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        st = net.train_session(xd, yd, xtd, ytd, n_epochs, lr, decay, mode=mode)
        b.record()
        torch.cuda.synchronize()
        rows = [{"epoch": e + 1, "train_loss": float(r[0]), "train_wrong": int(r[1]),
                 "test_wrong": int(r[2]), "test_loss": float(r[3]), "diverged": bool(r[4])}
                for e, r in enumerate(st.cpu().tolist())]
        return rows, a.elapsed_time(b) / 1e3, net.max_workers

    hog, t_hog, workers = run(chaos.HOGWILD_ATOMIC, epochs)
    seq, t_seq, _ = run(chaos.SEQUENTIAL, seq_epochs) if seq_epochs else ([], None, 1)
    out = {"session": f"{name} net, 60000 training + 10000 test samples, lr {lr} x {decay}/epoch",
           "hogwild": {"workers": workers, "epochs": epochs, "seconds": t_hog, "per_epoch": hog}}
    if seq_epochs:
        out["sequential"] = {"workers": 1, "epochs": seq_epochs, "seconds": t_seq, "per_epoch": seq}
        out["speedup_per_epoch"] = (t_seq / seq_epochs) / (t_hog / epochs)
    return out


def delay_sweep(chaos, wl, torch, epochs=5, lr=1e-3, decay=0.9):
    """Delayed pushes on the small net (chaos_set_push_delay): training
    samples/s at every resident worker for push delays k = 1 (the per-layer
    push), 2, 4, ..., 64 (two timed 60,000-sample epochs each, after one
    warm-up epoch), and the test-set loss and wrong count after `epochs`
    epochs (lr decaying by `decay` per epoch) against sequential per-sample
    SGD on the same data, with the push of a k-sample sum at lr and at lr / k
    (the mean of the k gradients)."""
    layers = wl.NETS["small"]
    p0 = wl.init_params(layers)
    x, y = wl.train_set(60000)
    xt, yt = wl.test_set(10000)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    xtd, ytd = torch.from_numpy(xt).cuda(), torch.from_numpy(yt).cuda()
    flops, _ = train_flops_per_sample(layers)

    def quality(net, mode, lr=lr):
        for e in range(epochs):
            net.train_epoch(xd, yd, lr * decay ** e, mode=mode, workers=net.max_workers)
        loss = torch.empty(10000, device="cuda")
        net.forward_backward(xtd, ytd, loss=loss)
        wrong = net.evaluate(xtd, ytd)
        torch.cuda.synchronize()
        return float(loss.double().mean()), int(wrong.item())

    seq = quality(chaos.Net(layers, p0), chaos.SEQUENTIAL)
    initial = mean_test_loss(chaos.Net(layers, p0), torch, xtd, ytd)
    points = []
    for k in (1, 2, 4, 8, 16, 32, 64):
        net = chaos.Net(layers, p0)
        net.set_push_delay(k)
        net.train_epoch(xd, yd, lr, workers=net.max_workers)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(2):
            net.train_epoch(xd, yd, lr, workers=net.max_workers)
        b.record()
        torch.cuda.synchronize()
        sps = 2 * 60000 / (a.elapsed_time(b) / 1e3)
        q = quality(_fresh(chaos, layers, p0, k), chaos.HOGWILD_ATOMIC)
        qm = quality(_fresh(chaos, layers, p0, k), chaos.HOGWILD_ATOMIC, lr / k)
        points.append({"push_delay": k, "workers": net.max_workers, "samples_per_s": sps,
                       "tflops": sps * flops / 1e12, "test_loss": q[0], "test_wrong": q[1],
                       "test_loss_lr_over_k": qm[0], "test_wrong_lr_over_k": qm[1],
                       # a run that ends above the untrained loss has diverged:
                       # its rate is not a speed-up
                       "converging": bool(q[0] < initial),
                       "converging_lr_over_k": bool(qm[0] < initial)})
    return {"sweep": "small net, delayed pushes (atomic Hogwild, every resident worker)",
            "epochs_for_quality": epochs, "lr": lr, "decay": decay,
            "initial_test_loss": initial,
            "sequential": {"test_loss": seq[0], "test_wrong": seq[1]}, "points": points}


def _fresh(chaos, layers, p0, k):
    net = chaos.Net(layers, p0)
    net.set_push_delay(k)
    return net


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--net", default="large")
    ap.add_argument("--workers", type=int, default=0)
    ap.add_argument("--mode", default="atomic", choices=["atomic", "racy", "sequential"])
    ap.add_argument("--samples", type=int, default=60000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-rows", action="store_true")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the benchmark line, print one JSON line with training "
                         "throughput against the number of Hogwild workers for the small, "
                         "medium and large nets")
    ap.add_argument("--model", action="store_true",
                    help="instead of the benchmark line, fit the Section III-C performance "
                         "model to measurements of --net and print its parameters, its "
                         "prediction accuracy and a what-if table as one JSON line")
    ap.add_argument("--session", type=int, default=0, metavar="EPOCHS",
                    help="instead of the benchmark line, run a whole Training + Validation + "
                         "Testing session of EPOCHS epochs of --net with every resident worker "
                         "(and --seq-epochs epochs with one worker) and print per-epoch "
                         "statistics as one JSON line")
    ap.add_argument("--delay-sweep", action="store_true",
                    help="instead of the benchmark line, print one JSON line with the small "
                         "net's training throughput and final test loss against the push "
                         "delay (chaos_set_push_delay)")
    ap.add_argument("--seq-epochs", type=int, default=1)
    ap.add_argument("--decay", type=float, default=1.0)
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB (calibrates "
                         "the FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.copy_mib:
        import torch
        n = args.copy_mib * (1 << 20) // 4
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4}), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the path shards by samples across GPUs, see the design notes)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_1506_09067_amd import chaos, workloads as wl

    torch.cuda.set_device(0)
    if args.sweep:
        print(json.dumps(worker_sweep(chaos, wl, torch)), flush=True)
        return
    if args.model:
        print(json.dumps(model_fit(chaos, wl, torch, args.net)), flush=True)
        return
    if args.delay_sweep:
        print(json.dumps(delay_sweep(chaos, wl, torch)), flush=True)
        return
    if args.session:
        print(json.dumps(training_session(chaos, wl, torch, args.net, args.session, 1e-3,
                                          args.decay, args.seq_epochs)), flush=True)
        return
    layers = wl.NETS[args.net]
    p0 = wl.init_params(layers)
    x, y = wl.train_set(args.samples)
    xd = torch.from_numpy(x).cuda()
    yd = torch.from_numpy(y).cuda()
    xt, yt = wl.test_set(10000)
    xtd, ytd = torch.from_numpy(xt).cuda(), torch.from_numpy(yt).cuda()
    net = chaos.Net(layers, p0)
    initial_test_loss = mean_test_loss(net, torch, xtd, ytd)
    mode = {"atomic": chaos.HOGWILD_ATOMIC, "racy": chaos.HOGWILD_RACY,
            "sequential": chaos.SEQUENTIAL}[args.mode]
    workers = args.workers or net.default_workers
    if mode == chaos.SEQUENTIAL:
        workers = 1
    flops, fwd_flops = train_flops_per_sample(layers)

    for _ in range(args.warmup):
        net.train_epoch(xd, yd, 1e-3, mode=mode, workers=workers)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t0 = time.perf_counter()
    for s in range(args.steps):
        ev[s][0].record(stream)
        net.train_epoch(xd, yd, 1e-3, mode=mode, workers=workers)
        ev[s][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    launch_ms = [a.elapsed_time(b) for a, b in ev]
    total_ms = sum(launch_ms)
    value = args.samples * args.steps / (total_ms / 1e3)
    avg_launch_s = total_ms / 1e3 / args.steps
    achieved = flops * args.samples / avg_launch_s / 1e12
    traffic = measured_traffic(args.net, workers, args.samples)
    w = net.get_params()
    torch.cuda.synchronize()
    finite = bool(torch.isfinite(w).all().item())
    headline_quality = row_quality(initial_test_loss, mean_test_loss(net, torch, xtd, ytd))

    rows = None
    if not args.no_rows:
        rows = {}
        for name in ("small", "medium", "large_table1"):
            if name != args.net:
                rows[f"train_{name}_{args.samples}"] = train_row(
                    chaos, wl, torch, name, xd, yd, x, y, xtd, ytd, args.steps,
                    not args.no_cpu_baseline)
        rows[f"train_small_replicas_8x8_{args.samples}"] = train_row(
            chaos, wl, torch, "small", xd, yd, x, y, xtd, ytd, args.steps, False, replicas=(8, 8))
        xb, yb = wl.batch_set(16384)
        xbd, ybd = torch.from_numpy(xb).cuda(), torch.from_numpy(yb).cuda()
        g = torch.empty(net.n_params, device="cuda")
        net.forward_backward(xbd, ybd, grad_sum=g)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        net.forward_backward(xbd, ybd, grad_sum=g)
        b.record(stream)
        torch.cuda.synchronize()
        bg_sps = 16384 / (a.elapsed_time(b) / 1e3)
        bg_flops = flops - 2 * net.n_params  # forward + backward, no update
        rows["batch_gradient_16384"] = {"samples_per_s": bg_sps, "ms": a.elapsed_time(b),
                                        "flop_per_sample": bg_flops,
                                        "tflops": bg_sps * bg_flops / 1e12,
                                        "frac_fp32_peak": bg_sps * bg_flops / 1e12 / PEAK_FP32_TFLOPS}
        if not args.no_cpu_baseline:
            rows["batch_gradient_16384"]["cpu_oracle"] = cpu_batch_baseline(layers, p0, xb, yb)
        net.evaluate(xtd, ytd)
        torch.cuda.synchronize()
        a.record(stream)
        wrong = net.evaluate(xtd, ytd)
        b.record(stream)
        torch.cuda.synchronize()
        rows["test_forward_10000"] = {"samples_per_s": 10000 / (a.elapsed_time(b) / 1e3),
                                      "ms": a.elapsed_time(b),
                                      "tflops": fwd_flops * 10000 / (a.elapsed_time(b) / 1e3) / 1e12,
                                      "frac_fp32_peak": fwd_flops * 10000 / (a.elapsed_time(b) / 1e3)
                                      / 1e12 / PEAK_FP32_TFLOPS,
                                      "n_wrong": int(wrong.item())}

    upd = update_stream(torch, net.n_params, value) if mode != chaos.SEQUENTIAL else None
    cpu = None if args.no_cpu_baseline else cpu_baseline(layers, p0, x, y)
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "training samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": total_ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"CHAOS Training epoch, {args.net} net, {args.samples} synthetic "
                               f"29x29 samples, Hogwild ({args.mode}) with {workers} workers, lr 1e-3",
                   "net": args.net, "samples_per_step": args.samples, "workers": workers,
                   "mode": args.mode, "params": net.n_params,
                   "train_flop_per_sample": flops},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_FP32_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_FP32_TFLOPS, "traffic": traffic},
        "update_stream": upd,
        "cpu_baseline": cpu,
        "rows": rows,
        "wall_s": wall,
        "weights_finite": finite,
        "quality": headline_quality,
        "launch_ms": launch_ms,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
