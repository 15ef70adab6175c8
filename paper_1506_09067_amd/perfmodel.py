"""The CHAOS speed-up formula and performance model (Sections III-B and III-C),
refitted to measurements of this implementation on one MI355X.

Section III-B gives the speed-up of p processing units over one,
    S_p = T_1 / T_p,
with T_p = (a i + b it + c) + (d + e i / p_i + f i / p_i + g it / p_it) ep,
p_i = min(p, i), p_it = min(p, it): a, b, c set-up work per image / per
test image / once, d per-epoch serialisation, e one training image
(forward + back-propagation), f one validation image, g one test image.

Section III-C models the execution time as computation plus memory
contention,
    T = T_comp + T_mem,
    T_comp = ((Prep + 4 i + 2 it + 10 ep) / s
              + ((FProp + BProp) / s) (i / p_i) ep
              + (FProp / s) (i / p_i) ep
              + (FProp / s) (it / p_it) ep) * CPI * OperationFactor,
    T_mem = MemoryContention(p) * i * ep / p,
where s is the speed of one processing unit, FProp / BProp the operation
counts of forward and back-propagation, CPI * OperationFactor a penalty
fitted per architecture, and MemoryContention(p) the time lost per round of
p images when p workers update the shared weights.

On the GPU a processing unit is one Hogwild worker.  The refit takes
  * FProp, BProp: the dense FLOP counts of one sample (forward, and the rest
    of a training step);
  * s: the FP32 matrix peak of one compute unit (157.3 TFLOP/s / 256);
  * CPI * OperationFactor: from the per-sample time of a single worker
    (no contention), so that T_comp reproduces it exactly;
  * the forward penalty likewise from the measured forward (Validation /
    Testing) rate;
  * MemoryContention(p): from the measured Training epoch time at p workers,
    the excess over T_comp per round of p images.
Prediction at a worker count that was not measured interpolates
MemoryContention linearly in log p; beyond the largest measured p it
continues the power law of the last measured interval (contention grows
steeply once the update stream saturates), below the smallest it holds the
first value.  The prediction accuracy is the paper's
alpha = |measured - predicted| / predicted * 100 %.

Pure Python: no GPU code; bench.py --model supplies the measurements.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

PEAK_FP32_PER_CU = 157.3e12 / 256  # FLOP/s of one compute unit (one worker's unit)


def speedup(p, i, it, ep, a, b, c, d, e, f, g):
    """S_p of Section III-B for p processing units."""
    pi, pit = min(p, i), min(p, it)
    seq = a * i + b * it + c
    t1 = seq + (d + e * i + f * i + g * it) * ep
    tp = seq + (d + e * i / pi + f * i / pi + g * it / pit) * ep
    return t1 / tp


def accuracy(measured, predicted):
    """alpha = |mu - psi| / psi * 100 % (Section IV, prediction accuracy)."""
    return abs(measured - predicted) / predicted * 100.0


@dataclass
class Model:
    """Section III-C with per-architecture constants fitted on the GPU."""
    fprop: float                  # FLOP of one forward pass
    bprop: float                  # FLOP of the rest of one training step
    s: float = PEAK_FP32_PER_CU   # FLOP/s of one processing unit
    penalty_train: float = 1.0    # CPI * OperationFactor of a training step
    penalty_fwd: float = 1.0      # the same for a forward pass
    prep: float = 0.0             # Prep: operations of the sequential preparation
    contention: dict = field(default_factory=dict)  # p -> MemoryContention(p), s per round

    def t_train(self):
        """Seconds per training sample of one worker without contention."""
        return (self.fprop + self.bprop) / self.s * self.penalty_train

    def t_fwd(self):
        """Seconds per forward-only sample of one worker."""
        return self.fprop / self.s * self.penalty_fwd

    def memory_contention(self, p):
        if not self.contention:
            return 0.0
        ps = sorted(self.contention)
        if p <= ps[0]:
            return self.contention[ps[0]]
        if p >= ps[-1]:
            last = self.contention[ps[-1]]
            if len(ps) > 1 and last > 0 and self.contention[ps[-2]] > 0 and p > ps[-1]:
                k = math.log(last / self.contention[ps[-2]]) / math.log(ps[-1] / ps[-2])
                return last * (p / ps[-1]) ** max(k, 0.0)
            return last
        for lo, hi in zip(ps, ps[1:]):
            if lo <= p <= hi:
                w = (math.log(p) - math.log(lo)) / (math.log(hi) - math.log(lo))
                return (1 - w) * self.contention[lo] + w * self.contention[hi]
        raise AssertionError("unreachable")

    def t_seq(self, i, it, ep):
        """Row (2): the sequential operations (Prep + 4 i + 2 it + 10 ep) / s
        under the training penalty.  On the GPU Prep is 0 (the weights are
        drawn by the caller) and the rest is a few microseconds, but the term
        is kept as the paper states it."""
        return (self.prep + 4 * i + 2 * it + 10 * ep) / self.s * self.penalty_train

    def t_comp(self, i, it, ep, p, validate=True):
        """Rows (2)-(6) without T_mem: the sequential operations, then
        Training, Validation (optional) and Testing over ep epochs with p
        workers."""
        pi, pit = min(p, i), min(p, it)
        t = self.t_seq(i, it, ep)
        t += self.t_train() * (i / pi) * ep
        if validate:
            t += self.t_fwd() * (i / pi) * ep
        t += self.t_fwd() * (it / pit) * ep
        return t

    def t_mem(self, i, ep, p):
        return self.memory_contention(p) * i * ep / p

    def predict(self, i, it, ep, p, validate=True):
        return self.t_comp(i, it, ep, p, validate) + self.t_mem(i, ep, p)

    def predict_training(self, i, ep, p):
        """Training passes only (what bench.py times)."""
        pi = min(p, i)
        return self.t_train() * (i / pi) * ep + self.t_mem(i, ep, p)


def fit(fprop, bprop, t_train_one, t_fwd_one, train_epochs, s=PEAK_FP32_PER_CU):
    """Fit the model.

    t_train_one: seconds per training sample of one worker alone;
    t_fwd_one: seconds per forward sample of one worker (may be derived from a
    many-worker forward rate times the worker count: forward passes do not
    contend);
    train_epochs: {p: (i, seconds)} measured Training epochs over i samples
    with p workers.
    """
    m = Model(fprop=fprop, bprop=bprop, s=s)
    m.penalty_train = t_train_one * s / (fprop + bprop)
    m.penalty_fwd = t_fwd_one * s / fprop
    for p, (i, secs) in sorted(train_epochs.items()):
        comp = m.t_train() * i / min(p, i)
        m.contention[p] = max(0.0, (secs - comp) * p / i)
    return m
