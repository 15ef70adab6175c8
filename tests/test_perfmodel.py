"""The speed-up formula (Section III-B) and the performance model (Section
III-C) as refitted for the GPU: closed forms and a planted-parameter fit."""
import math

import pytest

from paper_1506_09067_amd import perfmodel as pm


def test_speedup_is_linear_without_sequential_work():
    # only the per-image terms: S_p = p while p <= min(i, it)
    for p in (1, 2, 7, 64, 244):
        assert pm.speedup(p, 60000, 10000, 15, 0, 0, 0, 0, 3.0, 1.0, 1.0) == pytest.approx(p)


def test_speedup_saturates_at_the_image_counts():
    # p beyond both image counts: every unit holds one image, no further gain
    s_big = pm.speedup(10 ** 6, 100, 100, 1, 0, 0, 0, 0, 1.0, 1.0, 1.0)
    assert s_big == pytest.approx(100.0)
    assert pm.speedup(10 ** 7, 100, 100, 1, 0, 0, 0, 0, 1.0, 1.0, 1.0) == pytest.approx(s_big)


def test_speedup_amdahl_limit_from_sequential_work():
    # sequential share q of T_1: S_p -> 1 / q as p grows (i, it large)
    i, it, ep = 10 ** 9, 10 ** 9, 1
    a = 1.0  # per-image preparation: sequential
    e = 9.0  # per-image training: parallel
    q = a * i / (a * i + e * i)
    assert pm.speedup(10 ** 8, i, it, ep, a, 0, 0, 0, e, 0, 0) == pytest.approx(1 / q, rel=1e-6)


def test_accuracy_is_the_relative_deviation_from_the_prediction():
    assert pm.accuracy(115.4, 100.0) == pytest.approx(15.4)
    assert pm.accuracy(84.6, 100.0) == pytest.approx(15.4)
    assert pm.accuracy(5.0, 5.0) == 0.0


def test_model_with_one_worker_is_the_per_sample_sum():
    m = pm.Model(fprop=2e6, bprop=4e6, s=1e9, penalty_train=3.0, penalty_fwd=2.0)
    assert m.t_train() == pytest.approx(6e6 / 1e9 * 3.0)
    assert m.t_fwd() == pytest.approx(2e6 / 1e9 * 2.0)
    i, it, ep = 1000, 200, 3
    seq = (4 * i + 2 * it + 10 * ep) / 1e9 * 3.0  # row (2), Prep = 0
    assert m.t_seq(i, it, ep) == pytest.approx(seq)
    want = (m.t_train() * i + m.t_fwd() * i + m.t_fwd() * it) * ep
    assert m.predict(i, it, ep, 1) == pytest.approx(seq + want)
    # no contention: p workers divide every term but the sequential one
    assert m.predict(i, it, ep, 8) == pytest.approx(m.t_comp(i, it, ep, 8))
    assert m.t_comp(i, it, ep, 8) == pytest.approx(seq + want / 8)
    assert m.predict(i, it, ep, 10 ** 6) == pytest.approx(
        seq + (m.t_train() + m.t_fwd() + m.t_fwd()) * ep)
    m.prep = 5e5
    assert m.t_seq(i, it, ep) == pytest.approx((5e5 + 4 * i + 2 * it + 10 * ep) / 1e9 * 3.0)


def test_memory_term_follows_the_formula():
    m = pm.Model(fprop=1.0, bprop=1.0, contention={4: 2e-3})
    assert m.t_mem(60000, 15, 4) == pytest.approx(2e-3 * 60000 * 15 / 4)


def test_contention_interpolates_in_log_p_and_extrapolates_the_last_power_law():
    m = pm.Model(fprop=1.0, bprop=1.0, contention={4: 1.0, 64: 3.0})
    assert m.memory_contention(2) == 1.0                  # held below the first point
    assert m.memory_contention(16) == pytest.approx(2.0)  # halfway in log p
    assert m.memory_contention(8) == pytest.approx(1.5)
    # beyond the last point: MC grows as p^k with k from the last interval
    k = math.log(3.0) / math.log(16.0)
    assert m.memory_contention(128) == pytest.approx(3.0 * 2 ** k)
    assert m.memory_contention(1024) == pytest.approx(3.0 * 16 ** k)
    # a vanishing first value cannot define a power law: hold
    flat = pm.Model(fprop=1.0, bprop=1.0, contention={4: 0.0, 64: 3.0})
    assert flat.memory_contention(256) == 3.0


def test_fit_recovers_planted_parameters():
    fprop, bprop, s = 3.0e6, 6.0e6, 6.0e11
    truth = pm.Model(fprop=fprop, bprop=bprop, s=s, penalty_train=4.5, penalty_fwd=2.5,
                     contention={1: 0.0, 4: 1e-6, 16: 4e-6, 64: 2e-5, 256: 1e-4})
    epochs = {p: (60000, truth.predict_training(60000, 1, p)) for p in truth.contention}
    m = pm.fit(fprop, bprop, truth.t_train(), truth.t_fwd(), epochs, s=s)
    assert m.penalty_train == pytest.approx(4.5)
    assert m.penalty_fwd == pytest.approx(2.5)
    for p, c in truth.contention.items():
        assert m.contention[p] == pytest.approx(c, rel=1e-9, abs=1e-15)
    for p in (2, 8, 32, 128):
        assert m.predict_training(60000, 1, p) == pytest.approx(truth.predict_training(60000, 1, p))
    # and a session prediction from the fitted model equals the planted one
    assert m.predict(60000, 10000, 15, 256) == pytest.approx(truth.predict(60000, 10000, 15, 256))


def test_doubling_epochs_or_images_doubles_the_time():
    # up to the sequential term of row (2), which is a few microseconds here
    m = pm.Model(fprop=1e6, bprop=2e6, s=1e9, contention={240: 1e-4})
    base = m.predict(60000, 10000, 70, 240)
    assert m.predict(60000, 10000, 140, 240) == pytest.approx(2 * base, rel=1e-4)
    assert m.predict(120000, 20000, 70, 240) == pytest.approx(2 * base, rel=1e-4)
    assert math.isfinite(m.predict(60000, 10000, 70, 480))
