"""Pins of the oracle's losses, gradients and SGD pass (CPU only)."""
import math

import numpy as np
import pytest

from oracle import prng, sgd

RNG = np.random.default_rng(1234)


def test_closed_forms_at_zero_margin():
    y = np.array([1.0, -1.0])
    m = np.zeros(2)
    assert np.allclose(sgd.loss_value(y * m, "logistic"), math.log(2.0))
    assert np.allclose(sgd.loss_coef(m, y, "logistic"), -y / 2)
    assert np.allclose(sgd.loss_value(y * m, "hinge"), 1.0)
    assert np.allclose(sgd.loss_coef(m, y, "hinge"), -y)


def test_logistic_coef_extremes_do_not_overflow():
    m = np.array([800.0, -800.0])
    y = np.array([1.0, 1.0])
    c = sgd.loss_coef(m, y, "logistic")
    assert c[0] == pytest.approx(0.0, abs=1e-300) and c[1] == pytest.approx(-1.0)
    assert np.isfinite(sgd.loss_value(y * m, "logistic")).all()


@pytest.mark.parametrize("loss", ["logistic", "hinge"])
def test_coef_is_loss_derivative(loss):
    y = np.array([1.0, -1.0, 1.0, -1.0])
    m = np.array([0.3, -0.7, 2.5, 0.4])       # hinge: away from y m = 1
    h = 1e-6
    num = (sgd.loss_value(y * (m + h), loss) - sgd.loss_value(y * (m - h), loss)) / (2 * h)
    assert np.allclose(sgd.loss_coef(m, y, loss), num, rtol=1e-6, atol=1e-9)


def test_hinge_kink_has_zero_subgradient():
    assert sgd.loss_coef(np.array([1.0, -1.0]), np.array([1.0, -1.0]), "hinge").tolist() == [0.0, 0.0]


def _batch_objective(w, X, y, loss, l2):
    return np.mean(sgd.loss_value(y * (X @ w), loss)) + 0.5 * l2 * w @ w


@pytest.mark.parametrize("loss,l2", [("logistic", 0.0), ("logistic", 0.3), ("hinge", 0.1)])
def test_single_step_is_minus_lr_times_finite_difference_gradient(loss, l2):
    D, B = 6, 4
    X = RNG.standard_normal((B, D))
    y = np.where(RNG.random(B) < 0.5, -1.0, 1.0)
    w0 = 0.1 * RNG.standard_normal(D)
    if loss == "hinge":
        assert np.all(np.abs(y * (X @ w0) - 1) > 1e-3)
    sched = np.arange(B)
    lr = 0.7
    w1 = sgd.sgd_pass_dense(w0, X, y, sched, batch=B, loss=loss, lr_kind="const", lr0=lr, l2=l2, rnd=0)
    h = 1e-6
    g = np.array([(_batch_objective(w0 + h * e, X, y, loss, l2) -
                   _batch_objective(w0 - h * e, X, y, loss, l2)) / (2 * h) for e in np.eye(D)])
    assert np.allclose(w1, w0 - lr * g, rtol=1e-6, atol=1e-8)


def test_hand_computed_two_steps():
    # x = (1, 2), y = +1, eta = 0.5, w0 = 0, logistic:
    # step 1: m = 0, c = -1/2, w1 = 0.5 * (1, 2) / 2 = (0.25, 0.5)
    # step 2: m = 1.25, c = -1 / (1 + e^1.25), w2 = w1 - 0.5 * c * (1, 2)
    X = np.array([[1.0, 2.0]])
    y = np.array([1.0])
    w1 = sgd.sgd_pass_dense(np.zeros(2), X, y, np.array([0]), batch=1, loss="logistic",
                            lr_kind="const", lr0=0.5, l2=0.0, rnd=0)
    assert np.allclose(w1, [0.25, 0.5])
    w2 = sgd.sgd_pass_dense(w1, X, y, np.array([0]), batch=1, loss="logistic",
                            lr_kind="const", lr0=0.5, l2=0.0, rnd=1)
    c = -1.0 / (1.0 + math.exp(1.25))
    assert np.allclose(w2, [0.25 - 0.5 * c, 0.5 - 0.5 * c * 2])


def test_step_counter_spans_rounds():
    # one sample, one step per round: round r uses t = r + 1, so from w = 0 the
    # hinge step is eta_t * y * x with eta_t = lr0 / sqrt(r + 1).
    X = np.array([[0.5, -1.0, 2.0]])
    y = np.array([-1.0])
    for r in (0, 1, 5, 99):
        w = sgd.sgd_pass_dense(np.zeros(3), X, y, np.array([0]), batch=1, loss="hinge",
                               lr_kind="inv_sqrt", lr0=0.5, l2=0.0, rnd=r)
        assert np.allclose(w, 0.5 / math.sqrt(r + 1) * y[0] * X[0])
    # and within a round t = r * ceil(S / B) + k + 1: S = 5, B = 2 -> 3 steps.
    assert sgd.n_steps(5, 2) == 3 and sgd.n_steps(4, 2) == 2 and sgd.n_steps(0, 2) == 0


def test_round_steps_rule():
    # local_steps = 0: round r is pass r; L dividing K: consecutive blocks of
    # L steps of the sequence of passes
    assert sgd.round_steps(7, 0, 5) == (7, 0, 5)
    assert [sgd.round_steps(r, 2, 6) for r in range(4)] == [(0, 0, 2), (0, 2, 4), (0, 4, 6), (1, 0, 2)]
    assert [sgd.round_steps(r, 1, 3)[:2] for r in range(7)] == [(0, 0), (0, 1), (0, 2), (1, 0), (1, 1), (1, 2), (2, 0)]
    with pytest.raises(ValueError):
        sgd.round_steps(0, 4, 6)


def test_step_ranges_compose_to_the_pass():
    # running steps [0, a) then [a, K) of a pass is the pass; the step
    # counter t of the second block continues (pass q: t = q K + k + 1)
    rng = np.random.default_rng(5)
    S, D, B = 11, 4, 2
    X, y = rng.standard_normal((S, D)), np.where(rng.random(S) < 0.5, -1.0, 1.0)
    sched = rng.permutation(S)
    kw = dict(batch=B, loss="logistic", lr_kind="inv_sqrt", lr0=0.3, l2=0.01, rnd=3)
    w0 = rng.standard_normal(D)
    full = sgd.sgd_pass_dense(w0, X, y, sched, **kw)
    K = sgd.n_steps(S, B)
    for a in range(K + 1):
        part = sgd.sgd_pass_dense(w0, X, y, sched, steps=(0, a), **kw)
        part = sgd.sgd_pass_dense(part, X, y, sched, steps=(a, K), **kw)
        assert np.array_equal(part, full)
    # one step from w = 0 on a one-sample pass is eta_t y x with t = q K + k + 1
    w = sgd.sgd_pass_dense(np.zeros(D), X[:1], np.array([-1.0]), np.array([0]), batch=1, loss="hinge",
                           lr_kind="inv_sqrt", lr0=0.5, l2=0.0, rnd=4, steps=(0, 1))
    assert np.allclose(w, 0.5 / math.sqrt(4 * 1 + 0 + 1) * -1.0 * X[0])


def test_ragged_last_batch_uses_its_own_size():
    # S = 3, B = 2: second batch holds one sample and averages over one.
    X = np.array([[1.0], [1.0], [4.0]])
    y = np.array([1.0, 1.0, 1.0])
    w = sgd.sgd_pass_dense(np.zeros(1), X, y, np.array([0, 1, 2]), batch=2, loss="hinge",
                           lr_kind="const", lr0=0.1, l2=0.0, rnd=0)
    # step 1: m = 0 -> c = -1 both; g = -1; w = 0.1.  step 2: m = 0.4 < 1 -> g = -4; w = 0.5
    assert np.allclose(w, [0.5])


def _dense_to_csr(X):
    row_ptr, col, val = [0], [], []
    for r in X:
        nz = np.nonzero(r)[0]
        col += nz.tolist()
        val += r[nz].tolist()
        row_ptr.append(len(col))
    return (np.array(row_ptr, np.int64), np.array(col, np.int32), np.array(val, np.float32))


@pytest.mark.parametrize("loss,l2", [("logistic", 0.0), ("hinge", 1e-2)])
def test_csr_pass_equals_dense_pass_on_same_data(loss, l2):
    S, D, B = 23, 9, 4
    X = RNG.standard_normal((S, D)).astype(np.float32)
    X[RNG.random((S, D)) < 0.6] = 0.0
    X[:, 3] = np.where(RNG.random(S) < 0.5, 1.0, 0.0)    # a hot column repeated in a batch
    y = np.where(RNG.random(S) < 0.5, -1.0, 1.0).astype(np.float32)
    rp, col, val = _dense_to_csr(X)
    sched = prng.schedule(S, 0, 2, 3)
    w0 = 0.05 * RNG.standard_normal(D)
    kw = dict(batch=B, loss=loss, lr_kind="inv_sqrt", lr0=0.5, l2=l2, rnd=3)
    a = sgd.sgd_pass_dense(w0, X, y, sched, **kw)
    b = sgd.sgd_pass_csr(w0, rp, col, val, y, sched, **kw)
    assert np.allclose(a, b, rtol=1e-12, atol=1e-14)


def test_objective_matches_definition_and_csr():
    S, D = 17, 5
    X = RNG.standard_normal((S, D)).astype(np.float32)
    y = np.where(RNG.random(S) < 0.5, -1.0, 1.0).astype(np.float32)
    w = RNG.standard_normal(D)
    rp, col, val = _dense_to_csr(X)
    for loss, l2 in (("logistic", 0.0), ("hinge", 0.2)):
        a = sgd.objective_dense(w, X, y, loss, l2)
        b = sgd.objective_csr(w, rp, col, val, y, loss, l2)
        brute = sum(sgd.loss_value(np.array([float(y[s]) * float(X[s].astype(np.float64) @ w)]), loss)[0]
                    for s in range(S)) / S + 0.5 * l2 * float(w @ w)
        assert a == pytest.approx(brute, rel=1e-12) and b == pytest.approx(brute, rel=1e-12)


def test_sgd_decreases_objective_on_separable_data():
    S, D = 256, 8
    wstar = RNG.standard_normal(D)
    X = RNG.standard_normal((S, D))
    y = np.where(X @ wstar >= 0, 1.0, -1.0)
    w = np.zeros(D)
    f0 = sgd.objective_dense(w, X, y, "logistic", 0.0)
    for r in range(5):
        w = sgd.sgd_pass_dense(w, X, y, prng.schedule(S, 0, 0, r), batch=16, loss="logistic",
                               lr_kind="const", lr0=0.5, l2=0.0, rnd=r)
    assert sgd.objective_dense(w, X, y, "logistic", 0.0) < 0.5 * f0
    assert np.mean(np.sign(X @ w) == y) > 0.95


@pytest.mark.parametrize("loss,l2,lr_kind", [("hinge", 1e-2, "inv_sqrt"), ("logistic", 0.3, "const"),
                                             ("logistic", 0.0, "inv_sqrt")])
def test_scale_form_equals_dense_decay(loss, l2, lr_kind):
    # w = s v with s <- s (1 - eta l2) is the update w <- (1 - eta l2) w - eta g
    # written differently: the plain dense decay of the dense pass fixes it
    S, D, B = 41, 11, 5
    X = RNG.standard_normal((S, D)).astype(np.float32)
    X[RNG.random((S, D)) < 0.5] = 0.0
    X[:, 2] = np.where(RNG.random(S) < 0.7, 0.8, 0.0)      # repeated column inside a batch
    y = np.where(RNG.random(S) < 0.5, -1.0, 1.0).astype(np.float32)
    rp, col, val = _dense_to_csr(X)
    sched = prng.schedule(S, 3, 1, 2)
    w0 = 0.05 * RNG.standard_normal(D)
    kw = dict(batch=B, loss=loss, lr_kind=lr_kind, lr0=0.4, l2=l2, rnd=2)
    want = sgd.sgd_pass_dense(w0, X, y, sched, **kw)
    got = sgd.sgd_pass_csr_scaled(w0, rp, col, val, y, sched, **kw)
    assert np.allclose(got, want, rtol=1e-12, atol=1e-14)
    amb_a, amb_b = [], []
    sgd.sgd_pass_csr(w0, rp, col, val, y, sched, ambiguous=amb_a, **kw)
    sgd.sgd_pass_csr_scaled(w0, rp, col, val, y, sched, ambiguous=amb_b, **kw)
    assert amb_a == amb_b
    # a step range of the scaled pass continues from the model it was given
    mid = sgd.sgd_pass_csr_scaled(w0, rp, col, val, y, sched, steps=(0, 4), **kw)
    end = sgd.sgd_pass_csr_scaled(mid, rp, col, val, y, sched, steps=(4, sgd.n_steps(S, B)), **kw)
    assert np.allclose(end, want, rtol=1e-12, atol=1e-14)


def test_scale_form_shrinks_untouched_columns():
    # a column no sample touches decays by prod_t (1 - eta_t l2): hand-computed
    X = np.array([[1.0, 0.0], [0.5, 0.0]], np.float32)
    y = np.array([1.0, -1.0], np.float32)
    rp, col, val = _dense_to_csr(X)
    w0 = np.array([0.0, 2.0])
    out = sgd.sgd_pass_csr_scaled(w0, rp, col, val, y, np.array([0, 1]), batch=1, loss="hinge",
                                  lr_kind="const", lr0=0.5, l2=0.1, rnd=0)
    assert out[1] == pytest.approx(2.0 * 0.95 * 0.95, rel=1e-15)
