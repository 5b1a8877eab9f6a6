"""CPU checks of the GPU tests' error metrics (tests/parity_metrics.py)."""
import numpy as np
import pytest

from parity_metrics import STEP, TRAJ, check_layer, factor_error, informative, rel, theta_error


def test_informative_part_removes_the_identity_multiple():
    rng = np.random.default_rng(0)
    B = rng.standard_normal((7, 7))
    A = 3.5 * np.eye(7) + 1e-3 * (B + B.T)
    Ai = informative(A)
    assert abs(np.trace(Ai)) < 1e-12
    assert np.allclose(informative(Ai), Ai)
    assert np.allclose(informative(A - 2.0 * np.eye(7)), Ai)


def test_factor_error_sees_what_the_whole_tensor_metric_dilutes():
    rng = np.random.default_rng(1)
    d = 64
    B = rng.standard_normal((d, d))
    A = 31.6 * np.eye(d) + 1e-2 * (B + B.T)
    E = 1e-5 * rng.standard_normal((d, d))
    whole = rel(A + E, A)
    fe, floor, frac = factor_error(A + E, A)
    assert frac == pytest.approx(np.linalg.norm(informative(A)) / np.linalg.norm(A))
    assert fe == pytest.approx(whole / frac, rel=1e-9)
    assert fe > 50 * whole
    assert floor == pytest.approx(2.0 ** -22 / frac)


def test_factor_error_skips_a_multiple_of_the_identity():
    assert factor_error(np.eye(5) * 2.0, np.eye(5) * 2.0) is None
    assert factor_error(np.array([[3.0]]), np.array([[3.0]])) is None


def test_theta_error_is_relative_to_the_applied_step():
    rng = np.random.default_rng(2)
    th0 = rng.standard_normal((8, 9))
    step = 1e-3 * rng.standard_normal((8, 9))
    lr, wd = 0.1, 5e-5
    th1 = th0 * (1 - lr * wd) - step
    err = 1e-9 * rng.standard_normal((8, 9))
    te, floor = theta_error(th1 + err, th1, th0, lr, wd)
    assert te == pytest.approx(np.linalg.norm(err) / np.linalg.norm(step), rel=1e-6)
    assert floor == pytest.approx(2.0 ** -23 * np.linalg.norm(th1) / np.linalg.norm(step))
    assert theta_error(th0, th0 * (1 - lr * wd), th0, lr, wd) is None


def test_check_layer_gates():
    rng = np.random.default_rng(3)
    d = 16
    B = rng.standard_normal((d, d))
    A = 10.0 * np.eye(d) + 1e-2 * (B + B.T)
    m = rng.standard_normal((d, d))
    th0 = rng.standard_normal((d, d))
    th1 = th0 - 1e-2 * m
    st = {"L": A, "R": A, "mom": m, "mom_sgd": m}
    check_layer(st, st, th1, th1, th0, 0.1, 0.0, STEP, "same")
    # A mistake confined to the informative part, small on the whole tensor: caught by the factor gate.
    bad = dict(st, L=A + 2e-2 * np.linalg.norm(informative(A)) / d * np.ones((d, d)))
    assert rel(bad["L"], A) < STEP["whole"] * 100
    with pytest.raises(AssertionError, match="informative"):
        check_layer(bad, st, th1, th1, th0, 0.1, 0.0, TRAJ, "bad factor")
    # A wrong step of 2% of the update: caught by the parameter gate at one step, not by the whole tensor.
    th_bad = th1 - 2e-2 * (th1 - th0)
    assert rel(th_bad, th1) < STEP["whole"] * 100
    with pytest.raises(AssertionError, match="applied step"):
        check_layer(st, st, th_bad, th1, th0, 0.1, 0.0, STEP, "bad step")
