"""The embedding layer's cost model (host logic, CPU): coefficients fitted
to the committed MI355X measurements, validated by leaving each measured
configuration out of the fit and predicting it."""
import numpy as np

from paper_2112_02752_amd import cost


def test_coefficients_are_non_negative():
    m = cost.model()
    for p in cost.PHASES:
        assert (m.coef[p] >= 0).all(), (p, m.coef[p])


def test_nnls_recovers_a_known_solution():
    rng = np.random.default_rng(0)
    A = rng.uniform(0, 1, size=(30, 4))
    x_true = np.array([0.5, 0.0, 2.0, 1.0])
    x = cost._nnls(A, A @ x_true)
    np.testing.assert_allclose(x, x_true, atol=1e-9)


def test_leave_one_out_predicts_every_measured_step():
    res = cost.leave_one_out()
    assert len(res) >= 10
    step_err = np.array([abs(r["rel_err"]["step"]) for r in res])
    assert step_err.max() <= 0.25, step_err
    assert np.median(step_err) <= 0.10, step_err
    for p in cost.PHASES:
        assert np.median([abs(r["rel_err"][p]) for r in res]) <= 0.15, p


def test_prediction_grows_with_the_batch():
    small = cost.predict(100_000, 20_000, 50_000_000, 64)
    large = cost.predict(1_000_000, 150_000, 50_000_000, 64)
    for k in ("fwd", "dedup", "bwd_update", "step"):
        assert large[k] > small[k]
    ew = cost.predict(500_000, 62_000, 50_000_000, 64, opt="adagrad_ew")
    rw = cost.predict(500_000, 62_000, 50_000_000, 64, opt="adagrad")
    assert ew["bwd_update"] >= rw["bwd_update"]
