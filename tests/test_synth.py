"""The seeded workload generator: distributions and reproducibility."""
import math

import numpy as np
import pytest

import synth


def _zipf_pmf(n, s):
    k = np.arange(1, n + 1, dtype=np.float64)
    p = k ** -s
    return p / p.sum()


@pytest.mark.parametrize("s", [0.9, 1.0, 1.2])
def test_bounded_zipf_matches_pmf(s):
    """Chi-square of rank frequencies (identity scramble undone) vs k^-s / H_{n,s}."""
    n, N = 50, 200_000
    ts = synth.TableSpec(rows=n, len_kind=0, lmax=1, lam=0, id_dist=1, zipf_s=s)
    w = synth.Workload("z", 1234, (ts,), 4, "fp32", N, "sum", "sgd")
    b = synth.make_batch(w, 0, with_grad=False)
    assert len(b.indices) == N
    # invert the affine scramble: row -> rank
    row_of_rank = np.array([synth.rank_to_row(w, 0, r) for r in range(1, n + 1)])
    assert sorted(row_of_rank) == list(range(n))  # bijection
    rank_of_row = np.empty(n, np.int64)
    rank_of_row[row_of_rank] = np.arange(1, n + 1)
    counts = np.bincount(rank_of_row[b.indices] - 1, minlength=n)
    expected = _zipf_pmf(n, s) * N
    chi2 = ((counts - expected) ** 2 / expected).sum()
    # 49 degrees of freedom: the 0.999 quantile is ~85.4
    assert chi2 < 85.4, chi2


@pytest.mark.parametrize("name,head", [("c1", 0.107), ("c3", 0.184), ("c5", 0.0172)])
def test_head_frequency_matches_harmonic(name, head):
    w = synth.workload(name)
    b = synth.make_batch(w, 0, with_grad=False)
    hot = synth.rank_to_row(w, 0, 1)
    p1 = 1.0 / (_zipf_pmf_norm(w.tables[0].rows, w.tables[0].zipf_s))
    assert abs(p1 - head) < 0.002
    f = np.mean(b.indices == hot)
    assert abs(f - p1) < 5 * math.sqrt(p1 * (1 - p1) / len(b.indices)) + 1e-4


def _zipf_pmf_norm(n, s):
    # H_{n,s} by direct summation for small n, Euler-Maclaurin tail otherwise
    m = min(n, 1_000_000)
    k = np.arange(1, m + 1, dtype=np.float64)
    H = (k ** -s).sum()
    if n > m:
        a, b = m + 0.5, n + 0.5
        H += (b ** (1 - s) - a ** (1 - s)) / (1 - s) if s != 1 else math.log(b / a)
    return H


def test_batch_is_deterministic_and_step_dependent():
    w = synth.workload("c2")
    b0 = synth.make_batch(w, 3)
    b1 = synth.make_batch(w, 3)
    b2 = synth.make_batch(w, 4)
    np.testing.assert_array_equal(b0.offsets, b1.offsets)
    np.testing.assert_array_equal(b0.indices, b1.indices)
    np.testing.assert_array_equal(b0.grad, b1.grad)
    assert not np.array_equal(b0.indices[:1000], b2.indices[:1000])


def test_bag_lengths_and_ids_in_range():
    for name in ("c1", "c2", "c3", "c4"):
        w = synth.workload(name)
        b = synth.make_batch(w, 0, with_grad=False)
        lens = np.diff(b.offsets)
        B = w.bags_per_table
        for t, ts in enumerate(w.tables):
            lt = lens[t * B:(t + 1) * B]
            assert lt.min() >= 1 and lt.max() <= ts.lmax
            ids = b.indices[b.offsets[t * B]:b.offsets[(t + 1) * B]]
            assert ids.min() >= 0 and ids.max() < ts.rows
            if ts.len_kind == 2:
                assert np.all(lt == 1)


def test_poisson_lengths_moments():
    w = synth.workload("c3")
    lens = synth.bag_lengths(w, 0)
    assert abs(lens.mean() - 30.0) < 0.3
    assert abs(lens.var() - 30.0) < 2.0


def test_uniform_lengths_cover_range():
    w = synth.workload("c5")
    lens = synth.bag_lengths(w, 0)
    assert lens.min() == 1 and lens.max() == 100
    assert abs(lens.mean() - 50.5) < 0.5


def test_normal_grad_moments():
    g = synth.make_grad(synth.workload("c3"), 0)
    assert abs(g.mean()) < 0.005 and abs(g.std() - 1.0) < 0.005
    assert abs(((g - g.mean()) ** 4).mean() / g.var() ** 2 - 3.0) < 0.05


def test_weight_rows_match_dense_and_range():
    w = synth.scaled(synth.workload("c1"), rows_div=100)
    dense = synth.dense_weights(w)
    rows = np.array([0, 5, 999, 17], np.uint32)
    np.testing.assert_array_equal(synth.weight_rows(w, rows), dense[rows])
    assert dense.min() >= -0.01 and dense.max() < 0.01
    assert abs(dense.mean()) < 1e-3


def test_bf16_weights_are_rne_of_fp32():
    w32 = synth.scaled(synth.workload("c1"), rows_div=1000)
    from dataclasses import replace
    w16 = replace(w32, dtype="bf16")
    f = synth.dense_weights(w32)
    b = synth.dense_weights(w16)
    # RNE by integer arithmetic on the fp32 bits
    u = f.view(np.uint32).astype(np.uint64)
    rne = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    np.testing.assert_array_equal(b, rne)


def test_c4_table_sizes_loguniform_in_range():
    w = synth.workload("c4")
    rows = np.array(w.rows)
    assert rows.min() >= 1000 and rows.max() <= 40_000_000
    assert w.total_rows < 2 ** 32
