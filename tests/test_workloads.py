"""The seeded input generators: shapes, storage types, reproducibility and the
straggler models of the paper's simulation section at each workload's sizes."""
import numpy as np
import pytest
from scipy.special import gammaincinv

from workloads import ALL, BANDWIDTH, HEADLINE, LARGE, SMALL, TINY, gen


def test_names_unique_and_cyclic_sizes():
    assert len({w.name for w in ALL}) == len(ALL)
    for w in ALL:
        assert w.N == w.m and 0 <= w.s < w.m and w.delta == w.s + 1


@pytest.mark.parametrize("wl", ALL, ids=lambda w: w.name)
def test_patterns_in_range_and_reproducible(wl):
    count = min(wl.P, 1500)
    a = gen.psi(wl, count=count)
    assert a.shape == (count, wl.m) and a.dtype == np.int32
    assert a.min() >= 0 and a.max() <= wl.delta
    assert np.array_equal(a, gen.psi(wl, count=count))
    if count > 10:
        assert np.array_equal(a[7:11], gen.psi(wl, start=7, count=4))


def test_uniform_models():
    a = gen.psi(TINY)
    assert set(np.unique(a)) == set(range(TINY.delta + 1))
    h = gen.psi(HEADLINE, count=2000)
    zeros = (h == 0).sum(axis=1)
    assert zeros.min() >= HEADLINE.forced_zero
    # non-forced workers are uniform on {0..delta}: mean ~ delta/2 overall
    mean_rest = (h.sum(axis=1) / (HEADLINE.m - HEADLINE.forced_zero)).mean()
    assert abs(mean_rest - HEADLINE.delta / 2) < 0.05


def test_deadline_models():
    s = gen.psi(SMALL)
    # deadline = median full-completion time: about half the workers are done
    done = (s == SMALL.delta).mean()
    assert 0.4 < done < 0.6
    b = gen.psi(BANDWIDTH, count=1000)
    assert abs((b == BANDWIDTH.delta).mean() - 0.5) < 0.05   # fixed deadline = median completion
    assert BANDWIDTH.delta + gammaincinv(BANDWIDTH.delta, 0.5) == pytest.approx(19.6687, abs=1e-4)
    ls = gen.psi(LARGE, count=200, variant="ls")
    assert (ls == 0).sum(axis=1).min() >= LARGE.ls_forced_zero


def test_regression_data_and_labels():
    X, y, w = gen.regression_data(TINY)
    assert X.shape == (6, 32, 64) and X.dtype == np.float32 and (w == 0).all()
    X3, y3, w3 = gen.regression_data(HEADLINE, chunks=[0, 7])
    assert X3.shape == (2, 512, 16384) and set(np.unique(y3)) <= {0.0, 1.0}
    assert abs(X3.std() * np.sqrt(16384) - 1.0) < 0.01
    assert abs(w3.std() - 0.1) < 0.005
    # chunk subsets are consistent with the full draw
    Xs, ys, _ = gen.regression_data(SMALL, chunks=[3])
    Xa, ya, _ = gen.regression_data(SMALL)
    assert np.array_equal(Xs[0], Xa[3]) and np.array_equal(ys[0], ya[3])


def test_given_gradients_and_bf16_rounding():
    g = gen.given_chunk(LARGE.__class__(**{**LARGE.__dict__, "d": 4096}), 3)
    assert g.dtype == np.uint16
    f = np.array([1.0, 1.00390625, 1.01171875, -3.0, 1e-40], dtype=np.float32)
    bits = gen.f32_to_bf16_bits(f)
    back = (bits.astype(np.uint32) << 16).view(np.float32)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: ties go to the even mantissa (1.0)
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == 1.015625 and back[3] == -3.0
    R1 = gen.shared_R(50, 1)
    R2 = gen.shared_R(50, 2)
    assert np.array_equal(R1[0], R2[0]) and R2.dtype == np.float32


def test_random_orderings_are_orderings_of_the_support():
    A = gen.random_regular_graph(40, 5)
    Os = gen.random_orderings(A, 7, seed=3)
    assert Os.shape == (7, 40, 40)
    for O in Os:
        assert ((O != 0) == (A != 0)).all()
        for j in range(40):
            assert sorted(O[:, j][O[:, j] != 0]) == [1, 2, 3, 4, 5]
    assert not (Os[0] == Os[1]).all()
    assert (gen.random_orderings(A, 7, seed=3) == Os).all()
