"""Pins of the oracle's value-score variants (Appendix A: L2, Range, Var) and of
random reservation (Appendix D).  CPU only."""
import math

import numpy as np
import pytest
from scipy import stats

import oracle


@pytest.fixture(scope="module", autouse=True)
def _built():
    oracle.build(force=False)


def test_closed_forms():
    d = 16
    v = np.zeros((1, 5, d))
    v[0, 0] = 3.0                         # constant row
    v[0, 1, 4] = 1.0                      # unit vector
    v[0, 2] = np.arange(d)                # arithmetic sequence 0..d-1
    v[0, 3, :2] = (-2.0, 2.0)
    l2 = oracle.value_score(v, 5, oracle.VALUE_L2)[0]
    var = oracle.value_score(v, 5, oracle.VALUE_VAR)[0]
    rg = oracle.value_score(v, 5, oracle.VALUE_RANGE)[0]
    assert l2[0] == pytest.approx(3.0 * math.sqrt(d)) and var[0] == 0.0 and rg[0] == 0.0
    assert l2[1] == pytest.approx(1.0) and var[1] == pytest.approx((1 - 1 / d) / d) and rg[1] == 1.0
    # variance of 0..d-1 is (d^2 - 1) / 12
    assert var[2] == pytest.approx((d * d - 1) / 12.0)
    assert l2[2] == pytest.approx(math.sqrt((d - 1) * d * (2 * d - 1) / 6.0))
    assert l2[3] == pytest.approx(math.sqrt(8.0)) and rg[3] == 4.0
    assert l2[4] == 0.0 and var[4] == 0.0


def test_invariances():
    rng = np.random.default_rng(1)
    v = rng.standard_normal((3, 50, 64))
    var = oracle.value_score(v, 40, oracle.VALUE_VAR).astype(np.float64)
    l2 = oracle.value_score(v, 40, oracle.VALUE_L2).astype(np.float64)
    # Var is translation invariant and scales with the square; L2 is homogeneous
    np.testing.assert_allclose(oracle.value_score(v + 7.5, 40, oracle.VALUE_VAR), var, rtol=2e-6)
    np.testing.assert_allclose(oracle.value_score(v * 3, 40, oracle.VALUE_VAR), 9 * var, rtol=2e-6)
    np.testing.assert_allclose(oracle.value_score(-2 * v, 40, oracle.VALUE_L2), 2 * l2, rtol=2e-6)
    # L2^2 = d (Var + mu^2)
    mu = v[:, :40].mean(-1)
    np.testing.assert_allclose(l2 ** 2, 64 * (var + mu ** 2), rtol=1e-5)
    # permuting a row's elements changes none of the three
    perm = rng.permutation(64)
    for kind in (oracle.VALUE_L2, oracle.VALUE_VAR, oracle.VALUE_RANGE):
        np.testing.assert_allclose(oracle.value_score(v[..., perm], 40, kind),
                                   oracle.value_score(v, 40, kind), rtol=1e-6)


def test_random_reservation_scores():
    K = 4096
    u = oracle.value_score(None, K, oracle.VALUE_RANDOM, seed=5, rnd=3, n_inst=4, inst_base=10)
    assert u.shape == (4, K) and np.all((u > 0) & (u < 1))
    # they are the Philox words of purpose 2 through the uniform map
    for i in (0, 1, 2, 3, 1000, K - 1):
        x = oracle.philox4x32_10([i >> 2, 11, 3, 2], [5, 0])
        assert u[1, i] == oracle.uniform(int(x[i & 3]))
    assert stats.kstest(u.reshape(-1).astype(np.float64), "uniform").pvalue > 1e-4
    # the top N_v of i.i.d. uniforms is a uniformly random subset: every slot is
    # reserved with probability N_v / K over rounds
    Nv, hits = 64, np.zeros(256)
    for rnd in range(400):
        uu = oracle.value_score(None, 256, oracle.VALUE_RANDOM, seed=1, rnd=rnd, n_inst=1)[0]
        hits[np.argsort(-uu, kind="stable")[:Nv]] += 1
    assert stats.chisquare(hits).pvalue > 1e-4
    assert abs(hits.mean() / 400 - Nv / 256) < 1e-12
