"""Pins of the oracle's VaSE-DKV pieces (Sec. 3.2 with the CurDKV product score,
Eq. 4): the Gaussian projection G_t drawn afresh at every eviction step and the
score s_i = ||G^T k_i||^2 ||G^T v_i||^2.  CPU only."""
import math

import numpy as np
import pytest
from scipy import stats

import oracle


@pytest.fixture(scope="module", autouse=True)
def _built():
    oracle.build(force=False)


def test_cos2pi_against_libm():
    # 2^17 odd multiples of 2^-24 spread over (0, 1), plus the quadrant edges
    j = np.arange(0, 1 << 23, 64, dtype=np.int64)
    us = ((2 * j + 1) * 2.0 ** -24).astype(np.float32)
    got = np.array([oracle.cos2pi(float(u)) for u in us], dtype=np.float64)
    ref = np.cos(2 * np.pi * us.astype(np.float64))
    assert np.max(np.abs(got - ref)) < 3e-7
    for u, c in ((0.25, 0.0), (0.5, -1.0), (0.75, 0.0)):
        assert abs(float(oracle.cos2pi(u)) - c) < 1e-7


def test_gaussian_is_box_muller_of_its_philox_words():
    d, r, seed, inst, rnd = 16, 20, 0xDEADBEEF12345678, 77, 9
    g = oracle.dkv_gaussian(seed, inst, rnd, d, r)
    key = [seed & 0xFFFFFFFF, seed >> 32]
    for e in range(d * r):
        x = oracle.philox4x32_10([e >> 1, inst, rnd, 1], key)
        u1 = oracle.uniform(int(x[2 * (e & 1)]))
        u2 = oracle.uniform(int(x[2 * (e & 1) + 1]))
        z = math.sqrt(-2.0 * math.log(u1)) * math.cos(2 * math.pi * u2) / math.sqrt(r)
        assert abs(float(g.reshape(-1)[e]) - z) <= 2e-6 * max(1.0, abs(z)), e


def test_gaussian_distribution():
    d, r = 128, 20
    gs = np.concatenate([oracle.dkv_gaussian(3, i, 1, d, r).reshape(-1) for i in range(400)])
    gs = gs.astype(np.float64)
    assert abs(gs.mean()) < 4 * math.sqrt(1 / r / gs.size)
    assert abs(gs.var() * r - 1.0) < 0.01
    ks = stats.kstest(gs, "norm", args=(0.0, math.sqrt(1 / r)))
    assert ks.pvalue > 1e-4, ks
    # fourth moment of a Gaussian: 3 sigma^4
    assert abs(np.mean(gs ** 4) * r * r - 3.0) < 0.05


def test_gaussian_fresh_per_step_and_instance_reproducible():
    a = oracle.dkv_gaussian(1, 0, 5, 64)
    assert np.array_equal(a, oracle.dkv_gaussian(1, 0, 5, 64))
    for other in (oracle.dkv_gaussian(1, 0, 6, 64), oracle.dkv_gaussian(1, 1, 5, 64),
                  oracle.dkv_gaussian(2, 0, 5, 64)):
        assert not np.array_equal(a, other)
        # independent draws: correlation near zero
        assert abs(np.corrcoef(a.reshape(-1), other.reshape(-1))[0, 1]) < 0.1


def _kv(n, N, d, seed):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n, N, d)), rng.standard_normal((n, N, d)) * 3.0


def test_score_closed_forms():
    n, N, K, d = 2, 40, 32, 16
    k, v = _kv(n, N, d, 0)
    # one column, a unit vector e_c: s = k_c^2 v_c^2
    for c in (0, 7, 15):
        g = np.zeros((n, d, 1), dtype=np.float32)
        g[:, c, 0] = 1.0
        s = oracle.dkv_score_g(k, v, g, K)
        np.testing.assert_allclose(s, (k[:, :K, c] ** 2 * v[:, :K, c] ** 2).astype(np.float32),
                                   rtol=1e-6)
    # r = d and G = I: s = ||k||^2 ||v||^2
    g = np.broadcast_to(np.eye(d, dtype=np.float32), (n, d, d)).copy()
    s = oracle.dkv_score_g(k, v, g, K)
    ref = (np.sum(k[:, :K] ** 2, -1) * np.sum(v[:, :K] ** 2, -1)).astype(np.float32)
    np.testing.assert_allclose(s, ref, rtol=1e-6)


def test_score_invariances():
    n, N, K, d, r = 2, 24, 20, 16, 5
    k, v = _kv(n, N, d, 1)
    rng = np.random.default_rng(2)
    g = rng.standard_normal((n, d, r)).astype(np.float32)
    s = oracle.dkv_score_g(k, v, g, K).astype(np.float64)
    # an orthogonal change of basis applied to keys, values and G leaves s unchanged
    q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    gq = np.einsum("ab,nbr->nar", q, g.astype(np.float64))
    # G must stay exactly representable: compare against the fp64 definition instead
    s_rot = np.sum(np.einsum("nia,nar->nir", k[:, :K] @ q.T, gq) ** 2, -1) * \
        np.sum(np.einsum("nia,nar->nir", v[:, :K] @ q.T, gq) ** 2, -1)
    np.testing.assert_allclose(s, s_rot, rtol=2e-6)
    # scaling keys by a and values by b scales s by a^2 b^2
    s2 = oracle.dkv_score_g(k * 2.0, v * 0.5, g, K).astype(np.float64)
    np.testing.assert_allclose(s2, s, rtol=1e-6)
    # only slots below K are scored
    assert s.shape == (n, K)


def test_round_keeps_the_top_scores_and_the_buffer():
    n, N, K, d, B = 3, 160, 128, 32, 32
    k, v = _kv(n, N, d, 3)
    s, src = oracle.dkv_round(k, v, K, B, seed=11, rnd=2)
    np.testing.assert_array_equal(s, oracle.dkv_score(k, v, K, 11, 2))
    for i in range(n):
        keep = np.sort(np.argsort(-s[i], kind="stable")[:K - B])
        np.testing.assert_array_equal(src[i], np.concatenate([keep, np.arange(K, N)]))
    # a fresh projection each step changes the scores
    assert not np.array_equal(s, oracle.dkv_score(k, v, K, 11, 3))
