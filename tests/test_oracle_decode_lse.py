"""Pins of the oracle's decode-side integration: the persistent-slot log-sum-exp a
decode step hands the round, and the window score that completes each row's
normaliser with the buffer slots only.  CPU only."""
import math

import numpy as np
import pytest
import torch

import oracle


@pytest.fixture(scope="module", autouse=True)
def _built():
    oracle.build(force=False)


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def test_decode_lse_closed_forms():
    d = 4
    k = np.zeros((1, 6, d))
    q = np.zeros((1, 2, d))
    # q = 0: every score is 0, so the log-sum-exp over n slots is ln n
    for n in (1, 3, 6):
        assert oracle.decode_lse(q, k, n)[0, 0] == pytest.approx(math.log(n), abs=1e-15)
    # one key aligned with q: ln(e^{|q|^2/sqrt d} + (n-1))
    q[0, 1] = (2.0, 0, 0, 0)
    k[0, 2] = (3.0, 0, 0, 0)
    lse = oracle.decode_lse(q, k, 5)[0, 1]
    assert lse == pytest.approx(math.log(math.exp(6.0 / 2.0) + 4.0), rel=1e-14)
    # slots at and beyond n_persist do not count
    k[0, 5] = (100.0, 0, 0, 0)
    assert oracle.decode_lse(q, k, 5)[0, 1] == lse


def test_decode_lse_matches_torch_logsumexp():
    n, N, G, d = 3, 70, 5, 64
    q = _rand((n, G, d), 1)
    k = _rand((n, N, d), 2, 2.0)
    for npers in (1, 33, 70):
        ref = torch.logsumexp(torch.einsum("ngd,nkd->ngk", torch.from_numpy(q),
                                           torch.from_numpy(k[:, :npers])) / math.sqrt(d), -1)
        np.testing.assert_allclose(oracle.decode_lse(q, k, npers), ref.numpy(), rtol=1e-13)


def test_decode_lse_is_the_normaliser_of_decode():
    """softmax weights built from the lse reproduce the oracle's decode output"""
    n, N, G, d = 2, 40, 3, 16
    q, k, v = _rand((n, G, d), 3), _rand((n, N, d), 4), _rand((n, N, d), 5)
    lse = oracle.decode_lse(q, k, N)
    s = np.einsum("ngd,nkd->ngk", q, k) / math.sqrt(d)
    out = np.einsum("ngk,nkd->ngd", np.exp(s - lse[..., None]), v)
    np.testing.assert_allclose(out, oracle.decode(q, k, v, N), rtol=1e-12, atol=1e-14)


def test_score_lse_equals_score_with_true_normaliser():
    n, G, w, K, B, d, pool = 3, 2, 5, 50, 9, 32, 7
    q = _rand((n, G, w, d), 6)
    k = _rand((n, K + B, d), 7, 1.5)
    # the persistent part of each window row's normaliser, via the decode-side function
    lse = oracle.decode_lse(q.reshape(n, G * w, d), k, K).reshape(n, G, w)
    got = oracle.score_lse(q, k, K, pool, lse)
    ref = oracle.score(q, k, K, pool)
    np.testing.assert_allclose(got, ref, rtol=2e-7)


def test_score_lse_supplied_normaliser_closed_forms():
    """One row, P = 1: p_i = exp(s_i) / (exp(L) + sum over the buffer of exp(s)).
    L = -inf leaves the buffer sum alone, and raising L by one scales every
    candidate's score by 1/e once exp(L) dominates."""
    n, G, w, K, B, d = 1, 1, 3, 10, 4, 8
    q = _rand((n, G, w, d), 8)
    k = _rand((n, K + B, d), 9)
    s = np.einsum("d,kd->k", q[0, 0, 0], k[0]) / math.sqrt(d)
    for L in (-np.inf, -3.0, 1.25, 4.0):
        p = np.exp(s[:K]) / (math.exp(L) + np.exp(s[K:]).sum())
        one = oracle.score_lse(q[:, :, :1], k, K, 1, np.full((n, G, 1), L))
        np.testing.assert_allclose(one[0], p, rtol=1e-6)
    a = oracle.score_lse(q, k, K, 1, np.full((n, G, w), 50.0)).astype(np.float64)
    b = oracle.score_lse(q, k, K, 1, np.full((n, G, w), 51.0)).astype(np.float64)
    np.testing.assert_allclose(b, a * math.exp(-1.0), rtol=1e-6)


def test_score_lse_rejects_bad_args():
    q = np.zeros((1, 1, 1, 8))
    k = np.zeros((1, 10, 8))
    with pytest.raises(RuntimeError):
        oracle.score_lse(q, k, 10, 2, np.zeros((1, 1, 1)))     # even pool
    with pytest.raises(RuntimeError):
        oracle.decode_lse(np.zeros((1, 1, 8)), k, 11)          # n_persist > N
