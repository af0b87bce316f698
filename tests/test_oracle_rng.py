"""Pins for the oracle's random-number path (CPU only).

The paper never says how its sampling draws random numbers; the build fixes
Philox4x32-10 (Salmon et al., SC'11), a uniform in (0,1) from the top 23 bits of
one output word, and E = -ln u computed by a fixed fp32 operation sequence.
These tests pin each piece to something other than the oracle itself:

* Philox: the Random123 known-answer vectors, and an independent Philox stream
  (rocRAND's engine compiled for the host) over all four counter words and both
  key words;
* the uniform map: its definition on all boundary words, exactness in fp32;
* neglog: all 2^23 possible inputs against double-precision ``log``.
"""
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden")


def _kat_vectors():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            lhs, rhs = line.split(":")
            a = [int(x, 16) for x in lhs.split()]
            b = [int(x, 16) for x in rhs.split()]
            rows.append((a[:4], a[4:], b))
    return rows


@pytest.mark.parametrize("ctr,key,out", _kat_vectors())
def test_philox_known_answers(ctr, key, out):
    got = oracle.philox4x32_10(ctr, key)
    assert [int(x) for x in got] == out


@pytest.fixture(scope="module")
def rocrand_helper(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available to build the rocRAND host helper")
    exe = str(tmp_path_factory.mktemp("rr") / "rocrand_philox")
    src = os.path.join(HERE, "helpers", "rocrand_philox.cpp")
    subprocess.run([hipcc, "-x", "hip", "--offload-host-only", "-O1", "-w", "-o", exe, src],
                   check=True, capture_output=True)
    return exe


@pytest.mark.parametrize("seed,subseq,block", [
    (0, 0, 0),
    (0x123456789ABCDEF, 0, 0),
    (0x123456789ABCDEF, 5, 17),
    (7, 9, (1 << 32) + 3),              # carries into the second counter word
    (0xFFFFFFFFFFFFFFFF, (1 << 33) + 11, (1 << 32) - 2),
])
def test_philox_matches_rocrand_engine(rocrand_helper, seed, subseq, block):
    """rocRAND's stream is block i -> philox(ctr=(i_lo, i_hi, s_lo, s_hi), key=seed)."""
    n = 6
    res = subprocess.run([rocrand_helper, str(seed), str(subseq), str(4 * block), str(n)],
                         check=True, capture_output=True, text=True)
    lines = res.stdout.strip().splitlines()
    assert len(lines) == n
    key = [seed & 0xFFFFFFFF, seed >> 32]
    for i, line in enumerate(lines):
        c = block + i
        ctr = [c & 0xFFFFFFFF, (c >> 32) & 0xFFFFFFFF, subseq & 0xFFFFFFFF, subseq >> 32]
        want = [int(x, 16) for x in line.split()]
        assert [int(x) for x in oracle.philox4x32_10(ctr, key)] == want


def test_uniform_map_definition():
    for x in [0, 1, 511, 512, 0x12345678, 0xFFFFFE00, 0xFFFFFFFF]:
        u = oracle.uniform(x)
        assert u == ((2 * (x >> 9) + 1) / 2.0 ** 24)
        assert 0.0 < u < 1.0
        assert float(np.float32(u)) == u         # exact in fp32
    assert oracle.uniform(0) == 2.0 ** -24
    assert oracle.uniform(0xFFFFFFFF) == 1.0 - 2.0 ** -24


@pytest.fixture(scope="module")
def neglog_all():
    k = np.arange(1 << 23, dtype=np.uint64)
    u = ((2 * k + 1).astype(np.float64) * 2.0 ** -24).astype(np.float32)
    return u, oracle.neglog_array(u)


def test_neglog_exhaustive_accuracy(neglog_all):
    """Every possible input: |E - (-ln u)| <= 2 ulp of the fp32 result, E > 0."""
    u, E = neglog_all
    ref = -np.log(u.astype(np.float64))
    ulp = np.spacing(ref.astype(np.float32)).astype(np.float64)
    err = np.abs(E.astype(np.float64) - ref) / ulp
    assert np.all(E > 0)
    assert err.max() <= 2.0, err.max()


def test_neglog_monotone(neglog_all):
    """E is non-increasing in u, so the noise preserves the order of the uniforms."""
    _, E = neglog_all
    assert np.all(np.diff(E) <= 0)


def test_neglog_scalar_matches_array(neglog_all):
    u, E = neglog_all
    for i in [0, 1, 12345, (1 << 22), (1 << 23) - 1]:
        assert oracle.neglog(u[i]) == E[i]


def test_noise_counter_layout():
    """Slot i uses word i&3 of the block at counter (i>>2, inst, round, purpose)."""
    seed = 0xDEADBEEF12345678
    key = [seed & 0xFFFFFFFF, seed >> 32]
    for inst, rnd, slot in [(0, 0, 0), (3, 7, 5), (1000, 2, 4095), (7, 1, 8191)]:
        x = oracle.philox4x32_10([slot >> 2, inst, rnd, 0], key)[slot & 3]
        want = oracle.neglog(oracle.uniform(int(x)))
        assert oracle.noise(seed, inst, rnd, slot) == want


def test_exponential_distribution_moments():
    """E = -ln u over a large Philox sample has the Exp(1) mean and variance."""
    n = 1 << 16
    vals = np.array([oracle.noise(42, i >> 12, 3, i & 4095) for i in range(n)], dtype=np.float64)
    assert abs(vals.mean() - 1.0) < 4 / np.sqrt(n)
    assert abs(vals.var() - 1.0) < 10 / np.sqrt(n)
