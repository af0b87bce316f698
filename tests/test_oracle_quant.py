"""Pins of the oracle's Range-based per-token quantisation (Eq. 6, Sec. 4.3) and of its
full-precision reserve for the largest-Range rows (Sec. 7).  CPU only."""
import numpy as np
import pytest

import oracle


@pytest.fixture(scope="module", autouse=True)
def _built():
    oracle.build(force=False)


def _unpack(codes, bits, d):
    """Codes of each row as integers: code e at bits [e*bits, e*bits + bits), little-endian."""
    c = np.asarray(codes, dtype=np.uint8)
    bitsarr = np.unpackbits(c, axis=-1, bitorder="little")
    bitsarr = bitsarr.reshape(c.shape[:-1] + (d, bits))
    return (bitsarr * (1 << np.arange(bits))).sum(-1)


def test_hand_example_two_bits():
    # one row of 8 values, one group: z = 0, Delta = (3 - 0) / 3 = 1, codes
    # round(x): 0.5 -> 0 (ties to even), 1.4 -> 1, 2.6 -> 3
    x = np.array([[[0.0, 1.0, 2.0, 3.0, 0.5, 1.4, 2.6, 3.0]]], dtype=np.float32)
    r = oracle.quantize(x, 1, bits=2, group=8)
    np.testing.assert_array_equal(r["params"][0, 0, 0], [1.0, 0.0])
    # packed: 0 | 1<<2 | 2<<4 | 3<<6 = 0xE4, then 0 | 1<<2 | 3<<4 | 3<<6 = 0xF4
    np.testing.assert_array_equal(r["codes"][0, 0], [0xE4, 0xF4])
    out = oracle.dequantize(r["codes"], r["params"], 1, 2, 8, out_bf16=False)
    np.testing.assert_array_equal(out[0, 0], np.float32([0, 1, 2, 3, 0, 1, 3, 3]))
    # ties go to the even code: 1.5 -> 2, 2.5 -> 2, 0.5 -> 0; packed 0 | 3<<2 | 2<<4 |
    # 2<<6 = 0xAC and 0 | 3<<2 | 0<<4 | 1<<6 = 0x4C
    x2 = np.array([[[0.0, 3.0, 1.5, 2.5, 0.5, 3.0, 0.0, 1.0]]], dtype=np.float32)
    r2 = oracle.quantize(x2, 1, bits=2, group=8)
    np.testing.assert_array_equal(r2["codes"][0, 0], [0xAC, 0x4C])
    # mse = (0.5^2 + 0.4^2 + 0.4^2) / 8 in float32 inputs
    xs = x.astype(np.float64)[0, 0]
    ref = ((xs - out[0, 0].astype(np.float64)) ** 2).mean()
    assert r["mse"][0, 0] == pytest.approx(ref, rel=1e-7)


def _rows(n, N, d, seed, outliers=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, N, d))
    if outliers:
        x *= np.exp(rng.uniform(0.0, np.log(100.0), size=(n, N, 1)))
    return x.astype(np.float32)


@pytest.mark.parametrize("bits", [2, 4, 8])
@pytest.mark.parametrize("group", [32, 64, 128])
def test_error_bound_and_extremes(bits, group):
    d, K, N = 128, 40, 45
    x = _rows(3, N, d, seed=bits * 100 + group)
    r = oracle.quantize(x, K, bits, group)
    q = _unpack(r["codes"], bits, d)
    assert q.max() <= 2 ** bits - 1
    out = oracle.dequantize(r["codes"], r["params"], N, bits, group, out_bf16=False)
    xg = x[:, :K].reshape(3, K, d // group, group).astype(np.float64)
    og = out[:, :K].reshape(3, K, d // group, group).astype(np.float64)
    qg = q.reshape(3, K, d // group, group)
    delta = r["params"][..., 0].astype(np.float64)
    zero = r["params"][..., 1].astype(np.float64)
    # the quantisation error of Eq. 6 is at most half a step (plus fp32 rounding)
    err = np.abs(xg - og)
    bound = 0.5 * delta[..., None] * (1 + 2.0 ** -20) + 4 * 2.0 ** -24 * np.abs(xg)
    assert np.all(err <= bound)
    # the zero point is the group minimum and is reproduced exactly; the maximum
    # takes the top code
    np.testing.assert_array_equal(zero, xg.min(-1))
    amin = xg.argmin(-1)[..., None]
    amax = xg.argmax(-1)[..., None]
    assert np.all(np.take_along_axis(qg, amin, -1) == 0)
    assert np.all(np.take_along_axis(qg, amax, -1) == 2 ** bits - 1)
    np.testing.assert_array_equal(np.take_along_axis(og, amin, -1), np.take_along_axis(xg, amin, -1))
    # Delta is the group's Range over 2^b - 1
    np.testing.assert_allclose(delta, (xg.max(-1) - xg.min(-1)) / (2 ** bits - 1), rtol=2e-7)


def test_constant_and_grid_groups_are_exact():
    d = 64
    x = np.zeros((1, 3, d), dtype=np.float32)
    x[0, 0] = 2.5                                  # constant: Delta = 0, every code 0
    k = np.arange(d) % 16
    x[0, 1] = -1.0 + k * 0.125                     # on the 4-bit grid of [-1, 0.875]
    x[0, 2, :32] = 7.0
    x[0, 2, 32:] = np.linspace(-3, 3, 32, dtype=np.float32)
    r = oracle.quantize(x, 3, bits=4, group=d)
    assert r["params"][0, 0, 0, 0] == 0.0 and np.all(r["codes"][0, 0] == 0)
    np.testing.assert_array_equal(_unpack(r["codes"], 4, d)[0, 1], k)
    out = oracle.dequantize(r["codes"], r["params"], 3, 4, d, out_bf16=False)
    np.testing.assert_array_equal(out[0, :2], x[0, :2])
    assert r["mse"][0, 0] == 0.0 and r["mse"][0, 1] == 0.0
    # with group 32 the constant half of row 2 is exact as well
    r32 = oracle.quantize(x, 3, bits=4, group=32)
    o32 = oracle.dequantize(r32["codes"], r32["params"], 3, 4, 32, out_bf16=False)
    np.testing.assert_array_equal(o32[0, 2, :32], x[0, 2, :32])


def test_mse_matches_uniform_quantisation_noise():
    """For smooth data the error is uniform on [-Delta/2, Delta/2]: MSE ~ Delta^2 / 12."""
    d, K = 128, 2000
    rng = np.random.default_rng(5)
    x = rng.uniform(-1, 1, size=(1, K, d)).astype(np.float32)
    r = oracle.quantize(x, K, bits=4, group=d)
    delta = r["params"][0, :, 0, 0].astype(np.float64)
    ratio = r["mse"][0].astype(np.float64) / (delta ** 2 / 12)
    assert abs(ratio.mean() - 1.0) < 0.03
    # and the mse is the mean square of the reconstruction error
    out = oracle.dequantize(r["codes"], r["params"], K, 4, d, out_bf16=False)
    ref = ((x[0].astype(np.float64) - out[0].astype(np.float64)) ** 2).mean(-1)
    np.testing.assert_allclose(r["mse"][0], ref, rtol=1e-6)


def test_range_matches_eq5_and_correlates_with_error():
    """Range per token is Eq. 5 (the same value as the selection's Range) and, as the
    paper reports for the value cache, the reconstruction error grows with it."""
    x = _rows(2, 300, 128, seed=9)
    r = oracle.quantize(x, 300, bits=2, group=32)
    np.testing.assert_array_equal(r["range"], oracle.vrange(x, 300))
    lr = np.log(r["range"].astype(np.float64).ravel())
    lm = np.log(r["mse"].astype(np.float64).ravel())
    assert np.corrcoef(lr, lm)[0, 1] > 0.95


@pytest.mark.parametrize("Nv", [1, 7, 64])
def test_reserved_rows_are_the_largest_ranges(Nv):
    x = _rows(3, 70, 64, seed=Nv)
    x[1, 10] = x[1, 11] = x[1, 12] = 0.0
    x[1, 10, 0] = x[1, 11, 0] = x[1, 12, 0] = 1e4   # three equal Ranges: lower slots first
    r = oracle.quantize(x, 64, bits=4, group=32, Nv=Nv)
    for i in range(3):
        order = np.argsort(-r["range"][i], kind="stable")[:Nv]
        np.testing.assert_array_equal(r["hp_idx"][i], np.sort(order))
    # dequantisation puts the full-precision rows back in their slots
    hp_rows = np.stack([x[i, r["hp_idx"][i]] for i in range(3)])
    out = oracle.dequantize(r["codes"], r["params"], 70, 4, 32, out_bf16=False,
                            hp_rows=hp_rows, hp_idx=r["hp_idx"])
    for i in range(3):
        np.testing.assert_array_equal(out[i, r["hp_idx"][i]], x[i, r["hp_idx"][i]])
        rest = np.setdiff1d(np.arange(64), r["hp_idx"][i])
        if rest.size:
            assert not np.array_equal(out[i, rest], x[i, rest])
    if Nv < 3:
        np.testing.assert_array_equal(r["hp_idx"][1], np.arange(10, 10 + Nv))


def test_bf16_output_is_rounded_reconstruction():
    x = _rows(1, 10, 64, seed=3)
    r = oracle.quantize(x, 8, bits=8, group=64)
    o32 = oracle.dequantize(r["codes"], r["params"], 10, 8, 64, out_bf16=False)
    o16 = oracle.dequantize(r["codes"], r["params"], 10, 8, 64, out_bf16=True)
    import torch
    ref = torch.from_numpy(o32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(o16, ref)


def test_rejects_bad_args():
    x = np.zeros((1, 4, 64), dtype=np.float32)
    for kw in (dict(bits=3, group=32), dict(bits=4, group=48), dict(bits=4, group=32, Nv=5)):
        with pytest.raises(RuntimeError):
            oracle.quantize(x, 4, **kw)
