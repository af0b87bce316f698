"""The library's device random numbers against the oracle, bit for bit.

The selection keys attn / E (Sec. 3.2, sampling proportional to the pooled
score) and the DKV projections depend on E = -ln u and on Philox4x32-10 being
the same bits on both sides.  The helper librngprobe.so evaluates the
library's own device functions (csrc/rng.hpp) on every input:

* neg_log on all 2^23 values of the uniform map, against the oracle's
  independent implementation of the same binary32 operation sequence;
* cos(2 pi u) on every 64th uniform and around the quadrant edges;
* Philox4x32-10 on 4096 consecutive counters per key, 64-bit keys included.
"""
import ctypes
import os

import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

HELPER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "helpers", "librngprobe.so")


@pytest.fixture(scope="module")
def probe(gpu_lib):
    if not os.path.exists(HELPER):
        pytest.fail("tests/helpers/librngprobe.so is missing: run __graft_entry__.build()")
    lib = ctypes.CDLL(HELPER)
    P, U32 = ctypes.c_void_p, ctypes.c_uint32
    lib.rngprobe_neglog.argtypes = [P, U32, U32, P]
    lib.rngprobe_cos2pi.argtypes = [P, U32, U32, P]
    lib.rngprobe_philox.argtypes = [P, U32, U32, U32, U32, U32, U32, U32, P]
    for f in (lib.rngprobe_neglog, lib.rngprobe_cos2pi, lib.rngprobe_philox):
        f.restype = ctypes.c_int
    return lib


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _uniforms(words: np.ndarray) -> np.ndarray:
    """The uniform map u = (2 (x >> 9) + 1) 2^-24 for x = word << 9, exact in fp32."""
    return ((2.0 * words.astype(np.float64) + 1.0) * 2.0 ** -24).astype(np.float32)


def test_neglog_every_input_bitwise(probe):
    n = 1 << 23
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    assert probe.rngprobe_neglog(ctypes.c_void_p(out.data_ptr()), 0, n, _stream()) == 0
    torch.cuda.synchronize()
    gpu = out.cpu().numpy()
    ref = oracle.neglog_array(_uniforms(np.arange(n, dtype=np.uint32)))
    diff = np.nonzero(gpu.view(np.uint32) != ref.view(np.uint32))[0]
    assert diff.size == 0, "neg_log differs on %d of %d inputs, first at word %d: %r vs %r" % (
        diff.size, n, diff[0], gpu[diff[0]], ref[diff[0]])
    assert np.all(gpu > 0)


def test_cos2pi_bitwise(probe):
    n = 1 << 23
    words = np.concatenate([np.arange(0, n, 64, dtype=np.uint32)] +
                           [np.arange(max(0, e - 8), min(n, e + 8), dtype=np.uint32)
                            for e in (0, n // 4, n // 2, 3 * n // 4, n - 1)])
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    assert probe.rngprobe_cos2pi(ctypes.c_void_p(out.data_ptr()), 0, n, _stream()) == 0
    torch.cuda.synchronize()
    gpu = out.cpu().numpy()[words]
    ref = np.array([oracle.cos2pi(u) for u in _uniforms(words)], dtype=np.float32)
    np.testing.assert_array_equal(gpu.view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("ctr,key", [
    ((0, 0, 0, 0), (0, 0)),
    ((17, 2303, 41, 0), (0xDEADBEEF, 0x12345678)),      # a 64-bit seed, purpose 0
    ((0xFFFFF000, 0xFFFFFFFF, 7, 1), (1, 0xFFFFFFFF)),   # counter wrap, purpose 1
])
def test_philox_bitwise(probe, ctr, key):
    n = 4096
    out = torch.empty(4 * n, dtype=torch.int32, device="cuda")
    assert probe.rngprobe_philox(ctypes.c_void_p(out.data_ptr()), *ctr, *key, n, _stream()) == 0
    torch.cuda.synchronize()
    gpu = out.cpu().numpy().view(np.uint32).reshape(n, 4)
    for i in range(0, n, 97):
        c = ((ctr[0] + i) & 0xFFFFFFFF, ctr[1], ctr[2], ctr[3])
        np.testing.assert_array_equal(gpu[i], oracle.philox4x32_10(c, key))
