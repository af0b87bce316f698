"""Comparison helpers shared by the GPU parity tests (no method arithmetic here)."""
import numpy as np

# Score tolerance: fp32 scores within 1e-4 relative of the double-precision
# oracle; the absolute floor only covers values that underflow in fp32.
ATTN_RTOL = 1e-4
ATTN_ATOL = 1e-30
# Decode: 2e-2 absolute at bf16, plus the rounding of the stored bf16 output
# itself (half an ulp: 2^-8 relative); fp32 outputs: 1e-4 absolute + relative.
DEC_ATOL_BF16 = 2e-2
DEC_RTOL_BF16 = 2.0 ** -8
DEC_TOL_F32 = 1e-4


def assert_attn_close(got: np.ndarray, ref: np.ndarray, what: str = "attn") -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    bound = ATTN_RTOL * np.abs(ref) + ATTN_ATOL
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError("%s: %d of %d outside 1e-4 relative; worst at %s: got %r ref %r"
                             % (what, int(bad.sum()), bad.size, i, got[i], ref[i]))
    rel = err / np.maximum(np.abs(ref), 1e-300)
    return float(rel[np.abs(ref) > 1e-30].max(initial=0.0))


def assert_decode_close(got: np.ndarray, ref: np.ndarray, bf16: bool) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    if bf16:
        bound = DEC_ATOL_BF16 + DEC_RTOL_BF16 * np.abs(ref)
    else:
        bound = DEC_TOL_F32 * (1.0 + np.abs(ref))
    if (err > bound).any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError("decode: worst at %s: got %r ref %r (err %g)" % (i, got[i], ref[i], err[i]))
    return float(err.max())


def survivor_check(src: np.ndarray, K: int, B: int, vrange: np.ndarray, Nv: int) -> None:
    """Budget invariants of one round: |S| = K, buffer kept in order, R_V kept."""
    n = src.shape[0]
    assert src.shape == (n, K)
    assert np.all(np.diff(src, axis=1) > 0), "survivor map not strictly increasing"
    assert np.all(src[:, K - B:] == np.arange(K, K + B)[None, :]), "buffer not kept at the end"
    assert np.all(src[:, :K - B] < K)
    if Nv > 0:
        order = np.argsort(-vrange, axis=1, kind="stable")[:, :Nv]
        for i in range(n):
            assert np.isin(order[i], src[i]).all(), "reserved slot evicted in instance %d" % i


def explained_swaps(src_gpu: np.ndarray, src_ref: np.ndarray, keys_ref: np.ndarray, K: int,
                    rtol: float):
    """Differences between two survivor maps, as boundary swaps.

    Returns a list of (instance, evicted_by_gpu, evicted_by_oracle, relative key gap)
    and raises if a difference is not a swap of candidates whose oracle keys lie
    within `rtol` (relative) of each other.
    """
    swaps = []
    for i in np.nonzero((src_gpu != src_ref).any(axis=1))[0]:
        kept_g = set(src_gpu[i][src_gpu[i] < K].tolist())
        kept_r = set(src_ref[i][src_ref[i] < K].tolist())
        only_r = sorted(kept_r - kept_g, key=lambda s: keys_ref[i, s])   # GPU evicted these
        only_g = sorted(kept_g - kept_r, key=lambda s: keys_ref[i, s])   # oracle evicted these
        assert len(only_r) == len(only_g), "instance %d: survivor counts differ" % i
        for a, b in zip(only_r, only_g):
            ka, kb = float(keys_ref[i, a]), float(keys_ref[i, b])
            gap = abs(ka - kb) / max(abs(ka), abs(kb), 1e-300)
            assert gap <= rtol, ("instance %d: slots %d/%d swapped with key gap %g > %g"
                                 % (i, a, b, gap, rtol))
            swaps.append((int(i), int(a), int(b), gap))
    return swaps


def raw(t):
    """Host numpy copy of a tensor's raw bits (bf16 as uint16), for byte-exact checks."""
    import torch
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().copy()


def from_raw(a, dtype):
    """Inverse of raw(): a torch tensor of `dtype` over the same bits."""
    import torch
    if dtype == torch.bfloat16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a))
