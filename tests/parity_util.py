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


# P4 contract: a boundary swap between the GPU's and the oracle's survivor sets is
# allowed when the two slots' oracle keys differ by less than 1e-6 relative
SWAP_CONTRACT = 1e-6
# two IEEE fp32 divides (attn / E on each side) and the fp32 rounding of the
# oracle's score: 2^-22 relative covers them
_KEY_ROUNDING = 2.0 ** -22


def explained_swaps(src_gpu, src_ref, keys_ref, K, attn_gpu, attn_ref, src_from_gpu=None):
    """Differences between the GPU's and the oracle's survivor maps, as boundary swaps.

    A slot a kept by the oracle and evicted by the GPU, and a slot b kept by the
    GPU and evicted by the oracle, are a swap.  Both sides draw the same E from the
    same Philox words, so key_gpu(s) / key_ref(s) = attn_gpu(s) / attn_ref(s) up to
    the rounding of the two divides: with e_s the measured relative error of slot
    s's GPU score, key_ref(a) >= key_ref(b) and key_gpu(b) >= key_gpu(a) give

        (key_ref(a) - key_ref(b)) / key_ref(a) <= e_a + e_b + 2^-22.

    Every pair (a, b) of an instance must satisfy the contract (gap < 1e-6) or
    this derived bound.  With src_from_gpu (the oracle's selection run on the
    GPU's own scores) the GPU map must equal it bit for bit, so that every
    difference comes from the scores and none from selection.

    Returns a dict: count (swapped pairs), max_gap, over_contract (pairs whose gap
    is >= 1e-6 and which the derived bound explains), swaps (list of (instance,
    evicted_by_gpu, evicted_by_oracle, gap, bound)).
    """
    src_gpu = np.asarray(src_gpu)
    src_ref = np.asarray(src_ref)
    if src_from_gpu is not None:
        np.testing.assert_array_equal(src_gpu, src_from_gpu)
    ag = np.asarray(attn_gpu, np.float64)
    ar = np.asarray(attn_ref, np.float64)
    err = np.abs(ag - ar) / np.maximum(np.abs(ar), 1e-300)
    out = {"count": 0, "max_gap": 0.0, "over_contract": 0, "swaps": []}
    for i in np.nonzero((src_gpu != src_ref).any(axis=1))[0]:
        kept_g = set(src_gpu[i][src_gpu[i] < K].tolist())
        kept_r = set(src_ref[i][src_ref[i] < K].tolist())
        only_r = sorted(kept_r - kept_g)      # the GPU evicted these
        only_g = sorted(kept_g - kept_r)      # the oracle evicted these
        assert len(only_r) == len(only_g), "instance %d: survivor counts differ" % i
        for a in only_r:
            for b in only_g:
                ka, kb = float(keys_ref[i, a]), float(keys_ref[i, b])
                gap = (ka - kb) / max(abs(ka), 1e-300)
                bound = err[i, a] + err[i, b] + _KEY_ROUNDING
                assert gap < SWAP_CONTRACT or gap <= bound * (1 + 1e-6), (
                    "instance %d: slots %d/%d swapped with key gap %.3g, above the 1e-6 contract "
                    "and the %.3g their score errors explain" % (i, a, b, gap, bound))
                out["max_gap"] = max(out["max_gap"], gap)
                out["over_contract"] += int(gap >= SWAP_CONTRACT)
        for a, b in zip(only_r, only_g):
            ka, kb = float(keys_ref[i, a]), float(keys_ref[i, b])
            out["swaps"].append((int(i), int(a), int(b), (ka - kb) / max(abs(ka), 1e-300),
                                 float(err[i, a] + err[i, b] + _KEY_ROUNDING)))
        out["count"] += len(only_r)
    return out


def swap_report(name, stats_list, n_rounds, n_evicted):
    """One line for the test log: swaps over all checked rounds against evictions."""
    cnt = sum(s["count"] for s in stats_list)
    gap = max([s["max_gap"] for s in stats_list] + [0.0])
    over = sum(s["over_contract"] for s in stats_list)
    line = ("%s: %d checked rounds, %d evictions, %d boundary swaps, largest key gap %.3g "
            "(%d at or above 1e-6, each within its derived bound)" % (name, n_rounds, n_evicted, cnt,
                                                                      gap, over))
    print(line)
    return {"swaps": cnt, "max_gap": gap, "over_contract": over, "evictions": n_evicted}


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
