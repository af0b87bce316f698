"""Pins of the oracle's compaction under an order map (CPU only).

The order map keeps survivors in their slots and records the temporal order
separately; read through the map, the cache must be exactly the stable
compaction of the temporal cache (Sec. 2: after a round the cache holds the K
survivors), which numpy fancy indexing and the oracle's own stable compaction
both define independently of the map.
"""
import numpy as np
import pytest

import oracle


def random_src(rng, n_inst, K, B):
    """Valid survivor maps: K - B sorted candidates of [0, K), then the buffer."""
    out = np.empty((n_inst, K), np.int32)
    for i in range(n_inst):
        keep = np.sort(rng.choice(K, K - B, replace=False))
        out[i] = np.concatenate([keep, np.arange(K, K + B)])
    return out


def random_perm(rng, n_inst, K):
    return np.stack([rng.permutation(K) for _ in range(n_inst)]).astype(np.int32)


def temporal(x, ord_map):
    """The temporal cache seen through the order map: rank t < K at slot ord[t]."""
    K = ord_map.shape[1]
    rows = np.arange(x.shape[0])[:, None]
    return np.concatenate([x[rows, ord_map], x[:, K:]], axis=1)


def test_identity_map_moves_buffer_into_evicted_slots():
    rng = np.random.default_rng(0)
    K, B = 40, 6
    src = random_src(rng, 3, K, B)
    ident = np.tile(np.arange(K, dtype=np.int32), (3, 1))
    o_new, moves = oracle.order_compact(ident, src, B)
    for i in range(3):
        evicted = np.setdiff1d(np.arange(K), src[i, :K - B])
        np.testing.assert_array_equal(moves[i], evicted)           # holes are the evicted slots
        np.testing.assert_array_equal(o_new[i, :K - B], src[i, :K - B])
        np.testing.assert_array_equal(o_new[i, K - B:], evicted)


@pytest.mark.parametrize("K,B,n_inst,seed", [(16, 1, 4, 1), (64, 8, 5, 2), (130, 33, 3, 3),
                                             (9, 8, 6, 4)])
def test_map_view_equals_stable_compaction(K, B, n_inst, seed):
    rng = np.random.default_rng(seed)
    N, d = K + B, 3
    x = rng.standard_normal((n_inst, N, d)).astype(np.float32)
    y = rng.standard_normal((n_inst, N, d)).astype(np.float32)
    ord_map = random_perm(rng, n_inst, K)
    src = random_src(rng, n_inst, K, B)
    want_x = np.take_along_axis(temporal(x, ord_map), src[:, :, None].astype(np.int64), axis=1)
    want_y = np.take_along_axis(temporal(y, ord_map), src[:, :, None].astype(np.int64), axis=1)
    before = x.copy()
    o_new, moves = oracle.order_compact(ord_map, src, B)
    oracle.apply_moves(x, y, moves, K)
    # the new map is a permutation of the K slots and only B rows were written
    assert np.all(np.sort(o_new, axis=1) == np.arange(K))
    assert np.all(np.sort(moves, axis=1)[:, 1:] > np.sort(moves, axis=1)[:, :-1])
    changed = (x[:, :K] != before[:, :K]).any(axis=2)
    assert changed.sum(axis=1).max() <= B
    for i in range(n_inst):
        untouched = np.setdiff1d(np.arange(K), moves[i])
        np.testing.assert_array_equal(x[i, untouched], before[i, untouched])
    # read through the new map, the cache is the stable compaction
    np.testing.assert_array_equal(temporal(x, o_new)[:, :K], want_x)
    np.testing.assert_array_equal(temporal(y, o_new)[:, :K], want_y)


def test_rounds_track_the_stable_oracle():
    """Ten rounds from the identity map: the map view always equals the oracle's
    stable in-place compaction applied round after round."""
    rng = np.random.default_rng(7)
    n_inst, K, B, d = 3, 48, 8, 4
    N = K + B
    x = rng.integers(0, 1 << 16, (n_inst, N, d)).astype(np.uint16)
    y = rng.integers(0, 1 << 16, (n_inst, N, d)).astype(np.uint16)
    sx, sy = x.copy(), y.copy()          # stable layout
    ord_map = np.tile(np.arange(K, dtype=np.int32), (n_inst, 1))
    for _ in range(10):
        src = random_src(rng, n_inst, K, B)
        oracle.compact(sx, sy, src)
        ord_map, moves = oracle.order_compact(ord_map, src, B)
        oracle.apply_moves(x, y, moves, K)
        np.testing.assert_array_equal(temporal(x, ord_map)[:, :K], sx[:, :K])
        np.testing.assert_array_equal(temporal(y, ord_map)[:, :K], sy[:, :K])
        fresh = rng.integers(0, 1 << 16, (n_inst, B, d)).astype(np.uint16)
        fresh2 = rng.integers(0, 1 << 16, (n_inst, B, d)).astype(np.uint16)
        for a, b_ in ((x, fresh), (sx, fresh), (y, fresh2), (sy, fresh2)):
            a[:, K:] = b_


def test_invalid_maps_are_rejected():
    K, B = 10, 2
    ident = np.arange(K, dtype=np.int32)[None]
    bad = np.concatenate([np.arange(K - B - 1), [K - 1, K - 1], np.arange(K, K + B - 1)])[None]
    with pytest.raises(Exception):
        oracle.order_compact(ident, bad.astype(np.int32), B)       # a repeated survivor
    with pytest.raises(Exception):
        oracle.order_compact(ident, np.full((1, K), K + 5, np.int32), B)
