"""The boundary-swap check of the end-to-end parity tests, on planted cases (CPU).

explained_swaps must accept a swap only when the two slots' oracle keys lie
within the 1e-6 contract or within the bound that the slots' measured score
errors give, and must reject a GPU map that differs from the oracle's
selection on the GPU's own scores.
"""
import numpy as np
import pytest

from parity_util import SWAP_CONTRACT, explained_swaps


def _case(gap_rel, err_a=0.0, err_b=0.0):
    # one instance, K = 6, B = 2: buffer slots 6, 7 at the end; candidates 0..5,
    # the oracle evicts slots 4 and 5 (smallest keys), the GPU evicts 3 and 5
    K = 6
    keys = np.array([[9.0, 8.0, 7.0, 1.0, 1.0 - gap_rel, 0.5]], np.float32)
    src_ref = np.array([[0, 1, 2, 3, 6, 7]], np.int32)
    src_gpu = np.array([[0, 1, 2, 4, 6, 7]], np.int32)
    attn_ref = np.ones((1, K), np.float64)
    attn_gpu = attn_ref.copy()
    attn_gpu[0, 3] *= 1 - err_a
    attn_gpu[0, 4] *= 1 + err_b
    return src_gpu, src_ref, keys, K, attn_gpu, attn_ref


def test_identical_maps_have_no_swaps():
    src_gpu, src_ref, keys, K, ag, ar = _case(1e-7)
    st = explained_swaps(src_ref, src_ref, keys, K, ag, ar)
    assert st["count"] == 0 and st["max_gap"] == 0.0


def test_swap_inside_the_contract_passes():
    st = explained_swaps(*_case(5e-7))
    assert st["count"] == 1 and st["over_contract"] == 0
    assert 4e-7 < st["max_gap"] < SWAP_CONTRACT


def test_swap_explained_by_measured_errors_passes():
    # a gap of 3e-6 is above the contract, but the two scores were off by 2e-6 each
    st = explained_swaps(*_case(3e-6, err_a=2e-6, err_b=2e-6))
    assert st["count"] == 1 and st["over_contract"] == 1


def test_unexplained_swap_fails():
    with pytest.raises(AssertionError, match="above the 1e-6 contract"):
        explained_swaps(*_case(3e-6, err_a=1e-7, err_b=1e-7))
    with pytest.raises(AssertionError):
        explained_swaps(*_case(2e-4, err_a=1e-5, err_b=1e-5))


def test_selection_must_match_the_oracle_on_gpu_scores():
    src_gpu, src_ref, keys, K, ag, ar = _case(5e-7)
    with pytest.raises(AssertionError):
        explained_swaps(src_gpu, src_ref, keys, K, ag, ar, src_from_gpu=src_ref)
    explained_swaps(src_gpu, src_ref, keys, K, ag, ar, src_from_gpu=src_gpu)
