"""The device status word: data the method is not defined on is reported, not faulted on.

Eq. (1)'s softmax needs a positive finite normaliser for every window row, and
Sec. 3.2 samples in proportion to non-negative finite scores.  Inputs outside
that (a NaN or infinite key, query or value element; a NaN, infinite or
negative score into selection) must set the documented VASE_STATUS_* bit in the
caller's word, leave every kernel completing normally, and still give a valid
survivor map.  Clean inputs leave the word untouched.
"""
import numpy as np
import pytest
import torch

from paper_2606_03928_amd import synth, vase

from parity_util import survivor_check

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")

# (config, instances): the fused kernel (one workgroup per instance), slots split
# over workgroups (few instances), two row slabs (G*w = 1280), and fp32 (VALU path)
PATHS = [("qwen3-8b", 512), ("qwen3-8b", 8), ("qwen3-14b", 4), ("tiny", None)]


def _cfg(name):
    return synth.CONFIGS[name]


def _word():
    return torch.zeros(1, dtype=torch.int32, device=DEV)


def _round(x, cfg, st_score, st_select, value_kind=vase.VALUE_RANGE, ord=None):
    attn, vr = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool,
                          value_kind=value_kind, status=st_score, ord=ord)
    if vr is None:
        vr = torch.zeros_like(attn)
    src = vase.select(attn, vr, cfg.K, cfg.B, cfg.Nv, 5, 1, status=st_select)
    torch.cuda.synchronize()
    return attn, vr, src


@pytest.mark.parametrize("name,n", PATHS)
def test_clean_round_leaves_the_word_alone(name, n):
    cfg = _cfg(name)
    x = synth.make_round_inputs(cfg, DEV, seed=5, n_inst=n)
    a, b = _word(), _word()
    _round(x, cfg, a, b)
    assert a.item() == 0 and b.item() == 0


@pytest.mark.parametrize("name,n", PATHS)
@pytest.mark.parametrize("what", ["k_nan", "k_inf", "q_inf", "q_nan"])
def test_nonfinite_key_or_query_sets_row_norm(name, n, what):
    cfg = _cfg(name)
    x = synth.make_round_inputs(cfg, DEV, seed=6, n_inst=n)
    inst = x["k"].shape[0] - 1
    if what == "k_nan":
        x["k"][inst, 37, 5] = float("nan")
    elif what == "k_inf":
        x["k"][inst, cfg.K + 3, 0] = float("inf")        # a buffer slot: every row sums over it
    elif what == "q_inf":
        x["q_win"][inst, 0, 1, 9] = float("-inf")
    else:
        x["q_win"][0, cfg.G - 1, cfg.w - 1, 0] = float("nan")
    st, ss = _word(), _word()
    _, vr, src = _round(x, cfg, st, ss)
    assert st.item() & vase.STATUS_ROW_NORM
    assert not st.item() & vase.STATUS_VALUE_ROW
    # the NaN scores reach selection, which reports them and still emits a valid map
    assert ss.item() & vase.STATUS_SELECT_ATTN
    survivor_check(src.cpu().numpy(), cfg.K, cfg.B, np.zeros((src.shape[0], cfg.K)), 0)


@pytest.mark.parametrize("name,n", PATHS)
def test_nonfinite_value_row_sets_value_row(name, n):
    cfg = _cfg(name)
    x = synth.make_round_inputs(cfg, DEV, seed=7, n_inst=n)
    inst = x["k"].shape[0] // 2
    x["v"][inst, cfg.K - 1, cfg.d - 1] = float("nan")      # the last candidate row
    st = _word()
    _round(x, cfg, st, None)
    assert st.item() == vase.STATUS_VALUE_ROW
    # a buffer row is not a candidate: its value score is not computed, nor checked
    y = synth.make_round_inputs(cfg, DEV, seed=7, n_inst=n)
    y["v"][inst, cfg.K, 0] = float("inf")
    st = _word()
    _round(y, cfg, st, None)
    assert st.item() == 0
    # with the value scores supplied (VALUE_SKIP) no value row is read
    st = _word()
    _round(x, cfg, st, None, value_kind=vase.VALUE_SKIP)
    assert st.item() == 0


def test_value_row_checked_under_the_order_map():
    cfg = _cfg("qwen3-8b")
    x = synth.make_round_inputs(cfg, DEV, seed=8, n_inst=512)
    x["v"][300, 17, 3] = float("inf")
    ord_map = vase.identity_order(512, cfg.K, DEV)
    st = _word()
    _round(x, cfg, st, None, ord=ord_map)
    assert st.item() == vase.STATUS_VALUE_ROW


@pytest.mark.parametrize("bad", ["nan", "inf", "neg", "negzero"])
def test_select_reports_scores_outside_the_contract(bad):
    K, B, Nv, n = 4096, 128, 128, 64
    g = torch.Generator(device=DEV)
    g.manual_seed(3)
    attn = torch.rand((n, K), generator=g, device=DEV) * 1e-3
    vr = torch.rand((n, K), generator=g, device=DEV)
    val = {"nan": float("nan"), "inf": float("inf"), "neg": -1e-4, "negzero": -0.0}[bad]
    a2 = attn.clone()
    a2[7, 100:104] = val          # at most N_v = 128 slots are reserved: one of these is a candidate
    st = _word()
    src = vase.select(a2, vr, K, B, Nv, 1, 2, status=st)
    torch.cuda.synchronize()
    assert st.item() == vase.STATUS_SELECT_ATTN
    survivor_check(src.cpu().numpy(), K, B, np.zeros((n, K)), 0)
    v2 = vr.clone()
    v2[9, 4000] = val
    st = _word()
    src = vase.select(attn, v2, K, B, Nv, 1, 2, status=st)
    torch.cuda.synchronize()
    assert st.item() == vase.STATUS_SELECT_VALUE
    survivor_check(src.cpu().numpy(), K, B, np.zeros((n, K)), 0)
    # the word is never cleared by the library: a later clean call keeps the bit
    vase.select(attn, vr, K, B, Nv, 1, 2, status=st)
    torch.cuda.synchronize()
    assert st.item() == vase.STATUS_SELECT_VALUE


def test_status_is_optional_and_changes_no_output():
    cfg = _cfg("qwen3-8b")
    x = synth.make_round_inputs(cfg, DEV, seed=9, n_inst=512)
    a0, v0, s0 = _round(x, cfg, None, None)
    a1, v1, s1 = _round(x, cfg, _word(), _word())
    assert torch.equal(a0, a1) and torch.equal(v0, v1) and torch.equal(s0, s1)
