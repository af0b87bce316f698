"""GPU parity of the decode-side integration: decode attention that also returns the
persistent-slot log-sum-exp, the decode step (append, window ring, attention,
normaliser part), and the one-pass window score that reuses it.

Bars:
  L1 out within the decode tolerance; the LSE within the fp32 error bound
     below, against the oracle's double-precision value;
  L2 the appended rows and the window ring are byte-exact;
  L3 the one-pass score within 1e-4 relative of the oracle's score (and of the
     two-pass GPU score), on every score-kernel path; with a supplied normaliser
     that is not the true one, it follows the oracle's score_lse instead;
  L4 whole periods (B decode steps, then a round with the one-pass score) end
     to end against the oracle, up to explained boundary swaps.

LSE bound: each score q.k/sqrt(d) is an fp32 dot product of d terms, off by at
most (d + 1) 2^-24 sum_e |q_e k_e| / sqrt(d); the log-sum-exp moves by at most
the largest score error, plus the relative error of the sum of n exponentials
((n + 8) 2^-24, exp2 included) and the final log and scaling (4 2^-24 |lse|).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_03928_amd import synth, vase

from parity_util import (assert_attn_close, assert_decode_close, explained_swaps, raw, swap_report,
                         survivor_check)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
EPS = 2.0 ** -24


@pytest.fixture(autouse=True)
def _lib(gpu_lib):
    yield
    torch.cuda.synchronize()


def _cfg(name, **kw):
    return synth.CONFIGS[name].with_(**kw) if kw else synth.CONFIGS[name]


def _lse_bound(q, k, n, ref):
    """q [n_inst, G, d], k [n_inst, >=n, d] (host float64), ref [n_inst, G]."""
    d = q.shape[-1]
    sabs = np.einsum("igd,ikd->igk", np.abs(q), np.abs(k[:, :n])).max(axis=-1) / math.sqrt(d)
    return (d + 1) * EPS * sabs + (n + 8) * EPS + 4 * EPS * np.abs(ref)


def _assert_lse_close(got, q, k, n, ref):
    got = np.asarray(got, np.float64)
    bound = _lse_bound(q, k, n, ref)
    err = np.abs(got - ref)
    if (err > bound).any():
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError("lse: worst at %s: got %r ref %r err %g bound %g"
                             % (i, got[i], ref[i], err[i], bound[i]))
    return float(err.max())


def _h64(t):
    return t.detach().cpu().double().numpy()


# --------------------------------------------------------------------------
# L1: decode attention with the persistent-slot LSE
# --------------------------------------------------------------------------
@pytest.mark.parametrize("name,kw,n_inst,nv,npers", [
    ("tiny", {}, None, 160, 128),
    ("tiny", {}, None, 128, 128),
    ("tiny", {}, None, 1, 1),
    ("tiny", dict(d=128), None, 100, 37),
    ("qwen3-1.7b", {}, None, 2176, 2048),          # many splits, boundary at K
    ("qwen3-1.7b", {}, None, 2048 + 37, 2048),
    ("qwen3-1.7b", dict(d=64, h_q=40), 3, 2176, 1),  # G = 5, one persistent slot
    ("qwen3-8b", {}, 300, 4224, 4096),             # several splits per instance
    ("qwen3-8b", {}, 300, 4100, 4096),
    # enough instances for one split per instance: the buffer rows share the
    # persistent slots' workgroup (n_persist a multiple of 16), or get one of
    # their own (n_persist = 4001)
    ("qwen3-8b", {}, 4096, 4224, 4096),
    ("qwen3-8b", {}, 4096, 4224, 4001),
    ("qwen3-32b", {}, 5, 8320, 8192),              # G = 8
    ("qwen3-32b", dict(d=64), 3, 8200, 8192),
])
def test_decode_lse_parity(name, kw, n_inst, nv, npers):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=31, n_inst=n_inst)
    out, lse = vase.decode_attn(x["k"], x["v"], x["q_dec"], cfg.K, cfg.B, nv, n_persist=npers)
    torch.cuda.synchronize()
    sample = slice(None) if x["k"].shape[0] <= 16 else [0, 1, x["k"].shape[0] - 1]
    q, k = x["q_dec"][sample].cpu(), x["k"][sample].cpu()
    ref_lse = oracle.decode_lse(q, k, npers)
    err = _assert_lse_close(lse[sample].cpu().numpy(), _h64(q), _h64(k), npers, ref_lse)
    ref_out = oracle.decode(q, k, x["v"][sample].cpu(), nv)
    assert_decode_close(out[sample].float().cpu().numpy(), ref_out, bf16=cfg.dtype == "bf16")
    # the plain call gives the same output bits
    out2 = vase.decode_attn(x["k"], x["v"], x["q_dec"], cfg.K, cfg.B, nv)
    torch.cuda.synchronize()
    if npers == nv:
        assert torch.equal(out, out2)
    print("%s %s n_valid=%d n_persist=%d: max lse error %.3g" % (name, kw, nv, npers, err))


# --------------------------------------------------------------------------
# L2 + L3 after one period of decode steps
# --------------------------------------------------------------------------
def _new_rows(cfg, n, pos, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(1000003 * seed + pos)
    kn = torch.randn((n, cfg.d), generator=g, device=DEV).to(cfg.torch_dtype)
    vn = torch.randn((n, cfg.d), generator=g, device=DEV)
    vn[torch.rand((n, 1), generator=g, device=DEV).expand_as(vn) < 0.05] *= 30.0
    q = torch.randn((n, cfg.G, cfg.d), generator=g, device=DEV).to(cfg.torch_dtype)
    return kn, vn.to(cfg.torch_dtype), q


def _period(cfg, x, q_win, lse_win, seed, check_every=0):
    """B decode steps into the buffer; returns the per-step (pos, out, q, kn, vn) checks."""
    n = x["k"].shape[0]
    checked = []
    for pos in range(cfg.B):
        kn, vn, q = _new_rows(cfg, n, pos, seed)
        out = vase.decode_step(x["k"], x["v"], kn, vn, q, cfg.K, cfg.B, pos, q_win, lse_win)
        if check_every and (pos % check_every == 0 or pos == cfg.B - 1):
            torch.cuda.synchronize()
            checked.append((pos, out.clone(), q.clone(), x["k"].clone(), x["v"].clone()))
        x.setdefault("_rows", []).append((kn, vn, q))
    return checked


@pytest.mark.parametrize("name,kw,n_inst,check_every", [
    ("tiny", {}, None, 1),                     # w = 8 < B = 32: the ring wraps four times
    ("tiny", dict(dtype="bf16", d=128), None, 5),
    ("qwen3-1.7b", {}, None, 16),
])
def test_decode_period_then_one_pass_score(name, kw, n_inst, check_every):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=41, n_inst=n_inst)
    n = x["k"].shape[0]
    q_win = torch.zeros_like(x["q_win"])
    lse_win = torch.full((n, cfg.G, cfg.w), float("nan"), dtype=torch.float32, device=DEV)
    k_before = raw(x["k"])
    checks = _period(cfg, x, q_win, lse_win, seed=3, check_every=check_every)
    torch.cuda.synchronize()
    # per-step outputs and persistent LSEs against the oracle over K + pos + 1 slots
    for pos, out, q, kc, vc in checks:
        ref = oracle.decode(q.cpu(), kc.cpu(), vc.cpu(), cfg.K + pos + 1)
        assert_decode_close(out.float().cpu().numpy(), ref, bf16=cfg.dtype == "bf16")
    # L2: the buffer holds the appended rows, the persistent slots are untouched,
    # and the ring holds the last w queries at slot pos % w
    kr, vr = raw(x["k"]), raw(x["v"])
    np.testing.assert_array_equal(kr[:, :cfg.K], k_before[:, :cfg.K])
    for pos, (kn, vn, q) in enumerate(x["_rows"]):
        np.testing.assert_array_equal(kr[:, cfg.K + pos], raw(kn))
        np.testing.assert_array_equal(vr[:, cfg.K + pos], raw(vn))
        if pos >= cfg.B - cfg.w:
            np.testing.assert_array_equal(raw(q_win)[:, :, pos % cfg.w], raw(q))
    # the ring's LSEs are the persistent normalisers of its queries
    qw = q_win.cpu()
    kh = x["k"].cpu()
    R = cfg.G * cfg.w
    ref_lse = oracle.decode_lse(qw.reshape(n, R, cfg.d), kh, cfg.K).reshape(n, cfg.G, cfg.w)
    _assert_lse_close(lse_win.cpu().numpy().reshape(n, R), _h64(qw).reshape(n, R, cfg.d),
                      _h64(kh), cfg.K, ref_lse.reshape(n, R))
    # L3: the one-pass score against the oracle and against the two-pass score
    attn1, vr1 = vase.score(x["k"], x["v"], q_win, cfg.K, cfg.B, cfg.pool, lse_win=lse_win)
    attn2, vr2 = vase.score(x["k"], x["v"], q_win, cfg.K, cfg.B, cfg.pool)
    torch.cuda.synchronize()
    ref_attn = oracle.score(qw, kh, cfg.K, cfg.pool)
    rel = assert_attn_close(attn1.cpu().numpy(), ref_attn)
    assert_attn_close(attn2.cpu().numpy(), ref_attn)
    assert torch.equal(vr1, vr2)
    print("%s %s: one-pass score max relative error %.3g" % (name, kw, rel))


# --------------------------------------------------------------------------
# L3 on every score-kernel path, with window LSEs from decode_attn
# --------------------------------------------------------------------------
def _window_lse(x, cfg):
    n = x["k"].shape[0]
    lse = torch.empty((n, cfg.G, cfg.w), dtype=torch.float32, device=DEV)
    col = torch.empty((n, cfg.G), dtype=torch.float32, device=DEV)
    for t in range(cfg.w):
        q = x["q_win"][:, :, t].contiguous()
        vase.decode_attn(x["k"], x["v"], q, cfg.K, cfg.B, cfg.K, n_persist=cfg.K, lse=col)
        lse[:, :, t] = col
    return lse


@pytest.mark.parametrize("name,kw,n_inst,sample", [
    ("tiny", {}, None, None),
    ("tiny", dict(d=128, w=5, K=100, B=13, pool=5), None, None),
    ("qwen3-1.7b", dict(d=64, pool=1), 4, None),
    ("qwen3-8b", {}, 12, None),                                   # several ranges per instance
    ("qwen3-14b", {}, 4, None),                                   # two row slabs, G = 5
    ("qwen3-8b", dict(K=1000, B=24, w=24), 6, None),              # ragged chunks and buffer
    ("qwen3-8b", {}, 512, [0, 1, 511]),                           # one workgroup per instance
    ("qwen3-8b", dict(d=64, w=64), 600, [0, 599]),
])
def test_one_pass_score_paths(name, kw, n_inst, sample):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=51, n_inst=n_inst)
    lse = _window_lse(x, cfg)
    for kind in (vase.VALUE_RANGE, vase.VALUE_RANDOM):
        attn1, vr1 = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, lse_win=lse,
                                value_kind=kind, seed=5, round=2)
        attn2, vr2 = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool,
                                value_kind=kind, seed=5, round=2)
        torch.cuda.synchronize()
        assert torch.equal(vr1, vr2)
        assert_attn_close(attn1.cpu().numpy(), attn2.cpu().numpy().astype(np.float64), "vs two-pass")
    sel = slice(None) if sample is None else sample
    ref = oracle.score(x["q_win"][sel].cpu(), x["k"][sel].cpu(), cfg.K, cfg.pool)
    rel = assert_attn_close(attn1[sel].cpu().numpy(), ref)
    print("%s %s: one-pass max relative error %.3g" % (name, kw, rel))


@pytest.mark.parametrize("name,kw,n_inst", [
    ("tiny", {}, None),
    ("qwen3-1.7b", {}, 3),
    ("qwen3-8b", {}, 2),
])
def test_one_pass_score_follows_supplied_normaliser(name, kw, n_inst):
    """The kernel uses lse_win as given: with a perturbed normaliser it matches the
    oracle's score_lse on the same perturbed input, not the true score."""
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=61, n_inst=n_inst)
    n = x["k"].shape[0]
    R = cfg.G * cfg.w
    qh, kh = x["q_win"].cpu(), x["k"].cpu()
    true = oracle.decode_lse(qh.reshape(n, R, cfg.d), kh, cfg.K)
    shift = np.random.default_rng(7).uniform(-0.7, 0.7, size=true.shape)
    lse_in = (true + shift).astype(np.float32)
    lse_dev = torch.from_numpy(lse_in.reshape(n, cfg.G, cfg.w)).to(DEV)
    attn, _ = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, lse_win=lse_dev)
    torch.cuda.synchronize()
    ref = oracle.score_lse(qh, kh, cfg.K, cfg.pool, lse_in.astype(np.float64).reshape(n, cfg.G, cfg.w))
    assert_attn_close(attn.cpu().numpy(), ref)
    assert not np.allclose(ref, oracle.score(qh, kh, cfg.K, cfg.pool), rtol=1e-3)


# --------------------------------------------------------------------------
# L4: periods end to end
# --------------------------------------------------------------------------
@pytest.mark.parametrize("name,periods", [("tiny", 3), ("qwen3-1.7b", 3)])
def test_periods_end_to_end(name, periods):
    cfg = _cfg(name)
    x = synth.make_round_inputs(cfg, DEV, seed=71)
    n = x["k"].shape[0]
    q_win = torch.zeros_like(x["q_win"])
    lse_win = torch.zeros((n, cfg.G, cfg.w), dtype=torch.float32, device=DEV)
    seed = 99
    swaps_all = []
    for per in range(periods):
        x.pop("_rows", None)
        _period(cfg, x, q_win, lse_win, seed=per)
        torch.cuda.synchronize()
        qh, kh, vh = q_win.cpu(), x["k"].cpu(), x["v"].cpu()
        attn, vr = vase.score(x["k"], x["v"], q_win, cfg.K, cfg.B, cfg.pool, lse_win=lse_win)
        src = vase.select(attn, vr, cfg.K, cfg.B, cfg.Nv, seed, per)
        out = vase.compact_decode(x["k"], x["v"], src, x["q_dec"], cfg.K, cfg.B)
        torch.cuda.synchronize()
        src_g = src.cpu().numpy()
        survivor_check(src_g, cfg.K, cfg.B, vr.cpu().numpy(), cfg.Nv)
        ref_attn = oracle.score(qh, kh, cfg.K, cfg.pool)
        assert_attn_close(attn.cpu().numpy(), ref_attn)
        ref_vr = oracle.vrange(vh, cfg.K)
        np.testing.assert_array_equal(vr.cpu().numpy(), ref_vr)
        ref_src, ref_keys = oracle.select(ref_attn, ref_vr, cfg.K, cfg.B, cfg.Nv, seed, per,
                                          return_keys=True)
        a_g = attn.cpu().numpy()
        swaps_all.append(explained_swaps(src_g, ref_src, ref_keys, cfg.K, a_g, ref_attn,
                                         src_from_gpu=oracle.select(a_g, ref_vr, cfg.K, cfg.B,
                                                                    cfg.Nv, seed, per)))
        kk, vv = raw(kh), raw(vh)
        oracle.compact(kk, vv, src_g)
        np.testing.assert_array_equal(raw(x["k"])[:, :cfg.K], kk[:, :cfg.K])
        np.testing.assert_array_equal(raw(x["v"])[:, :cfg.K], vv[:, :cfg.K])
        del out
    rep = swap_report("%s periods" % name, swaps_all, periods, periods * n * cfg.B)
    assert rep["swaps"] <= max(1, rep["evictions"] // 1000)
