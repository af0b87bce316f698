"""GPU parity of VaSE-DKV (Sec. 3.2 with CurDKV's product score, Eq. 4): the
HIP library through its C ABI against the CPU oracle on the same seeded inputs.

  D1 the per-step Gaussian projections G_t, bit-exact (both sides run the same
     fixed binary32 sequence from the same Philox words);
  D2 the scores s_i = ||G^T k_i||^2 ||G^T v_i||^2 within the error bound of
     the arithmetic: each projection p_j = sum_a k_a G_aj is off by at most
     eps * sum_a |k_a G_aj| (bf16 caches: G enters the MFMA as a two-term bf16
     split, relative error below 2^-16, plus fp32 accumulation; eps = 2^-15),
     carried through l = sum_j p_j^2 and s = l_K l_V, plus 1e-6 relative.
     With r = 20 that is about 1e-5 relative; with r = 1 a projection can
     cancel to far below its terms, and the bound, not a relative one, holds;
  D3 selection from identical scores, bit-exact (deterministic top K-B);
  D4 whole rounds: survivor sets agree except boundary swaps explained by the
     score tolerance;
  D5 the decode logits the score pass leaves (q_dec . k over all N slots):
     within fp32 accumulation error of q.k in float64, the scores unchanged bit
     for bit, and whole map-layout rounds whose decode reads them against the
     oracle.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03928_amd import synth, vase

from parity_util import assert_decode_close, from_raw, raw, survivor_check

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
DKV_EPS = 2.0 ** -15


@pytest.fixture(autouse=True)
def _lib(gpu_lib):
    yield
    torch.cuda.synchronize()


def _cfg(name, **kw):
    return synth.CONFIGS[name].with_(**kw) if kw else synth.CONFIGS[name]


@pytest.mark.parametrize("n_inst,base,d,r,seed,rnd", [
    (3, 0, 128, 20, 0, 0), (5, 1000, 64, 20, 0xDEADBEEFCAFE, 77), (2, 7, 128, 1, 3, 1),
    (2, 0, 128, 32, 9, 2 ** 31 + 5),
])
def test_projection_bitexact(n_inst, base, d, r, seed, rnd):
    g = vase.dkv_projection(n_inst, d, seed, rnd, r=r, inst_base=base, device=DEV)
    torch.cuda.synchronize()
    got = g.cpu().numpy()
    for i in range(n_inst):
        ref = oracle.dkv_gaussian(seed, base + i, rnd, d, r)
        np.testing.assert_array_equal(got[i].view(np.uint32), ref.view(np.uint32))


def _rel_err(got, ref):
    return float(np.max(np.abs(got.astype(np.float64) - ref) / np.maximum(np.abs(ref), 1e-30)))


def _bound(k, v, g, K):
    """Error bound of a DKV score computed with projections accurate to
    DKV_EPS * sum_a |x_a G_aj| (see the module docstring)."""
    gg = g.astype(np.float64)
    out = []
    for x in (k, v):
        xx = x[:, :K].double().numpy() if isinstance(x, torch.Tensor) else x[:, :K]
        p = np.einsum("nia,nar->nir", xx, gg)
        dp = DKV_EPS * np.einsum("nia,nar->nir", np.abs(xx), np.abs(gg))
        out.append((np.sum(p * p, -1), np.sum(2 * np.abs(p) * dp + dp * dp, -1)))
    (lk, dlk), (lv, dlv) = out
    return dlk * lv + lk * dlv + dlk * dlv + 1e-6 * lk * lv


def _assert_within(got, ref, bound):
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    bad = err > bound
    assert not bad.any(), (err[bad][:5], bound[bad][:5])


SCORE_CASES = [
    ("tiny", {}, None, 20),
    ("tiny", dict(dtype="bf16"), None, 20),
    ("qwen3-1.7b", {}, None, 20),
    ("qwen3-8b", {}, 48, 20),
    ("qwen3-8b", dict(d=64), 16, 20),
    ("qwen3-8b", dict(K=1000, B=24), 8, 20),          # ragged tiles
    ("qwen3-8b", {}, 8, 1),
    ("qwen3-8b", {}, 8, 32),
    ("qwen3-8b", dict(dtype="f32"), 4, 20),
]


@pytest.mark.parametrize("name,kw,n_inst,r", SCORE_CASES)
def test_score_parity(name, kw, n_inst, r):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=21, n_inst=n_inst)
    n = x["k"].shape[0]
    g = vase.dkv_projection(n, cfg.d, seed=5, round=3, r=r, device=DEV)
    s = vase.dkv_score(x["k"], x["v"], g, cfg.K, cfg.B)
    torch.cuda.synchronize()
    k_h, v_h = x["k"].cpu(), x["v"].cpu()
    ref = oracle.dkv_score_g(k_h, v_h, g.cpu().numpy(), cfg.K)
    _assert_within(s.cpu().numpy(), ref, _bound(k_h, v_h, g.cpu().numpy(), cfg.K))
    err = _rel_err(s.cpu().numpy(), ref)
    # and the oracle's own draw of G gives the same reference
    np.testing.assert_array_equal(ref, oracle.dkv_score(k_h, v_h, cfg.K, 5, 3, r=r))
    print("%s %s r=%d: max relative DKV score error %.3g" % (name, kw, r, err))


def test_full_8b_sampled():
    cfg = _cfg("qwen3-8b")
    x = synth.make_round_inputs(cfg, DEV, seed=22)
    n = cfg.n_inst
    g = vase.dkv_projection(n, cfg.d, seed=1, round=0, device=DEV)
    s = vase.dkv_score(x["k"], x["v"], g, cfg.K, cfg.B)
    torch.cuda.synchronize()
    sample = [0, 1, 1234, n - 1]
    ks, vs, gs = x["k"][sample].cpu(), x["v"][sample].cpu(), g[sample].cpu().numpy()
    ref = oracle.dkv_score_g(ks, vs, gs, cfg.K)
    _assert_within(s[sample].cpu().numpy(), ref, _bound(ks, vs, gs, cfg.K))
    assert torch.all(s >= 0) and torch.all(torch.isfinite(s))


@pytest.mark.parametrize("name,n_inst,rounds", [("tiny", None, 3), ("qwen3-1.7b", None, 20)])
def test_rounds_end_to_end(name, n_inst, rounds):
    cfg = _cfg(name)
    x = synth.make_round_inputs(cfg, DEV, seed=23, n_inst=n_inst)
    n = x["k"].shape[0]
    seed = 99
    zeros = torch.zeros((n, cfg.K), dtype=torch.float32, device=DEV)
    n_swaps = 0
    for rnd in range(rounds):
        k_h, v_h = x["k"].cpu(), x["v"].cpu()
        g = vase.dkv_projection(n, cfg.d, seed, rnd, device=DEV)
        s = vase.dkv_score(x["k"], x["v"], g, cfg.K, cfg.B)
        src = vase.select(s, zeros, cfg.K, cfg.B, 0, seed, rnd, flags=vase.DETERMINISTIC)
        out = vase.compact_decode(x["k"], x["v"], src, x["q_dec"], cfg.K, cfg.B)
        torch.cuda.synchronize()
        s_g, src_g = s.cpu().numpy(), src.cpu().numpy()
        survivor_check(src_g, cfg.K, cfg.B, np.zeros((n, cfg.K), np.float32), 0)
        # D3: selection from the GPU's scores is bit-exact
        np.testing.assert_array_equal(
            src_g, oracle.select(s_g, np.zeros_like(s_g), cfg.K, cfg.B, 0, seed, rnd,
                                 flags=oracle.FLAG_DETERMINISTIC))
        # D4: against the oracle's own round
        ref_s, ref_src = oracle.dkv_round(k_h, v_h, cfg.K, cfg.B, seed, rnd)
        bnd = _bound(k_h, v_h, g.cpu().numpy(), cfg.K)
        _assert_within(s_g, ref_s, bnd)
        for i in range(n):
            a, b = set(src_g[i].tolist()), set(ref_src[i].tolist())
            only_gpu, only_ref = sorted(a - b), sorted(b - a)
            assert len(only_gpu) == len(only_ref)
            for p, q in zip(only_gpu, only_ref):
                # a swap across the cut is allowed only between scores that the
                # error bound cannot tell apart
                assert abs(float(ref_s[i, p]) - float(ref_s[i, q])) <= bnd[i, p] + bnd[i, q]
            n_swaps += len(only_gpu)
        # compaction and decode of the GPU's own map, against the oracle
        kk, vv = raw(k_h), raw(v_h)
        oracle.compact(kk, vv, src_g)
        np.testing.assert_array_equal(raw(x["k"].cpu())[:, :cfg.K], kk[:, :cfg.K])
        ref_out = oracle.decode(x["q_dec"].cpu(), from_raw(kk, cfg.torch_dtype),
                                from_raw(vv, cfg.torch_dtype), cfg.K)
        assert_decode_close(out.float().cpu().numpy(), ref_out, bf16=cfg.dtype == "bf16")
        synth.refresh_buffer(x, cfg, step_seed=rnd)
    print("%s: %d DKV rounds, %d boundary swaps" % (name, rounds, n_swaps))


DL_CASES = [
    ("qwen3-1.7b", {}, None),
    ("qwen3-8b", {}, 48),
    ("qwen3-8b", dict(d=64), 16),
    ("qwen3-8b", dict(K=1000, B=23), 8),        # ragged tiles, N odd
    ("qwen3-14b", {}, 4),                        # G = 5, the buffer spanning a block
]


@pytest.mark.parametrize("name,kw,n_inst", DL_CASES)
def test_score_decode_logits(name, kw, n_inst):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=24, n_inst=n_inst)
    n, N = x["k"].shape[0], cfg.K + cfg.B
    g = vase.dkv_projection(n, cfg.d, seed=6, round=2, device=DEV)
    s0 = vase.dkv_score(x["k"], x["v"], g, cfg.K, cfg.B)
    dl = torch.full((n, cfg.G, N), float("nan"), dtype=torch.float32, device=DEV)
    s1 = vase.dkv_score(x["k"], x["v"], g, cfg.K, cfg.B, q_dec=x["q_dec"], dec_logits=dl)
    torch.cuda.synchronize()
    assert torch.equal(s0, s1)
    q = x["q_dec"].cpu().double()
    k = x["k"].cpu().double()
    ref = torch.matmul(q, k.transpose(1, 2))
    bound = torch.matmul(q.abs(), k.abs().transpose(1, 2))
    got = dl.cpu().double()
    assert torch.isfinite(got).all()
    err = (got - ref).abs()
    assert (err <= 1e-5 * bound + 1e-30).all(), float((err / bound.clamp_min(1e-30)).max())


@pytest.mark.parametrize("name,n_inst,rounds", [("qwen3-1.7b", None, 6), ("qwen3-8b", 32, 3)])
def test_map_rounds_with_decode_logits(name, n_inst, rounds):
    """DKV rounds under the order map whose decode takes the score's logits."""
    cfg = _cfg(name)
    x = synth.make_round_inputs(cfg, DEV, seed=25, n_inst=n_inst)
    n, K, B = x["k"].shape[0], cfg.K, cfg.B
    rb = vase.Round(n, K, B, cfg.d, cfg.G, cfg.w, cfg.torch_dtype, DEV, layout="map")
    assert rb.dec_logits is not None
    zeros = torch.zeros((n, K), dtype=torch.float32, device=DEV)
    phys = torch.empty((n, K), dtype=torch.float32, device=DEV)
    seed = 98
    for rnd in range(rounds):
        kt_h, vt_h = rb.temporal(x["k"]).cpu(), rb.temporal(x["v"]).cpu()
        g = vase.dkv_projection(n, cfg.d, seed, rnd, device=DEV)
        vase.dkv_score(x["k"], x["v"], g, K, B, out=phys, q_dec=x["q_dec"], dec_logits=rb.dec_logits)
        vase.order_scores(phys, rb.ord, 1, attn=rb.attn)
        vase.select(rb.attn, zeros, K, B, 0, seed, rnd, flags=vase.DETERMINISTIC, src=rb.src)
        out = vase.compact_decode_map(x["k"], x["v"], rb.src, rb.ord, K, B, q=x["q_dec"],
                                      dec_logits=rb.dec_logits)
        torch.cuda.synchronize()
        src_g = rb.src.cpu().numpy()
        survivor_check(src_g, K, B, np.zeros((n, K), np.float32), 0)
        kk, vv = raw(kt_h), raw(vt_h)
        oracle.compact(kk, vv, src_g)
        np.testing.assert_array_equal(raw(rb.temporal(x["k"]).cpu())[:, :K], kk[:, :K])
        np.testing.assert_array_equal(raw(rb.temporal(x["v"]).cpu())[:, :K], vv[:, :K])
        ref_out = oracle.decode(x["q_dec"].cpu(), from_raw(kk, cfg.torch_dtype),
                                from_raw(vv, cfg.torch_dtype), K)
        err = assert_decode_close(out.float().cpu().numpy(), ref_out, bf16=True)
        synth.refresh_buffer(x, cfg, step_seed=rnd)
    assert not torch.equal(rb.ord, vase.identity_order(n, K, DEV))
    print("%s: %d DKV map rounds from the score's logits, last decode error %.3g" % (name, rounds, err))
