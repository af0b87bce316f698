"""GPU parity of the value-score variants (Appendix A: L2, Var; Appendix D: random
reservation) through vase_score_ex, against the CPU oracle.

Bars:
  V1 L2 and Var within the fp32 error bound of their sums (below), Range and
     random reservation bit-exact;
  V2 the attention score of vase_score_ex is bit-identical to vase_score's;
  V3 a whole round with a variant selects, from the GPU's value scores and the
     oracle's attention score, the oracle's survivors up to boundary swaps that
     the attention tolerance explains.

Error bound for L2 and Var: both sum d terms in fp32, so the sum is within
gamma_d = d * 2^-24 of its exact value relative to the sum of |terms|
(here the terms are nonnegative); sqrt halves the relative error of L2.  Var is
two-pass: an error delta in the mean adds d * delta^2 to the sum of squares,
with |delta| <= gamma_d * mean|v|.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03928_amd import synth, vase

from parity_util import assert_attn_close, explained_swaps, survivor_check, swap_report

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
KINDS = {"l2": vase.VALUE_L2, "var": vase.VALUE_VAR, "range": vase.VALUE_RANGE}


@pytest.fixture(autouse=True)
def _lib(gpu_lib):
    yield
    torch.cuda.synchronize()


def _cfg(name, **kw):
    return synth.CONFIGS[name].with_(**kw) if kw else synth.CONFIGS[name]


def _assert_value_close(got, v_rows, ref, kind):
    """got, ref: [n, K] scores; v_rows: the [n, K, d] value rows they came from."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if kind == vase.VALUE_RANGE:
        np.testing.assert_array_equal(got, ref)
        return 0.0
    v = np.asarray(v_rows, np.float64)
    d = v.shape[-1]
    gamma = (d + 2) * 2.0 ** -24
    if kind == vase.VALUE_L2:
        bound = (gamma / 2 + 2.0 ** -24) * ref + 2.0 ** -24 * np.abs(ref)
    else:
        mabs = np.abs(v).mean(axis=-1)
        bound = (gamma + 2.0 ** -24) * ref + (gamma * mabs) ** 2 + 1e-37
    err = np.abs(got - ref)
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError("%d of %d outside the bound; worst at %s: got %r ref %r bound %g"
                             % (int(bad.sum()), bad.size, i, got[i], ref[i], bound[i]))
    rel = err / np.maximum(ref, 1e-300)
    return float(rel[ref > 0].max(initial=0.0))


CASES = [
    ("tiny", {}, None, None),
    ("tiny", dict(dtype="bf16"), None, None),
    ("tiny", dict(d=128, w=5, K=100, B=13, pool=5), None, None),    # ragged tiles
    ("qwen3-1.7b", dict(d=64, pool=1), 4, None),
    ("qwen3-8b", {}, 12, None),                                    # several ranges per instance
    ("qwen3-14b", {}, 4, None),                                    # two row slabs
    ("qwen3-8b", dict(K=1000, B=24, w=40), 6, None),               # ragged key chunks
    ("qwen3-8b", {}, 512, [0, 1, 255, 511]),                       # one workgroup per instance
    ("qwen3-8b", dict(d=64, w=64), 600, [0, 599]),
]


@pytest.mark.parametrize("kind", ["l2", "var", "range"])
@pytest.mark.parametrize("name,kw,n_inst,sample", CASES)
def test_value_score_parity(name, kw, n_inst, sample, kind):
    cfg = _cfg(name, **kw)
    kd = KINDS[kind]
    x = synth.make_round_inputs(cfg, DEV, seed=21, n_inst=n_inst)
    attn0, _ = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool)
    attn, val = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, value_kind=kd)
    torch.cuda.synchronize()
    assert torch.equal(attn, attn0)
    sel = slice(None) if sample is None else sample
    v_s = x["v"][sel].cpu()
    ref = oracle.value_score(v_s, cfg.K, kd)
    rel = _assert_value_close(val[sel].cpu().numpy(), v_s[:, :cfg.K].double().numpy(), ref, kd)
    print("%s %s %s: max relative error %.3g" % (name, kw, kind, rel))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_value_score_degenerate_rows(dtype):
    """Constant rows (Range = Var = 0), rows on a large offset (the two-pass Var
    must not cancel), zero rows and rows with one spike."""
    cfg = _cfg("qwen3-8b", dtype=dtype)
    x = synth.make_round_inputs(cfg, DEV, seed=5, n_inst=3)
    v = x["v"]
    v[0, 0:40] = 1.5
    v[0, 40:80] = -0.0
    v[0, 80:120] = 0.0
    v[1, :200] = 96.0 + (v[1, :200].float() * 0.25).to(v.dtype)
    v[2, :64] = 0.0
    v[2, :64, 7] = -3.0e4
    for kind in ("l2", "var", "range"):
        kd = KINDS[kind]
        _, val = vase.score(x["k"], v, x["q_win"], cfg.K, cfg.B, cfg.pool, value_kind=kd)
        torch.cuda.synchronize()
        v_h = v.cpu()
        ref = oracle.value_score(v_h, cfg.K, kd)
        _assert_value_close(val.cpu().numpy(), v_h[:, :cfg.K].double().numpy(), ref, kd)
        g = val.cpu().numpy()
        if kd != vase.VALUE_L2:
            assert np.all(g[0, 0:120] == 0.0), kind
        assert np.all(g[2, :64] > 0)


@pytest.mark.parametrize("n_inst,K,seed,rnd,base", [
    (3, 256, 0, 0, 0),
    (5, 1001, 7, 3, 100),                      # K not a multiple of 4
    (2, 4097, 2**64 - 1, 2**32 - 1, 2**32 - 2),  # extreme seed, round and instance ids
    (40, 2048, 12345, 17, 7),
])
def test_value_random_bitexact(n_inst, K, seed, rnd, base):
    cfg = _cfg("tiny", K=K, B=16)
    x = synth.make_round_inputs(cfg, DEV, seed=1, n_inst=n_inst)
    attn0, _ = vase.score(x["k"], x["v"], x["q_win"], K, cfg.B, cfg.pool)
    attn, val = vase.score(x["k"], x["v"], x["q_win"], K, cfg.B, cfg.pool,
                           value_kind=vase.VALUE_RANDOM, seed=seed, round=rnd, inst_base=base)
    torch.cuda.synchronize()
    assert torch.equal(attn, attn0)
    ref = oracle.value_score(None, K, oracle.VALUE_RANDOM, seed, rnd, base, n_inst)
    np.testing.assert_array_equal(val.cpu().numpy(), ref)
    u = val.cpu().numpy()
    assert np.all((u > 0) & (u < 1))


def test_value_random_bf16_fused_path():
    """The bf16 MFMA kernel skips the value rows under random reservation: its
    attention score must not change, on the path that pools in-kernel too."""
    cfg = _cfg("qwen3-8b")
    n = 512
    x = synth.make_round_inputs(cfg, DEV, seed=3, n_inst=n)
    attn0, _ = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool)
    attn, val = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool,
                           value_kind=vase.VALUE_RANDOM, seed=99, round=4)
    torch.cuda.synchronize()
    assert torch.equal(attn, attn0)
    ref = oracle.value_score(None, cfg.K, oracle.VALUE_RANDOM, 99, 4, 0, n)
    np.testing.assert_array_equal(val.cpu().numpy(), ref)


@pytest.mark.parametrize("kind", ["l2", "var", "random"])
def test_round_with_value_variant(kind):
    cfg = _cfg("qwen3-1.7b")
    n = 24
    kd = vase.VALUE_RANDOM if kind == "random" else KINDS[kind]
    seed, rnd = 77, 5
    x = synth.make_round_inputs(cfg, DEV, seed=4, n_inst=n)
    q_h, k_h = x["q_win"].cpu(), x["k"].cpu()
    rb = vase.Round(n, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w, cfg.torch_dtype, DEV)
    rb.run(x["k"], x["v"], x["q_win"], x["q_dec"], cfg.Nv, cfg.pool, seed=seed, rnd=rnd,
           value_kind=kd)
    torch.cuda.synchronize()
    val = rb.vrange.cpu().numpy()
    src = rb.src.cpu().numpy()
    survivor_check(src, cfg.K, cfg.B, val, cfg.Nv)
    ref_attn = oracle.score(q_h, k_h, cfg.K, cfg.pool)
    assert_attn_close(rb.attn.cpu().numpy(), ref_attn)
    if kd == vase.VALUE_RANDOM:
        np.testing.assert_array_equal(val, oracle.value_score(None, cfg.K, kd, seed, rnd, 0, n))
    ref_src, ref_keys = oracle.select(ref_attn, val, cfg.K, cfg.B, cfg.Nv, seed, rnd,
                                      return_keys=True)
    a_g = rb.attn.cpu().numpy()
    st = explained_swaps(src, ref_src, ref_keys, cfg.K, a_g, ref_attn,
                         src_from_gpu=oracle.select(a_g, val, cfg.K, cfg.B, cfg.Nv, seed, rnd))
    rep = swap_report("value variant %s" % kind, [st], 1, n * cfg.B)
    assert rep["swaps"] <= max(1, rep["evictions"] // 1000)


# --------------------------------------------------------------------------
# value scores carried from one round's compaction to the next round
# --------------------------------------------------------------------------
@pytest.mark.parametrize("kind", ["range", "l2", "var"])
@pytest.mark.parametrize("name,kw,n_inst", [
    ("qwen3-8b", {}, 512),                       # the fused compaction + decode kernel
    ("qwen3-8b", {}, 12),                        # compaction split over workgroups, then decode
    ("tiny", {}, None),                          # fp32
    ("qwen3-1.7b", dict(d=64), 600),             # d = 64, fused
])
def test_compaction_carries_value_scores(name, kw, n_inst, kind):
    cfg = _cfg(name, **kw)
    kd = KINDS[kind]
    x = synth.make_round_inputs(cfg, DEV, seed=91, n_inst=n_inst)
    attn, vr = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool)
    src = vase.select(attn, vr, cfg.K, cfg.B, cfg.Nv, 5, 1)
    carried = torch.full_like(vr, float("nan"))
    vase.compact_decode(x["k"], x["v"], src, x["q_dec"], cfg.K, cfg.B, vrange_out=carried,
                        value_kind=kd)
    torch.cuda.synchronize()
    # the same arithmetic as the score kernel's on the compacted rows, bit for bit
    _, fresh = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, value_kind=kd)
    torch.cuda.synchronize()
    assert torch.equal(carried, fresh)
    sel = slice(None) if x["v"].shape[0] <= 16 else [0, x["v"].shape[0] - 1]
    v_h = x["v"][sel].cpu()
    ref = oracle.value_score(v_h, cfg.K, kd)
    _assert_value_close(carried[sel].cpu().numpy(), v_h[:, :cfg.K].double().numpy(), ref, kd)


@pytest.mark.parametrize("one_pass", [False, True])
def test_score_skip_leaves_value_scores(one_pass):
    """SKIP changes no window score (two-pass, and one-pass with supplied normalisers)
    and leaves the caller's value scores untouched."""
    cfg = _cfg("qwen3-8b")
    x = synth.make_round_inputs(cfg, DEV, seed=92, n_inst=512)
    lse = None
    if one_pass:
        g = torch.Generator(device="cpu").manual_seed(5)
        lse = (torch.randn((512, cfg.G, cfg.w), generator=g) + 6.0).to(DEV)
    attn0, _ = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, lse_win=lse)
    sentinel = torch.full((512, cfg.K), 7.25, dtype=torch.float32, device=DEV)
    attn, vr = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, vrange=sentinel,
                          value_kind=vase.VALUE_SKIP, lse_win=lse)
    attn2, _ = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool,
                          value_kind=vase.VALUE_SKIP, lse_win=lse)   # no value buffer at all
    torch.cuda.synchronize()
    assert torch.equal(attn, attn0) and torch.equal(attn2, attn0)
    assert torch.all(vr == 7.25)


@pytest.mark.parametrize("name,n_inst,kind", [
    ("qwen3-1.7b", None, vase.VALUE_RANGE),      # 8 instances: split compaction path
    ("qwen3-8b", 512, vase.VALUE_RANGE),         # fused path
    ("qwen3-8b", 512, vase.VALUE_VAR),
])
def test_rounds_with_carried_scores_match(name, n_inst, kind):
    """Consecutive rounds with the value scores carried by the compaction select,
    move and decode exactly what rounds that recompute them do."""
    cfg = _cfg(name)
    a = synth.make_round_inputs(cfg, DEV, seed=93, n_inst=n_inst)
    b = {k_: t.clone() for k_, t in a.items()}
    n = a["k"].shape[0]
    ra = vase.Round(n, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w, cfg.torch_dtype, DEV)
    rb = vase.Round(n, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w, cfg.torch_dtype, DEV)
    for rnd in range(4):
        oa = ra.run(a["k"], a["v"], a["q_win"], a["q_dec"], cfg.Nv, cfg.pool, seed=3, rnd=rnd,
                    value_kind=kind, carry=True)
        ob = rb.run(b["k"], b["v"], b["q_win"], b["q_dec"], cfg.Nv, cfg.pool, seed=3, rnd=rnd,
                    value_kind=kind)
        torch.cuda.synchronize()
        assert torch.equal(ra.src, rb.src), rnd
        assert torch.equal(oa, ob) and torch.equal(a["k"], b["k"]) and torch.equal(a["v"], b["v"])
        synth.refresh_buffer(a, cfg, step_seed=rnd)
        synth.refresh_buffer(b, cfg, step_seed=rnd)
    assert ra.carried_kind == kind
