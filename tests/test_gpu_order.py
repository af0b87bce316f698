"""GPU parity of the round under an order map (the C ABI against the CPU oracle).

With an order map ord (ord[t] = slot of temporal rank t) the cache X stands for
the temporal cache T[t] = X[ord[t]].  Every output of the map calls must equal
what the oracle computes on T with the stable layout:
  O1 scores: with the identity map, bit-identical to vase_score_ex (the same
     kernels, pooled in the same order); with any map, within 1e-4 of the
     oracle on T, value scores bit-exact;
  O2 order_scores: the box filter over temporal ranks, bit-exact against the
     same fp32 additions done on the host;
  O3 compaction: the new map equals the oracle's order compaction, the cache
     bytes equal the oracle's moves applied to X (survivors untouched), so the
     map view is the stable compaction of T; decode within the bf16 tolerance;
     carried value scores bit-exact by rank;
  O4 whole rounds end to end (tiny, Qwen3-1.7B shape; carried value scores on
     and off), against the oracle on the map view;
  O5 the full Qwen3-8B-shaped workload in the benchmark's launch configuration,
     two rounds (the second on a scrambled map), sampled against the oracle;
  O6 decode logits left by the score pass: within fp32 accumulation error of
     q.k in float64, the scores unchanged bit for bit, and the compaction's
     decode from them bit-identical to the one that reads K.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_03928_amd import synth, vase

from parity_util import (assert_attn_close, assert_decode_close, explained_swaps, from_raw, raw,
                         swap_report,
                         survivor_check)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


@pytest.fixture(autouse=True)
def _lib(gpu_lib):
    yield
    torch.cuda.synchronize()


def _cfg(name, **kw):
    return synth.CONFIGS[name].with_(**kw) if kw else synth.CONFIGS[name]


def _random_order(n, K, seed):
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return torch.stack([torch.randperm(K, generator=g) for _ in range(n)]).to(torch.int32)


def _scatter(t, ord_map, K):
    """The physical cache X with X[ord[r]] = t[r] for ranks r < K (buffer unchanged)."""
    x = t.clone()
    idx = ord_map.to(t.device).long()[:, :, None].expand(-1, -1, t.shape[2])
    x[:, :K] = x[:, :K].scatter(1, idx, t[:, :K])
    return x


def _temporal(x, ord_map, K):
    idx = ord_map.to(x.device).long()[:, :, None].expand(-1, -1, x.shape[2])
    return torch.cat([torch.gather(x[:, :K], 1, idx), x[:, K:]], dim=1)


def _valid_src(n, K, B, seed):
    rng = np.random.default_rng(seed)
    rows = []
    for i in range(n):
        keep = np.sort(rng.choice(K, K - B, replace=False))
        rows.append(np.concatenate([keep, np.arange(K, K + B)]))
    return np.stack(rows).astype(np.int32)


# --------------------------------------------------------------------------
# O1: scores under the map
# --------------------------------------------------------------------------
SCORE_CASES = [
    # name, overrides, instances (covering every score-kernel path)
    ("tiny", {}, None),                                   # fp32 VALU path
    ("qwen3-1.7b", {}, None),                             # split slot ranges
    ("qwen3-8b", {}, 512),                                # one workgroup per instance, in-kernel pool
    ("qwen3-14b", {}, 4),                                 # row slabs + split ranges
    ("qwen3-14b", {}, 600),                               # row slabs, one range: pool kernel
    ("qwen3-8b", dict(K=1000, B=24, w=40, d=64), 520),    # ragged, d = 64
]
KINDS = [vase.VALUE_RANGE, vase.VALUE_L2, vase.VALUE_VAR, vase.VALUE_RANDOM]


@pytest.mark.parametrize("name,kw,n_inst", SCORE_CASES)
def test_identity_map_scores_are_bitwise(name, kw, n_inst):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=31, n_inst=n_inst)
    n = x["k"].shape[0]
    ident = vase.identity_order(n, cfg.K, DEV)
    for kind in KINDS:
        a1, v1 = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, value_kind=kind,
                            seed=5, round=3)
        a2, v2 = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, value_kind=kind,
                            seed=5, round=3, ord=ident)
        torch.cuda.synchronize()
        assert torch.equal(a1, a2), kind
        assert torch.equal(v1, v2), kind


@pytest.mark.parametrize("name,kw,n_inst", SCORE_CASES)
def test_permuted_map_scores_match_oracle(name, kw, n_inst):
    cfg = _cfg(name, **kw)
    t = synth.make_round_inputs(cfg, DEV, seed=32, n_inst=n_inst)
    n = t["k"].shape[0]
    ord_map = _random_order(n, cfg.K, seed=n).to(DEV)
    xk, xv = _scatter(t["k"], ord_map, cfg.K), _scatter(t["v"], ord_map, cfg.K)
    attn, vr = vase.score(xk, xv, t["q_win"], cfg.K, cfg.B, cfg.pool, ord=ord_map)
    a_ref, v_ref = vase.score(t["k"], t["v"], t["q_win"], cfg.K, cfg.B, cfg.pool)
    torch.cuda.synchronize()
    sample = list(range(n)) if n <= 16 else [0, 1, n // 2, n - 1]
    ref = oracle.score(t["q_win"][sample].cpu(), t["k"][sample].cpu(), cfg.K, cfg.pool)
    rel = assert_attn_close(attn[sample].cpu().numpy(), ref)
    np.testing.assert_array_equal(vr[sample].cpu().numpy(),
                                  oracle.vrange(t["v"][sample].cpu(), cfg.K))
    # the stable-layout score of T and the map score of X differ only by the
    # summation order of the row normalisers
    assert_attn_close(attn.cpu().numpy(), a_ref.cpu().numpy().astype(np.float64), what="map vs stable")
    assert torch.equal(vr, v_ref)
    print("%s: max relative score error under a random map %.3g" % (name, rel))


def test_permuted_map_one_pass_score():
    """The one-pass score (supplied persistent LSE) under a map: the persistent part
    of each row's normaliser does not depend on the slot order."""
    cfg = _cfg("qwen3-8b")
    t = synth.make_round_inputs(cfg, DEV, seed=33, n_inst=512)
    n = 512
    ord_map = _random_order(n, cfg.K, seed=4).to(DEV)
    xk, xv = _scatter(t["k"], ord_map, cfg.K), _scatter(t["v"], ord_map, cfg.K)
    sample = [0, 255, 511]
    # the persistent part of each window row's normaliser, in float64 on the device
    lse = torch.empty((n, cfg.G, cfg.w), dtype=torch.float32, device=DEV)
    for s0 in range(0, n, 64):
        qq = t["q_win"][s0:s0 + 64].double().reshape(-1, cfg.G * cfg.w, cfg.d)
        kk = t["k"][s0:s0 + 64, :cfg.K].double().transpose(1, 2).contiguous()
        sc = torch.matmul(qq, kk) / cfg.d ** 0.5
        lse[s0:s0 + 64] = torch.logsumexp(sc, dim=2).reshape(-1, cfg.G, cfg.w).float()
        del qq, kk, sc
    attn, _ = vase.score(xk, xv, t["q_win"], cfg.K, cfg.B, cfg.pool, ord=ord_map, lse_win=lse)
    torch.cuda.synchronize()
    ref = oracle.score(t["q_win"][sample].cpu(), t["k"][sample].cpu(), cfg.K, cfg.pool)
    assert_attn_close(attn[sample].cpu().numpy(), ref)


# --------------------------------------------------------------------------
# O2: the reordering step alone
# --------------------------------------------------------------------------
@pytest.mark.parametrize("K,pool,n", [(128, 7, 3), (1000, 1, 2), (4096, 31, 2), (37, 255, 2)])
def test_order_scores_definition(K, pool, n):
    g = torch.Generator(device="cpu")
    g.manual_seed(K + pool)
    phys = torch.rand((n, K), generator=g, dtype=torch.float32)
    vphys = torch.rand((n, K), generator=g, dtype=torch.float32)
    ord_map = _random_order(n, K, seed=K)
    attn, vr = vase.order_scores(phys.to(DEV), ord_map.to(DEV), pool, vrange_phys=vphys.to(DEV))
    torch.cuda.synchronize()
    # host: the same fp32 additions in rank order, then the division by P
    p, o = phys.numpy(), ord_map.numpy()
    h = pool // 2
    want = np.zeros((n, K), np.float32)
    for i in range(n):
        seq = p[i, o[i]]
        for t_ in range(K):
            s = np.float32(0.0)
            for u in range(t_ - h, t_ + h + 1):
                s = np.float32(s + (seq[u] if 0 <= u < K else np.float32(0.0)))
            want[i, t_] = np.float32(s / np.float32(pool))
    np.testing.assert_array_equal(attn.cpu().numpy(), want)
    np.testing.assert_array_equal(vr.cpu().numpy(), np.take_along_axis(vphys.numpy(), o, axis=1))


# --------------------------------------------------------------------------
# O3: compaction (+ decode) under the map
# --------------------------------------------------------------------------
COMPACT_CASES = [
    # name, overrides, instances, map ("identity" or "random"), sampled instances
    ("tiny", {}, None, "random", None),
    ("tiny", dict(dtype="bf16", d=64), 5, "identity", None),
    ("qwen3-1.7b", {}, None, "random", None),
    ("qwen3-8b", {}, 1024, "random", [0, 1, 513, 1023]),
    ("qwen3-8b", dict(dtype="f32"), 64, "random", [0, 63]),
    ("qwen3-14b", dict(d=64), 70, "random", [0, 69]),            # G = 5, B = 256
    ("qwen3-32b", {}, 40, "random", [0, 39]),                     # G = 8, K = 8192
    ("qwen3-8b", dict(K=1000, B=500), 9, "random", None),        # half the candidates evicted
    ("qwen3-8b", dict(K=130, B=130), 4, "random", None),         # every candidate evicted
]


@pytest.mark.parametrize("carry", [False, True, "gather"])
@pytest.mark.parametrize("name,kw,n_inst,maps,sample", COMPACT_CASES)
def test_compact_decode_map_parity(name, kw, n_inst, maps, sample, carry):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=34, n_inst=n_inst)
    n = x["k"].shape[0]
    sample = list(range(n)) if sample is None else sample
    K, B = cfg.K, cfg.B
    ord_map = (vase.identity_order(n, K, DEV) if maps == "identity"
               else _random_order(n, K, seed=n + 9).to(DEV))
    src = _valid_src(n, K, B, seed=n)
    ord0 = ord_map.cpu().numpy()
    k0, v0 = raw(x["k"][sample].cpu()), raw(x["v"][sample].cpu())
    vr = torch.full((n, K), -1.0, dtype=torch.float32, device=DEV) if carry else None
    vin = None
    if carry == "gather":
        # the current candidates' Range by temporal rank, as the selection saw it,
        # in the output buffer itself (the survivors' scores are gathered in place)
        vr.copy_(torch.from_numpy(oracle.vrange(_temporal(x["v"].cpu(), ord_map.cpu(), K), K)))
        vin = vr
    out = vase.compact_decode_map(x["k"], x["v"], torch.from_numpy(src).to(DEV), ord_map, K, B,
                                  q=x["q_dec"], vrange_out=vr, vrange_in=vin)
    torch.cuda.synchronize()
    o_new, moves = oracle.order_compact(ord0, src, B)
    np.testing.assert_array_equal(ord_map.cpu().numpy(), o_new)
    oracle.apply_moves(k0, v0, moves[sample], K)
    np.testing.assert_array_equal(raw(x["k"][sample].cpu()), k0)   # buffer rows untouched too
    np.testing.assert_array_equal(raw(x["v"][sample].cpu()), v0)
    kt = _temporal(from_raw(k0, cfg.torch_dtype), torch.from_numpy(o_new[sample]), K)
    vt = _temporal(from_raw(v0, cfg.torch_dtype), torch.from_numpy(o_new[sample]), K)
    ref = oracle.decode(x["q_dec"][sample].cpu(), kt, vt, K)
    err = assert_decode_close(out[sample].float().cpu().numpy(), ref, bf16=cfg.dtype == "bf16")
    if carry:
        np.testing.assert_array_equal(vr[sample].cpu().numpy(), oracle.vrange(vt, K))
    print("%s n=%d: max abs decode error %.3g" % (name, n, err))


@pytest.mark.parametrize("carry", [False, True, "gather"])
@pytest.mark.parametrize("name,kw,n_inst", [
    ("qwen3-8b", {}, 300),
    ("tiny", {}, None),                                   # fp32, d = 64
    ("qwen3-14b", dict(d=64), 40),                       # B = 256
    ("qwen3-8b", dict(dtype="f32", K=1000, B=500), 9),    # half the candidates evicted
    ("qwen3-8b", dict(K=33, B=32, Nv=1), 5),              # one survivor
    ("tiny", dict(K=1, B=1, w=1, Nv=0), None),            # every candidate evicted, K = 1
])
def test_compact_map_without_decode(name, kw, n_inst, carry):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=35, n_inst=n_inst)
    n, K, B = x["k"].shape[0], cfg.K, cfg.B
    ord_map = _random_order(n, K, seed=1).to(DEV)
    src = _valid_src(n, K, B, seed=2)
    ord0 = ord_map.cpu().numpy()
    k0, v0 = raw(x["k"].cpu()), raw(x["v"].cpu())
    vr = torch.full((n, K), -1.0, dtype=torch.float32, device=DEV) if carry else None
    vin = None
    if carry == "gather":
        # the candidates' Range by temporal rank in the output buffer itself
        vr.copy_(torch.from_numpy(oracle.vrange(_temporal(x["v"].cpu(), ord_map.cpu(), K), K)))
        vin = vr
    assert vase.compact_decode_map(x["k"], x["v"], torch.from_numpy(src).to(DEV), ord_map, K, B,
                                   vrange_out=vr, vrange_in=vin) is None
    torch.cuda.synchronize()
    o_new, moves = oracle.order_compact(ord0, src, B)
    np.testing.assert_array_equal(ord_map.cpu().numpy(), o_new)
    oracle.apply_moves(k0, v0, moves, K)
    np.testing.assert_array_equal(raw(x["k"].cpu()), k0)
    np.testing.assert_array_equal(raw(x["v"].cpu()), v0)
    if carry:
        vt = _temporal(from_raw(v0, cfg.torch_dtype), torch.from_numpy(o_new), K)
        np.testing.assert_array_equal(vr.cpu().numpy(), oracle.vrange(vt, K))


@pytest.mark.parametrize("kind", ["range", "l2", "var"])
@pytest.mark.parametrize("gather", [False, True])
@pytest.mark.parametrize("name,kw,n_inst", [("qwen3-8b", {}, 64), ("tiny", {}, None)])
def test_compact_map_alone_value_kinds(name, kw, n_inst, kind, gather):
    # the compaction alone leaves the value scores a fresh score of the compacted
    # cache would give, bit for bit, for every kind: survivors' gathered by rank
    # (gather) or read from their rows, the moved rows' from the copy
    cfg = _cfg(name, **kw)
    kd = {"range": vase.VALUE_RANGE, "l2": vase.VALUE_L2, "var": vase.VALUE_VAR}[kind]
    x = synth.make_round_inputs(cfg, DEV, seed=36, n_inst=n_inst)
    n, K, B = x["k"].shape[0], cfg.K, cfg.B
    ord_map = _random_order(n, K, seed=3).to(DEV)
    attn, vr = vase.score(x["k"], x["v"], x["q_win"], K, B, cfg.pool, value_kind=kd, ord=ord_map)
    src = vase.select(attn, vr, K, B, cfg.Nv, 5, 1)
    out = vr if gather else torch.full_like(vr, float("nan"))
    vase.compact_decode_map(x["k"], x["v"], src, ord_map, K, B, vrange_out=out,
                            vrange_in=vr if gather else None, value_kind=kd)
    torch.cuda.synchronize()
    _, fresh = vase.score(x["k"], x["v"], x["q_win"], K, B, cfg.pool, value_kind=kd, ord=ord_map)
    torch.cuda.synchronize()
    assert torch.equal(out, fresh)


# --------------------------------------------------------------------------
# O4: rounds end to end under the map
# --------------------------------------------------------------------------
@pytest.mark.parametrize("name,n_inst,rounds,check_every,carry,decode", [
    ("tiny", None, 6, 1, False, True),
    ("tiny", None, 6, 1, True, True),
    ("qwen3-1.7b", None, 40, 8, True, True),
    ("qwen3-8b", 64, 5, 2, True, True),
    # the round alone: compaction without a decode step, value scores carried
    ("tiny", None, 6, 1, True, False),
    ("qwen3-8b", 64, 5, 2, True, False),
])
def test_map_rounds_end_to_end(name, n_inst, rounds, check_every, carry, decode):
    cfg = _cfg(name)
    seed = 77
    x = synth.make_round_inputs(cfg, DEV, seed=3, n_inst=n_inst)
    n = x["k"].shape[0]
    rb = vase.Round(n, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w, cfg.torch_dtype, DEV, layout="map")
    swaps_all = []
    for rnd in range(rounds):
        check = rnd % check_every == 0 or rnd == rounds - 1
        if check:
            kt_h = rb.temporal(x["k"]).cpu()
            vt_h = rb.temporal(x["v"]).cpu()
            q_h = x["q_win"].cpu()
        out = rb.run(x["k"], x["v"], x["q_win"], x["q_dec"] if decode else None, cfg.Nv, cfg.pool,
                     seed=seed, rnd=rnd, carry=carry)
        torch.cuda.synchronize()
        assert (out is None) == (not decode)
        src_g = rb.src.cpu().numpy()
        if check:
            ref_attn = oracle.score(q_h, kt_h, cfg.K, cfg.pool)
            assert_attn_close(rb.attn.cpu().numpy(), ref_attn)
            ref_vr = oracle.vrange(vt_h, cfg.K)
            ref_src, ref_keys = oracle.select(ref_attn, ref_vr, cfg.K, cfg.B, cfg.Nv, seed, rnd,
                                              return_keys=True)
            a_g = rb.attn.cpu().numpy()
            # the selection's value scores are Range of the candidates, bit-exact on the
            # GPU whether computed by the score or carried (checked below)
            swaps_all.append(explained_swaps(src_g, ref_src, ref_keys, cfg.K, a_g, ref_attn,
                                             src_from_gpu=oracle.select(a_g, ref_vr, cfg.K, cfg.B,
                                                                        cfg.Nv, seed, rnd)))
            survivor_check(src_g, cfg.K, cfg.B, ref_vr, cfg.Nv)
            # the map view after compaction is the stable compaction of T with the GPU's map
            kk, vv = raw(kt_h), raw(vt_h)
            oracle.compact(kk, vv, src_g)
            np.testing.assert_array_equal(raw(rb.temporal(x["k"]).cpu())[:, :cfg.K], kk[:, :cfg.K])
            np.testing.assert_array_equal(raw(rb.temporal(x["v"]).cpu())[:, :cfg.K], vv[:, :cfg.K])
            if decode:
                ref_out = oracle.decode(x["q_dec"].cpu(), from_raw(kk, cfg.torch_dtype),
                                        from_raw(vv, cfg.torch_dtype), cfg.K)
                assert_decode_close(out.float().cpu().numpy(), ref_out, bf16=cfg.dtype == "bf16")
            if carry:
                np.testing.assert_array_equal(rb.vrange.cpu().numpy(),
                                              oracle.vrange(from_raw(vv, cfg.torch_dtype), cfg.K))
        synth.refresh_buffer(x, cfg, step_seed=rnd)
    # the map really scrambles the slots after a few rounds
    assert not torch.equal(rb.ord, vase.identity_order(n, cfg.K, DEV))
    rep = swap_report("%s under the map" % name, swaps_all, len(swaps_all),
                      len(swaps_all) * n * cfg.B)
    assert rep["swaps"] <= max(1, rep["evictions"] // 1000)


# --------------------------------------------------------------------------
# O5: the full Qwen3-8B-shaped workload, benchmark launch configuration
# --------------------------------------------------------------------------
def test_full_8b_map_rounds_sampled():
    cfg = _cfg("qwen3-8b")
    x = synth.make_round_inputs(cfg, DEV, seed=0)
    n = cfg.n_inst
    sample = [0, 1, 777, 1500, n - 2, n - 1]
    rb = vase.Round(n, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w, cfg.torch_dtype, DEV, layout="map")
    rb.run(x["k"], x["v"], x["q_win"], x["q_dec"], cfg.Nv, cfg.pool, seed=0, rnd=0, carry=True)
    synth.refresh_buffer(x, cfg, step_seed=0)
    # second round: a scrambled map, carried value scores, the one-call launch shape
    kt_s = rb.temporal(x["k"])[sample].cpu()
    vt_s = rb.temporal(x["v"])[sample].cpu()
    ord_before = rb.ord.clone()
    out = rb.run(x["k"], x["v"], x["q_win"], x["q_dec"], cfg.Nv, cfg.pool, seed=0, rnd=1,
                 carry=True)
    torch.cuda.synchronize()
    assert not torch.equal(ord_before, vase.identity_order(n, cfg.K, DEV))
    src = rb.src.long()
    assert torch.all(src[:, 1:] > src[:, :-1])
    assert torch.all(src[:, cfg.K - cfg.B:] == torch.arange(cfg.K, cfg.N, device=DEV))
    # every map is a permutation of the K slots
    assert torch.equal(torch.sort(rb.ord, dim=1).values, vase.identity_order(n, cfg.K, DEV))
    ref_attn = oracle.score(x["q_win"][sample].cpu(), kt_s, cfg.K, cfg.pool)
    assert_attn_close(rb.attn[sample].cpu().numpy(), ref_attn)
    ref_vr = oracle.vrange(vt_s, cfg.K)
    a_s = rb.attn[sample].cpu().numpy()
    ref_src = np.stack([oracle.select(a_s[j:j + 1], ref_vr[j:j + 1], cfg.K, cfg.B, cfg.Nv, 0, 1,
                                      inst_base=i)[0] for j, i in enumerate(sample)])
    np.testing.assert_array_equal(rb.src[sample].cpu().numpy(), ref_src)
    kk, vv = raw(kt_s), raw(vt_s)
    oracle.compact(kk, vv, ref_src)
    np.testing.assert_array_equal(raw(rb.temporal(x["k"])[sample].cpu())[:, :cfg.K], kk[:, :cfg.K])
    np.testing.assert_array_equal(raw(rb.temporal(x["v"])[sample].cpu())[:, :cfg.K], vv[:, :cfg.K])
    ref_out = oracle.decode(x["q_dec"][sample].cpu(), from_raw(kk, torch.bfloat16),
                            from_raw(vv, torch.bfloat16), cfg.K)
    assert_decode_close(out[sample].float().cpu().numpy(), ref_out, bf16=True)


# --------------------------------------------------------------------------
# O6: decode logits from the score pass
# --------------------------------------------------------------------------
DL_CASES = [
    # name, overrides, instances (bf16; every score-kernel path)
    ("qwen3-1.7b", {}, None),                             # split slot ranges, 4 waves
    ("qwen3-8b", {}, 512),                                # one workgroup per instance
    ("qwen3-14b", {}, 4),                                 # row slabs + split ranges, G = 5
    ("qwen3-14b", {}, 600),                               # row slabs, one range
    ("qwen3-32b", {}, 6),                                 # G = 8
    ("qwen3-8b", dict(K=1000, B=24, w=40, d=64), 520),    # ragged, d = 64
    ("qwen3-8b", dict(K=999, B=22, w=8), 3),              # N odd, a partial last chunk
]


def _dl_scores(cfg, x, ord_map):
    n, N = x["k"].shape[0], cfg.K + cfg.B
    dl = torch.full((n, cfg.G, N), float("nan"), dtype=torch.float32, device=DEV)
    a, v = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, ord=ord_map,
                      q_dec=x["q_dec"], dec_logits=dl)
    return a, v, dl


@pytest.mark.parametrize("name,kw,n_inst", DL_CASES)
def test_score_decode_logits(name, kw, n_inst):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=36, n_inst=n_inst)
    n = x["k"].shape[0]
    ord_map = _random_order(n, cfg.K, seed=n + 3).to(DEV)
    a0, v0 = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool, ord=ord_map)
    a1, v1, dl = _dl_scores(cfg, x, ord_map)
    torch.cuda.synchronize()
    assert torch.equal(a0, a1) and torch.equal(v0, v1)
    sample = list(range(n)) if n <= 16 else [0, 1, n // 2, n - 1]
    q = x["q_dec"][sample].cpu().double()
    k = x["k"][sample].cpu().double()
    ref = torch.matmul(q, k.transpose(1, 2))                  # [s, G, N], exact products
    bound = torch.matmul(q.abs(), k.abs().transpose(1, 2))
    got = dl[sample].cpu().double()
    assert torch.isfinite(got).all()
    err = (got - ref).abs()
    # fp32 accumulation of d bf16 products: far below d * 2^-24 of sum |q_i k_i|
    assert (err <= 1e-5 * bound + 1e-30).all(), float((err / bound.clamp_min(1e-30)).max())
    print("%s: decode logits max error %.3g of sum |q k|" % (name, float((err / bound).max())))



@pytest.mark.parametrize("pattern", ["late_outlier", "row_spread"])
def test_exact_path_under_the_map_with_logits(pattern):
    # inputs that send pass 1 to its exact row maxima, in the headline launch
    # configuration (one workgroup per instance, pooling through the map, decode
    # logits): with the identity map the scores equal the plain score's bit for
    # bit, whose exact path is checked against the oracle, and the logits hold
    cfg = _cfg("qwen3-8b")
    n = 512
    x = synth.make_round_inputs(cfg, DEV, seed=13, n_inst=n)
    if pattern == "late_outlier":
        x["k"][:, 3000] *= 50.0
    else:
        x["q_win"][:, :, 1::2] *= 6.0
    a0, v0 = vase.score(x["k"], x["v"], x["q_win"], cfg.K, cfg.B, cfg.pool)
    a1, v1, dl = _dl_scores(cfg, x, vase.identity_order(n, cfg.K, DEV))
    torch.cuda.synchronize()
    assert torch.equal(a0, a1) and torch.equal(v0, v1)
    sample = [0, n - 1]
    q = x["q_dec"][sample].cpu().double()
    k = x["k"][sample].cpu().double()
    ref = torch.matmul(q, k.transpose(1, 2))
    bound = torch.matmul(q.abs(), k.abs().transpose(1, 2))
    err = (dl[sample].cpu().double() - ref).abs()
    assert (err <= 1e-5 * bound + 1e-30).all()

DL_COMPACT_CASES = [
    ("qwen3-1.7b", {}, None, [0, 7]),
    ("qwen3-8b", {}, 1024, [0, 1, 513, 1023]),
    ("qwen3-14b", dict(d=64), 70, [0, 69]),                      # G = 5, B = 256
    ("qwen3-8b", dict(K=1000, B=500), 9, None),                  # half the candidates evicted
    ("qwen3-8b", dict(K=130, B=130), 4, None),                   # every candidate evicted
    ("qwen3-8b", dict(K=999, B=22, w=8), 3, None),               # N odd
]


@pytest.mark.parametrize("carry", [False, "gather"])
@pytest.mark.parametrize("name,kw,n_inst,sample", DL_COMPACT_CASES)
def test_compact_decode_from_logits_is_bitwise(name, kw, n_inst, sample, carry):
    cfg = _cfg(name, **kw)
    x = synth.make_round_inputs(cfg, DEV, seed=37, n_inst=n_inst)
    n = x["k"].shape[0]
    sample = list(range(n)) if sample is None else sample
    K, B = cfg.K, cfg.B
    ord_map = _random_order(n, K, seed=n + 5).to(DEV)
    _, _, dl = _dl_scores(cfg, x, ord_map)
    src = torch.from_numpy(_valid_src(n, K, B, seed=n + 1)).to(DEV)
    res = []
    for use in (False, True):
        k, v, o = x["k"].clone(), x["v"].clone(), ord_map.clone()
        vr = vin = None
        if carry:
            vr = torch.from_numpy(oracle.vrange(_temporal(x["v"].cpu(), ord_map.cpu(), K), K)).to(DEV)
            vin = vr
        out = vase.compact_decode_map(k, v, src, o, K, B, q=x["q_dec"], vrange_out=vr,
                                      vrange_in=vin, dec_logits=dl if use else None)
        torch.cuda.synchronize()
        res.append((out, k, v, o, vr))
    (o0, k0, v0, m0, r0), (o1, k1, v1, m1, r1) = res
    assert np.array_equal(raw(o0), raw(o1))
    assert torch.equal(m0, m1) and np.array_equal(raw(k0), raw(k1)) and np.array_equal(raw(v0), raw(v1))
    if carry:
        assert torch.equal(r0, r1)
    # and against the oracle on the compacted map view
    kt = _temporal(k1[sample].cpu(), m1[sample].cpu(), K)
    vt = _temporal(v1[sample].cpu(), m1[sample].cpu(), K)
    ref = oracle.decode(x["q_dec"][sample].cpu(), kt, vt, K)
    err = assert_decode_close(o1[sample].float().cpu().numpy(), ref, bf16=True)
    print("%s n=%d: decode from the score's logits, max abs error %.3g" % (name, n, err))


def test_rounds_with_and_without_decode_logits_agree():
    """Whole rounds under the map: the decode logits path changes no output bit."""
    cfg = _cfg("qwen3-8b")
    x0 = synth.make_round_inputs(cfg, DEV, seed=38, n_inst=96)
    x1 = {k_: t.clone() for k_, t in x0.items()}
    n = 96
    rbs = [vase.Round(n, cfg.K, cfg.B, cfg.d, cfg.G, cfg.w, cfg.torch_dtype, DEV, layout="map",
                      dec_logits=use) for use in (False, True)]
    assert rbs[0].dec_logits is None and rbs[1].dec_logits is not None
    for rnd in range(4):
        outs = []
        for rb, x in zip(rbs, (x0, x1)):
            outs.append(rb.run(x["k"], x["v"], x["q_win"], x["q_dec"], cfg.Nv, cfg.pool, seed=9,
                               rnd=rnd, carry=True).clone())
            synth.refresh_buffer(x, cfg, step_seed=rnd)
        torch.cuda.synchronize()
        assert np.array_equal(raw(outs[0]), raw(outs[1])), rnd
        assert torch.equal(rbs[0].src, rbs[1].src) and torch.equal(rbs[0].ord, rbs[1].ord), rnd
        assert torch.equal(rbs[0].attn, rbs[1].attn) and torch.equal(rbs[0].vrange, rbs[1].vrange)
    assert np.array_equal(raw(x0["k"]), raw(x1["k"])) and np.array_equal(raw(x0["v"]), raw(x1["v"]))
