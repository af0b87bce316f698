"""Pins for the oracle's round steps (CPU only).

Each step is checked against something other than the oracle's own code:
closed forms worked by hand, library routines that compute the same
definition (torch's softmax and scaled-dot-product attention, avg_pool1d,
amax/amin, numpy's stable sort and fancy indexing), brute-force enumeration of
the sampling distribution on tiny inputs, and the invariants the paper's
periodic-eviction framework implies (Sec. 2: the cache returns to K slots, the
buffer is protected; Sec. 3.2: the reserved slots survive, every candidate with
positive weight has a positive retention probability).
"""
import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2606_03928_amd import synth


# --------------------------------------------------------------------------
# Step 1: scores
# --------------------------------------------------------------------------
def test_score_closed_form_two_slots():
    """One query, two slots: p0 = e / (e + 1) when s0 = 1 and s1 = 0."""
    d = 4
    q = np.zeros((1, 1, d)); q[0, 0, 0] = 2.0
    k = np.zeros((1, 2, d)); k[0, 0, 0] = 1.0           # s0 = 2*1/sqrt(4) = 1, s1 = 0
    attn, abar = oracle.score(q, k, K=1, pool=1, return_abar=True)
    assert abar[0, 0] == pytest.approx(math.e / (math.e + 1), rel=1e-15)
    assert abar[0, 1] == pytest.approx(1 / (math.e + 1), rel=1e-15)
    assert attn[0, 0] == np.float32(math.e / (math.e + 1))


def test_score_single_row_is_softmax():
    """G = w = 1, P = 1: the score is one softmax row over all N slots, cut to K."""
    g = torch.Generator().manual_seed(1)
    n_inst, N, K, d = 3, 40, 32, 64
    q = torch.randn(n_inst, 1, d, generator=g, dtype=torch.float64)
    k = torch.randn(n_inst, N, d, generator=g, dtype=torch.float64)
    attn, abar = oracle.score(q, k, K=K, pool=1, return_abar=True)
    ref = torch.softmax((q @ k.transpose(1, 2)).squeeze(1) / math.sqrt(d), dim=-1)
    np.testing.assert_allclose(abar, ref.numpy(), rtol=1e-12, atol=0)
    np.testing.assert_array_equal(attn, ref[:, :K].numpy().astype(np.float32))


@pytest.mark.parametrize("G,w,pool,sinks", [(2, 8, 7, 0), (4, 16, 5, 4), (3, 5, 1, 2)])
def test_score_matches_sdpa_mean_and_avgpool(G, w, pool, sinks):
    """Window mean of SDPA probabilities (V = identity), then avg_pool1d."""
    cfg = synth.CONFIGS["tiny"].with_(h_q=2 * G, w=w, pool=pool, sinks=sinks, K=48, B=16,
                                      dtype="f32")
    x = synth.make_round_inputs(cfg, "cpu", seed=5)
    attn, abar = oracle.score(x["q_win"], x["k"], K=cfg.K, pool=pool, return_abar=True)
    n, N, d = x["k"].shape
    q = x["q_win"].double().reshape(n, G * w, d)
    k = x["k"].double()
    eye = torch.eye(N, dtype=torch.float64).expand(n, N, N)
    p = F.scaled_dot_product_attention(q, k, eye)          # [n, R, N] probabilities
    ref_abar = p.mean(dim=1)
    np.testing.assert_allclose(abar, ref_abar.numpy(), rtol=1e-10, atol=1e-300)
    pooled = F.avg_pool1d(ref_abar[:, None, :cfg.K], kernel_size=pool, stride=1,
                          padding=pool // 2, count_include_pad=True)[:, 0, :]
    np.testing.assert_allclose(attn, pooled.numpy().astype(np.float32), rtol=1e-6, atol=1e-30)


def test_score_rows_sum_to_one():
    cfg = synth.CONFIGS["tiny"]
    x = synth.make_round_inputs(cfg, "cpu", seed=2)
    _, abar = oracle.score(x["q_win"], x["k"], K=cfg.K, pool=cfg.pool, return_abar=True)
    np.testing.assert_allclose(abar.sum(axis=1), 1.0, rtol=1e-12)


def test_score_pool_one_is_identity():
    cfg = synth.CONFIGS["tiny"]
    x = synth.make_round_inputs(cfg, "cpu", seed=3)
    attn, abar = oracle.score(x["q_win"], x["k"], K=cfg.K, pool=1, return_abar=True)
    np.testing.assert_array_equal(attn, abar[:, :cfg.K].astype(np.float32))


# --------------------------------------------------------------------------
# Step 2: Range
# --------------------------------------------------------------------------
def test_vrange_hand_values():
    v = np.zeros((1, 3, 4))
    v[0, 0] = [3.0, -1.0, 2.0, 0.5]      # 4
    v[0, 1] = [-2.5, -2.5, -2.5, -2.5]   # 0
    v[0, 2] = [1e-3, 7.0, -0.25, 0.0]    # 7.25
    out = oracle.vrange(v, K=2)
    assert out.tolist() == [[4.0, 0.0]]
    out = oracle.vrange(v, K=3)
    assert out[0, 2] == np.float32(7.25)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_vrange_matches_amax_minus_amin(dtype):
    cfg = synth.CONFIGS["tiny"].with_(dtype=dtype, out_p=0.1)
    x = synth.make_round_inputs(cfg, "cpu", seed=4)
    out = oracle.vrange(x["v"], K=cfg.K)
    vv = x["v"][:, :cfg.K].double()
    ref = (vv.amax(dim=-1) - vv.amin(dim=-1)).float().numpy()
    np.testing.assert_array_equal(out, ref)


# --------------------------------------------------------------------------
# Steps 3-6: selection
# --------------------------------------------------------------------------
def _survivor_sets(src, K, B):
    """Per instance: the set of candidate slots in [0, K) that survived."""
    out = []
    for row in src:
        assert np.all(np.diff(row) > 0), "src must be strictly increasing"
        s = set(int(x) for x in row if x < K)
        assert set(int(x) for x in row if x >= K) == set(range(K, K + B))
        out.append(s)
    return out


def _rand_scores(n, K, seed):
    rng = np.random.default_rng(seed)
    attn = rng.dirichlet(np.ones(K), size=n).astype(np.float32)
    vr = (rng.gamma(2.0, 1.0, size=(n, K)) * (1 + 40 * (rng.random((n, K)) < 0.03)))
    return attn, vr.astype(np.float32)


@pytest.mark.parametrize("K,B,Nv", [(128, 32, 8), (64, 8, 0), (40, 8, 32), (256, 64, 64)])
def test_select_budget_invariants(K, B, Nv):
    """|S| = K, buffer kept, exactly B evicted, all from C, reserved set kept."""
    n = 64
    attn, vr = _rand_scores(n, K, seed=K + B + Nv)
    src = oracle.select(attn, vr, K, B, Nv, seed=11, rnd=3)
    assert src.shape == (n, K)
    for i, s in enumerate(_survivor_sets(src, K, B)):
        assert len(s) == K - B
        order = np.argsort(-vr[i], kind="stable")
        assert set(order[:Nv].tolist()) <= s       # R_V survives
    # stability of the map: buffer tokens land at the end
    np.testing.assert_array_equal(src[:, K - B:], np.arange(K, K + B)[None, :].repeat(n, 0))


@pytest.mark.parametrize("Nv", [0, 6])
def test_select_deterministic_is_stable_topk(Nv):
    """Without noise, the fill is SnapKV's top-k (the ablation of Sec. 4.1 that drops the sampling)."""
    K, B, n = 64, 16, 32
    attn, vr = _rand_scores(n, K, seed=9)
    src = oracle.select(attn, vr, K, B, Nv, seed=0, rnd=0, flags=oracle.FLAG_DETERMINISTIC)
    for i in range(n):
        rv = np.argsort(-vr[i], kind="stable")[:Nv]
        cand = np.setdiff1d(np.arange(K), rv)
        order = cand[np.argsort(-attn[i][cand], kind="stable")]
        keep = np.sort(np.concatenate([rv, order[:K - Nv - B], np.arange(K, K + B)]))
        np.testing.assert_array_equal(src[i], keep)


def test_select_ties_prefer_lower_slot():
    K, B, Nv = 16, 4, 3
    vr = np.ones((1, K), np.float32)           # all tied: R_V = slots 0, 1, 2
    attn = np.full((1, K), 0.5, np.float32)    # all tied: evict the 4 highest slots of C
    src = oracle.select(attn, vr, K, B, Nv, 0, 0, flags=oracle.FLAG_DETERMINISTIC)
    np.testing.assert_array_equal(src[0], list(range(12)) + list(range(16, 20)))


def test_select_zero_weights_go_first():
    """Slots with weight 0 get key 0; survivors among them are taken by slot order."""
    K, B = 6, 2
    attn = np.array([[0.5, 0.0, 0.3, 0.0, 0.2, 0.0]], np.float32)
    vr = np.zeros((1, K), np.float32)
    for rnd in range(20):
        src = oracle.select(attn, vr, K, B, 0, seed=5, rnd=rnd)
        assert src[0].tolist() == [0, 1, 2, 4, 6, 7]


def _successive_sampling_probs(w, m):
    """P(T) for weighted sampling of m items without replacement, by enumeration."""
    w = np.asarray(w, dtype=np.float64)
    Z = w.sum()
    probs = {}
    for perm in itertools.permutations(range(len(w)), m):
        p, rem = 1.0, Z
        for j in perm:
            p *= w[j] / rem
            rem -= w[j]
        key = frozenset(perm)
        probs[key] = probs.get(key, 0.0) + p
    return probs


def _empirical(attn_row, vr_row, K, B, Nv, n, seed, rnd=0):
    attn = np.repeat(attn_row[None, :], n, 0).astype(np.float32)
    vr = np.repeat(vr_row[None, :], n, 0).astype(np.float32)
    src = oracle.select(attn, vr, K, B, Nv, seed=seed, rnd=rnd)
    return _survivor_sets(src, K, B)


@pytest.mark.parametrize("weights,B", [
    ([0.4, 0.25, 0.15, 0.1, 0.06, 0.04], 3),
    ([0.3, 0.3, 0.2, 0.1, 0.1], 2),
    ([0.7, 0.1, 0.1, 0.05, 0.05], 1),
])
def test_sampling_distribution_brute_force(weights, B):
    """Exponential-key selection has the successive-sampling law (G-test)."""
    from scipy import stats
    K = len(weights)
    m = K - B
    w = np.asarray(weights, np.float32)
    exact = _successive_sampling_probs(w.astype(np.float64), m)
    n = 1 << 17
    sets = _empirical(w, np.zeros(K, np.float32), K, B, 0, n, seed=1234)
    counts = {}
    for s in sets:
        counts[frozenset(s)] = counts.get(frozenset(s), 0) + 1
    keys = sorted(exact, key=lambda x: sorted(x))
    assert set(counts) <= set(keys)
    obs = np.array([counts.get(k_, 0) for k_ in keys], dtype=np.float64)
    exp = np.array([exact[k_] for k_ in keys]) * n
    assert abs(exp.sum() - n) < 1e-6 * n
    mask = exp >= 5
    obs_m = np.append(obs[mask], obs[~mask].sum())
    exp_m = np.append(exp[mask], exp[~mask].sum())
    if exp_m[-1] == 0:
        obs_m, exp_m = obs_m[:-1], exp_m[:-1]
    g, p = stats.power_divergence(obs_m, exp_m, lambda_="log-likelihood")
    assert p > 1e-4, (g, p)


def test_sampling_single_survivor_closed_form():
    """m = 1: the survivor is slot i with probability w_i / Z."""
    w = np.array([0.5, 0.3, 0.15, 0.05], np.float32)
    K, B = 4, 3
    n = 1 << 17
    sets = _empirical(w, np.zeros(K, np.float32), K, B, 0, n, seed=77)
    freq = np.zeros(K)
    for s in sets:
        (i,) = tuple(s)
        freq[i] += 1
    p = w.astype(np.float64) / w.sum()
    sd = np.sqrt(p * (1 - p) / n)
    assert np.all(np.abs(freq / n - p) < 5 * sd)


def test_sampling_with_reserved_slots():
    """R_V always survives; the rest is sampled from C = [K] \\ R_V only."""
    from scipy import stats
    K, B, Nv = 8, 3, 2
    w = np.array([0.2, 0.05, 0.1, 0.25, 0.1, 0.15, 0.05, 0.1], np.float32)
    vr = np.array([1, 9, 1, 1, 1, 1, 8, 1], np.float32)        # R_V = {1, 6}
    cand = [0, 2, 3, 4, 5, 7]
    m = K - Nv - B
    exact = _successive_sampling_probs(w[cand].astype(np.float64), m)
    n = 1 << 16
    sets = _empirical(w, vr, K, B, Nv, n, seed=99, rnd=5)
    counts = {}
    for s in sets:
        assert {1, 6} <= s
        c = frozenset(cand.index(i) for i in s - {1, 6})
        counts[c] = counts.get(c, 0) + 1
    keys = list(exact)
    obs = np.array([counts.get(k_, 0) for k_ in keys], dtype=np.float64)
    exp = np.array([exact[k_] for k_ in keys]) * n
    assert obs.sum() == n
    g, p = stats.power_divergence(obs, exp, lambda_="log-likelihood")
    assert p > 1e-4, (g, p)


def test_retention_lower_bound():
    """pi_i >= 1 - (1 - w_i / Z)^(K - |R|) for every candidate (Sec. 3.2)."""
    K, B = 12, 4
    m = K - B
    w = np.array([0.3, 0.2, 0.1, 0.1, 0.08, 0.06, 0.05, 0.04, 0.03, 0.02, 0.01, 0.01], np.float32)
    n = 1 << 15
    sets = _empirical(w, np.zeros(K, np.float32), K, B, 0, n, seed=3)
    pi = np.zeros(K)
    for s in sets:
        for i in s:
            pi[i] += 1
    pi /= n
    bound = 1 - (1 - w.astype(np.float64) / w.sum()) ** m
    assert np.all(pi > 0)
    assert np.all(pi >= bound - 5 * np.sqrt(bound * (1 - bound) / n) - 1e-12)


def test_select_rounds_and_instances_decorrelate():
    """Different (instance, round) counters give different samples."""
    K, B = 64, 16
    attn, vr = _rand_scores(1, K, seed=1)
    a = oracle.select(attn, vr, K, B, 4, seed=1, rnd=0)
    b = oracle.select(attn, vr, K, B, 4, seed=1, rnd=1)
    c = oracle.select(attn, vr, K, B, 4, seed=1, rnd=0, inst_base=1)
    d = oracle.select(attn, vr, K, B, 4, seed=2, rnd=0)
    assert not np.array_equal(a, b) and not np.array_equal(a, c) and not np.array_equal(a, d)
    np.testing.assert_array_equal(a, oracle.select(attn, vr, K, B, 4, seed=1, rnd=0))


def test_select_rejects_bad_budget():
    attn, vr = _rand_scores(1, 16, seed=0)
    with pytest.raises(RuntimeError):
        oracle.select(attn, vr, 16, 8, 9, seed=0, rnd=0)     # N_v + B > K


# --------------------------------------------------------------------------
# Step 7: compaction
# --------------------------------------------------------------------------
def _valid_src(rng, n, K, B):
    rows = []
    for _ in range(n):
        ev = rng.choice(K, size=B, replace=False)
        keep = np.setdiff1d(np.arange(K + B), ev)
        rows.append(keep)
    return np.stack(rows).astype(np.int32)


@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
def test_compact_matches_fancy_indexing(dtype):
    rng = np.random.default_rng(0)
    n, K, B, d = 5, 40, 8, 16
    k = rng.integers(0, 2 ** 15, size=(n, K + B, d)).astype(dtype)
    v = rng.integers(0, 2 ** 15, size=(n, K + B, d)).astype(dtype)
    srcs = _valid_src(rng, n, K, B)
    # adversarial maps: holes at the front, at the end, alternating
    srcs[0] = np.arange(B, K + B)
    srcs[1] = np.concatenate([np.arange(K - B), np.arange(K, K + B)])
    srcs[2] = np.setdiff1d(np.arange(K + B), np.arange(0, 2 * B, 2))
    ref_k = k[np.arange(n)[:, None], srcs]
    ref_v = v[np.arange(n)[:, None], srcs]
    kk, vv = k.copy(), v.copy()
    oracle.compact(kk, vv, srcs)
    np.testing.assert_array_equal(kk[:, :K], ref_k)
    np.testing.assert_array_equal(vv[:, :K], ref_v)


# --------------------------------------------------------------------------
# Step 8: decode attention
# --------------------------------------------------------------------------
@pytest.mark.parametrize("n_valid", [1, 37, 160])
def test_decode_matches_sdpa(n_valid):
    cfg = synth.CONFIGS["tiny"]
    x = synth.make_round_inputs(cfg, "cpu", seed=6)
    out = oracle.decode(x["q_dec"], x["k"], x["v"], n_valid)
    q = x["q_dec"].double()
    k = x["k"][:, :n_valid].double()
    v = x["v"][:, :n_valid].double()
    ref = F.scaled_dot_product_attention(q, k, v)
    np.testing.assert_allclose(out, ref.numpy(), rtol=1e-10, atol=1e-12)


def test_full_round_tiny_config():
    """The tiny workload end to end: budget holds, reserved outliers survive."""
    cfg = synth.CONFIGS["tiny"]
    x = synth.make_round_inputs(cfg, "cpu", seed=0)
    attn, vr, src = oracle.round_(x["q_win"], x["k"], x["v"], cfg.K, cfg.B, cfg.Nv, cfg.pool,
                                  seed=0, rnd=0)
    sets = _survivor_sets(src, cfg.K, cfg.B)
    for i, s in enumerate(sets):
        assert len(s) == cfg.K - cfg.B
        top = np.argsort(-vr[i], kind="stable")[:cfg.Nv]
        assert set(top.tolist()) <= s
    k = x["k"].numpy().copy()
    v = x["v"].numpy().copy()
    oracle.compact(k, v, src)
    np.testing.assert_array_equal(k[:, :cfg.K], x["k"].numpy()[np.arange(cfg.n_inst)[:, None], src])
