"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks one step of the oracle against something other than the
oracle's own formula: closed forms, brute force on tiny inputs, special cases
that reduce to a library routine or to a baseline method described in the
paper, and invariants the paper states.  A plausible slip in the oracle (a
dropped term, a wrong sign, a wrong index range, a transposed operand) fails at
least one of them.  No GPU is needed.
"""
import math

import numpy as np
import pytest
import torch

import workloads as W

S_ = dict(lambda_=0, rC=1, rE=2, DE=3, dmin=4, dmax=5, sdmin=6, sdmax=7, imp_mean=8, sbar_mean=9,
          mu_norm2=10, scale=11)


def f32(x):
    return np.ascontiguousarray(x, dtype=np.float32)


def rand_unit(seed, T, D, G=1, w=2, scale=1.0, offset=0.0):
    r = np.random.default_rng(seed)
    K = f32(r.standard_normal((T, D)) * scale + offset)
    Q = f32(r.standard_normal((G, w, D)))
    return K, Q


# --------------------------------------------------------------------------
# a1/a2: observation-window attention (Sec. 3 attention; Appendix A.1 SnapKV)
# --------------------------------------------------------------------------

def test_identical_keys_give_uniform_causal_attention(ora):
    # Every logit of a row is equal, so row j spreads its mass uniformly over
    # its P + j + 1 visible keys: a_i = mean_{g,j} 1 / (P + j + 1).
    T, D, G, w = 37, 16, 3, 4
    K = f32(np.tile(np.linspace(-1, 1, D), (T, 1)))
    Q = f32(np.random.default_rng(1).standard_normal((G, w, D)))
    r = ora.score_unit(K, Q, w, ora.Params(pool_kernel=1), trace=True)
    P = T - w
    expect = np.mean([1.0 / (P + j + 1) for j in range(w)])
    np.testing.assert_allclose(r["a"], expect, rtol=1e-13)
    # non-causal: every row sees all T keys
    r2 = ora.score_unit(K, Q, w, ora.Params(pool_kernel=1, causal=False), trace=True)
    np.testing.assert_allclose(r2["a"], 1.0 / T, rtol=1e-13)


def test_zero_queries_give_uniform_attention(ora):
    T, D, w = 20, 8, 3
    K, _ = rand_unit(2, T, D)
    Q = np.zeros((2, w, D), np.float32)
    r = ora.score_unit(K, Q, w, ora.Params(pool_kernel=1), trace=True)
    P = T - w
    np.testing.assert_allclose(r["a"], np.mean([1.0 / (P + j + 1) for j in range(w)]), rtol=1e-13)


def test_two_key_attention_is_a_sigmoid(ora):
    # T=2, w=1: the only non-window key gets sigmoid((q.k0 - q.k1)/sqrt(D)).
    K = f32([[1.0, 2.0], [0.5, -1.0]])
    Q = f32([[[0.75, 0.25]]])
    r = ora.score_unit(K, Q, 1, ora.Params(pool_kernel=1), trace=True)
    l0, l1 = (0.75 * 1 + 0.25 * 2) / math.sqrt(2), (0.75 * 0.5 - 0.25) / math.sqrt(2)
    assert r["a"][0] == pytest.approx(1 / (1 + math.exp(-(l0 - l1))), rel=1e-14)


def test_dominant_key_takes_all_attention(ora):
    T, D, w = 16, 8, 2
    K, _ = rand_unit(3, T, D, scale=0.01)
    K[5] = 0
    K[5, 0] = 40.0
    Q = np.zeros((1, w, D), np.float32)
    Q[0, :, 0] = 40.0
    r = ora.score_unit(f32(K), Q, w, ora.Params(pool_kernel=1), trace=True)
    assert r["a"][5] == pytest.approx(1.0, abs=1e-12)
    assert np.delete(r["a"], 5).max() < 1e-12


def test_attention_rows_are_distributions_and_key_shift_invariant(ora):
    # Adding one vector c to every key adds q.c to a whole row of logits: the
    # softmax and hence the importance must not move (normalisation per row).
    T, D, G, w = 50, 12, 2, 5
    K, Q = rand_unit(4, T, D, G, w)
    K = f32(np.round(K * 64) / 64)  # on a grid, so that the shift below is exact
    r = ora.score_unit(K, Q, w, ora.Params(pool_kernel=1), trace=True)
    np.testing.assert_allclose(r["rowmass"], 1.0, rtol=1e-13)
    c = f32(np.full(D, 0.5))  # exactly representable shift
    r2 = ora.score_unit(f32(K + c), Q, w, ora.Params(pool_kernel=1), trace=True)
    np.testing.assert_allclose(r2["a"], r["a"], rtol=1e-9)
    assert np.all(r["a"] > 0) and r["a"].sum() < 1.0


def test_grouped_query_heads_average(ora):
    # G query heads with identical rows give the importance of one head.
    T, D, w = 40, 8, 3
    K, Q1 = rand_unit(5, T, D, 1, w)
    Q3 = f32(np.repeat(Q1, 3, axis=0))
    a1 = ora.score_unit(K, Q1, w, trace=True)["a"]
    a3 = ora.score_unit(K, Q3, w, trace=True)["a"]
    np.testing.assert_allclose(a3, a1, rtol=1e-13)
    # and two different heads average their individual importances
    K, Q2 = rand_unit(6, T, D, 2, w)
    ab = ora.score_unit(K, Q2, w, trace=True)["a"]
    a_0 = ora.score_unit(K, Q2[:1], w, trace=True)["a"]
    a_1 = ora.score_unit(K, Q2[1:], w, trace=True)["a"]
    np.testing.assert_allclose(ab, 0.5 * (a_0 + a_1), rtol=1e-12)


def test_attention_matches_torch_sdpa_weights(ora):
    # The window-mean importance is the column mean of the causal attention
    # matrix of the window rows, which torch's softmax gives directly.
    T, D, G, w = 64, 16, 2, 6
    K, Q = rand_unit(7, T, D, G, w)
    a = ora.score_unit(K, Q, w, ora.Params(pool_kernel=1), trace=True)["a"]
    Kt = torch.tensor(K, dtype=torch.float64)
    Qt = torch.tensor(Q, dtype=torch.float64)
    logits = Qt @ Kt.T / math.sqrt(D)                     # [G, w, T]
    P = T - w
    mask = torch.arange(T)[None, :] > (P + torch.arange(w))[:, None]
    att = torch.softmax(logits.masked_fill(mask, -math.inf), dim=-1)
    np.testing.assert_allclose(a, att.mean(dim=(0, 1))[:P].numpy(), rtol=1e-12)


# --------------------------------------------------------------------------
# a3: average pooling, kernel 5 (Table 6)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("kp", [1, 3, 5, 7])
def test_pooling_matches_torch_avg_pool1d(ora, kp):
    T, D, w = 30, 8, 3
    K, Q = rand_unit(8, T, D, 1, w)
    r = ora.score_unit(K, Q, w, ora.Params(pool_kernel=kp), trace=True)
    a = torch.tensor(r["a"])[None, None, :]
    pooled = torch.nn.functional.avg_pool1d(a, kp, stride=1, padding=kp // 2, count_include_pad=True)
    np.testing.assert_allclose(r["imp"], pooled[0, 0].numpy(), rtol=1e-13)
    if kp == 1:
        np.testing.assert_array_equal(r["imp"], r["a"])


# --------------------------------------------------------------------------
# a4/a5/a6: anchors, cosine and Euclidean geometry (Eqs. (1)-(2), Appendix A.1)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_rC_is_mean_offdiagonal_cosine(ora, seed):
    T, D, w = 24, 10, 2
    K, Q = rand_unit(10 + seed, T, D, 1, w, offset=0.7)
    r = ora.score_unit(K, Q, w, trace=True)
    Kd = K.astype(np.float64)
    C = (Kd @ Kd.T) / np.outer(np.linalg.norm(Kd, axis=1), np.linalg.norm(Kd, axis=1))
    brute = (C.sum() - np.trace(C)) / (T * (T - 1))
    assert r["stats"][S_["rC"]] == pytest.approx(brute, abs=1e-12)
    # the cosine of each key to the others is bounded
    assert np.all(np.abs(r["cosmu"]) <= 1 + 1e-12)
    assert np.all((r["sC"] >= 0) & (r["sC"] <= 1))
    assert -1.0 / (T - 1) - 1e-12 <= r["stats"][S_["rC"]] <= 1 + 1e-12


def test_rC_closed_forms(ora):
    # orthonormal keys: all pairwise cosines 0 -> r_C = 0
    D, T = 8, 6
    K = f32(np.eye(D)[:T] * 3.0)
    Q = f32(np.ones((1, 1, D)))
    r = ora.score_unit(K, Q, 1, trace=True)
    assert r["stats"][S_["rC"]] == pytest.approx(0.0, abs=1e-15)
    # two antipodal keys: cosine -1 -> r_C = -1; mu = 0 -> s_C = 1/2
    K = f32([[1.0, 2.0, 0.0], [-2.0, -4.0, 0.0]])
    r = ora.score_unit(K, f32(np.ones((1, 1, 3))), 1, trace=True)
    assert r["stats"][S_["rC"]] == pytest.approx(-1.0, abs=1e-15)
    assert r["sC"][0] == pytest.approx(0.5, abs=1e-15)


def test_centroid_and_distances(ora):
    T, D, w = 33, 9, 4
    K, Q = rand_unit(20, T, D, 1, w, offset=1.3)
    r = ora.score_unit(K, Q, w, trace=True)
    Kd = K.astype(np.float64)
    np.testing.assert_allclose(r["kbar"], Kd.mean(axis=0), rtol=1e-13)
    # mean squared distance to the centroid = half the mean squared pairwise distance
    pair = ((Kd[:, None, :] - Kd[None, :, :]) ** 2).sum(-1)
    assert np.mean(r["dE"] ** 2) == pytest.approx(pair.sum() / (2 * T * T), rel=1e-12)
    # expansion identity of Sec. 4 (well conditioned here)
    kb = Kd.mean(axis=0)
    exp2 = (Kd ** 2).sum(1) - 2 * Kd @ kb + kb @ kb
    np.testing.assert_allclose(r["dE"] ** 2, exp2, rtol=1e-10)
    assert np.all(r["dE"] >= 0)
    # mu is the mean of the unit-normalised keys
    np.testing.assert_allclose(r["mu"], (Kd / np.linalg.norm(Kd, axis=1, keepdims=True)).mean(0), rtol=1e-13)


def test_rE_closed_form(ora):
    # keys +c e1 / -c e1 alternate (T even): centroid 0, every distance c, so
    # D_E = c.  With c = sqrt(D) ln 3, sigmoid(D_E / sqrt(D)) = 3/4 -> r_E = 1/2.
    D, T = 16, 10
    c = math.sqrt(D) * math.log(3.0)
    K = np.zeros((T, D), np.float32)
    K[0::2, 0] = c
    K[1::2, 0] = -c
    r = ora.score_unit(f32(K), f32(np.ones((1, 2, D))), 2, trace=True)
    c32 = float(np.float32(c))
    assert r["stats"][S_["DE"]] == pytest.approx(c32, rel=1e-14)
    assert r["stats"][S_["rE"]] == pytest.approx(2 - 2 / (1 + math.exp(-c32 / math.sqrt(D))), rel=1e-14)
    assert r["stats"][S_["rE"]] == pytest.approx(0.5, abs=1e-7)
    # a custom tau rescales the argument
    r2 = ora.score_unit(f32(K), f32(np.ones((1, 2, D))), 2, ora.Params(tau=c32), trace=True)
    assert r2["stats"][S_["rE"]] == pytest.approx(2 - 2 / (1 + math.exp(-1.0)), rel=1e-14)


def test_jensen_mean_distance_below_std(ora):
    # Appendix D: D_E <= D_std = sqrt(mean |k - kbar|^2)
    for seed in range(4):
        K, Q = rand_unit(30 + seed, 40, 12, 1, 3, offset=0.2 * seed)
        r = ora.score_unit(K, Q, 3, trace=True)
        dstd = math.sqrt(np.mean(r["dE"] ** 2))
        assert r["stats"][S_["DE"]] <= dstd + 1e-12
        assert 0 < r["stats"][S_["rE"]] <= 1


def test_minmax_preserves_order_and_ranges(ora):
    T, D, w = 60, 8, 4
    K, Q = rand_unit(40, T, D, 2, w, offset=0.5)
    r = ora.score_unit(K, Q, w, trace=True)
    P = T - w
    np.testing.assert_array_equal(np.argsort(r["sE"], kind="stable"), np.argsort(r["dE"][:P], kind="stable"))
    assert r["sE"].min() == 0.0 and r["sE"].max() < 1.0
    assert r["sbar"].min() == 0.0 and r["sbar"].max() < 1.0
    assert r["stats"][S_["dmin"]] == r["dE"][:P].min() and r["stats"][S_["dmax"]] == r["dE"][:P].max()


def test_window_keys_are_in_the_anchors_but_not_in_the_minmax(ora):
    # A far outlier inside the window moves the centroid (all-T anchors) but not
    # the min/max used for s_E (non-window keys only).
    T, D, w = 30, 6, 2
    K, Q = rand_unit(41, T, D, 1, w)
    K2 = K.copy()
    K2[-1] = 50.0
    r1 = ora.score_unit(K, Q, w, trace=True)
    r2 = ora.score_unit(f32(K2), Q, w, trace=True)
    assert not np.allclose(r1["kbar"], r2["kbar"])
    P = T - w
    assert r2["stats"][S_["dmax"]] == r2["dE"][:P].max() < r2["dE"][-1]


# --------------------------------------------------------------------------
# Degenerate heads (identical keys -> zero diversity)
# --------------------------------------------------------------------------

def test_identical_keys_zero_diversity_full_redundancy(ora):
    T, D, w = 25, 16, 3
    K = f32(np.tile(np.random.default_rng(9).standard_normal(D), (T, 1)))
    Q = f32(np.random.default_rng(10).standard_normal((2, w, D)))
    r = ora.score_unit(K, Q, w, trace=True)
    assert np.all(r["dE"] <= 1e-12 * np.abs(K).max())
    assert np.all(r["sE"] == 0.0) and np.all(r["sbar"] == 0.0)
    assert np.all(np.abs(r["sdiv"]) <= 1e-12)   # s_C = (1 - 1)/2 with khat.mu = 1
    for k in ("rC", "rE", "lambda_"):
        assert r["stats"][S_[k]] == pytest.approx(1.0, abs=1e-12)
    assert np.all(np.abs(r["S"]) <= 1e-12 * r["stats"][S_["imp_mean"]])
    # every score ties: the lowest positions are kept, then the window
    idx = ora.select_unit(np.zeros(T - w), T, w, 10)
    np.testing.assert_array_equal(idx, list(range(7)) + [22, 23, 24])


def test_zero_norm_key_normalises_to_zero(ora):
    T, D, w = 12, 4, 2
    K, Q = rand_unit(11, T, D, 1, w, offset=1.0)
    K[3] = 0.0
    r = ora.score_unit(f32(K), Q, w, trace=True)
    assert r["cosmu"][3] == 0.0 and r["sC"][3] == 0.5
    Kd = np.delete(K.astype(np.float64), 3, axis=0)
    mu = (Kd / np.linalg.norm(Kd, axis=1, keepdims=True)).sum(0) / T
    np.testing.assert_allclose(r["mu"], mu, rtol=1e-13)


def test_single_prefix_token(ora):
    # T = w + 1: one candidate; its normalised diversity is 0 and S = (1-lambda) S_imp.
    T, D, w = 5, 4, 4
    K, Q = rand_unit(12, T, D, 1, w)
    r = ora.score_unit(K, Q, w, trace=True)
    lam = r["stats"][S_["lambda_"]]
    assert r["sE"][0] == 0.0 and r["sbar"][0] == 0.0
    assert r["S"][0] == pytest.approx((1 - lam) * r["imp"][0], rel=1e-15)
    np.testing.assert_array_equal(ora.select_unit(r["S"], T, w, 5), [0, 1, 2, 3, 4])
    np.testing.assert_array_equal(ora.select_unit(r["S"], T, w, 4), [1, 2, 3, 4])


# --------------------------------------------------------------------------
# a7: rescale (Sec. 5.2) and final score (Eq. (7)); special cases
# --------------------------------------------------------------------------

def test_rescaled_diversity_matches_importance_mean(ora):
    T, D, w = 80, 16, 4
    K, Q = rand_unit(50, T, D, 3, w, offset=0.4)
    r = ora.score_unit(K, Q, w, trace=True)
    eps = 1e-6
    sb = r["stats"][S_["sbar_mean"]]
    assert np.mean(r["stilde"]) == pytest.approx(np.mean(r["imp"]) * sb / (sb + eps), rel=1e-12)
    assert np.mean(r["stilde"]) == pytest.approx(np.mean(r["imp"]), rel=1e-5)
    lam = r["stats"][S_["lambda_"]]
    # S is the convex blend; its mean equals the importance mean up to eps
    assert np.mean(r["S"]) == pytest.approx(np.mean(r["imp"]), rel=1e-5)
    np.testing.assert_allclose(r["S"], lam * r["stilde"] + (1 - lam) * r["imp"], rtol=1e-12)


def test_alpha_beta_zero_reduces_to_mixkv(ora):
    # alpha = beta = 0 leaves MixKV (Appendix A.1): diversity -khat.mu min-max
    # normalised and rescaled by mean(S_imp)/mean(sbar), weight lambda = r_C.
    T, D, w = 70, 16, 4
    K, Q = rand_unit(60, T, D, 2, w, offset=0.8)
    p = ora.Params(alpha=0.0, beta=0.0, eps=0.0)
    r = ora.score_unit(K, Q, w, p, trace=True)
    Kd = K.astype(np.float64)
    KN = Kd / np.linalg.norm(Kd, axis=1, keepdims=True)
    mu = KN.mean(axis=0)
    P = T - w
    sc = -KN[:P] @ mu
    sbar = (sc - sc.min()) / (sc.max() - sc.min())
    stil = sbar * np.mean(r["imp"]) / np.mean(sbar)
    rC = (T * T * (mu @ mu) - T) / (T * (T - 1))
    S = rC * stil + (1 - rC) * r["imp"]
    assert r["stats"][S_["lambda_"]] == pytest.approx(rC, rel=1e-12)
    np.testing.assert_allclose(r["S"], S, rtol=1e-10, atol=1e-18)


def test_lambda_zero_is_snapkv_and_lambda_one_alpha_one_is_centroid_distance(ora):
    T, D, w = 90, 16, 4
    K, Q = rand_unit(70, T, D, 2, w, offset=0.3)
    P = T - w
    r0 = ora.score_unit(K, Q, w, ora.Params(lambda_override=0.0), trace=True)
    np.testing.assert_array_equal(r0["S"], r0["imp"])
    # SnapKV top-k on pooled attention
    idx = ora.select_unit(r0["S"], T, w, 20)
    order = np.lexsort((np.arange(P), -r0["imp"]))[:16]
    np.testing.assert_array_equal(idx[:16], np.sort(order))
    # ranking purely by distance to the centroid (ManifoldKV-style ordering)
    r1 = ora.score_unit(K, Q, w, ora.Params(lambda_override=1.0, alpha=1.0), trace=True)
    d = np.linalg.norm(K.astype(np.float64) - K.astype(np.float64).mean(0), axis=1)[:P]
    idx1 = ora.select_unit(r1["S"], T, w, 20)
    np.testing.assert_array_equal(idx1[:16], np.sort(np.argsort(-d, kind="stable")[:16]))


def test_weights_follow_equations(ora):
    # Eq. (3)/(6): alpha and beta weight the Euclidean terms.
    T, D, w = 50, 8, 2
    K, Q = rand_unit(80, T, D, 1, w, offset=0.6)
    for a, b in [(0.8, 0.6), (0.3, 0.9), (1.0, 0.0)]:
        r = ora.score_unit(K, Q, w, ora.Params(alpha=a, beta=b), trace=True)
        st = r["stats"]
        assert st[S_["lambda_"]] == pytest.approx(b * st[S_["rE"]] + (1 - b) * st[S_["rC"]], rel=1e-14)
        np.testing.assert_allclose(r["sdiv"], a * r["sE"] + (1 - a) * r["sC"], rtol=1e-14)


def test_gqa_unit_mapping_in_batch_driver(ora):
    # The batch driver maps query head q to KV head q // G and sequences by cu_seqlens.
    wl = W.custom(5, L=2, Hq=6, Hkv=2, D=16, w=3, seqlens=[40, 23], dtype="f32", group=8)
    S, st = ora.score(wl.K, wl.Q, wl.L, wl.Hq, wl.Hkv, wl.cu_seqlens, wl.D, wl.w)
    cu = wl.cu_seqlens
    for l in range(2):
        for h in range(2):
            for s in range(2):
                r = ora.score_unit(wl.K[l, h, cu[s]:cu[s + 1]], wl.Q[l, h * 3:(h + 1) * 3, s], wl.w)
                off = cu[s] - s * wl.w
                np.testing.assert_array_equal(S[l, h, off:off + (cu[s + 1] - cu[s]) - wl.w], r["S"])
                np.testing.assert_array_equal(st[l, h, s], r["stats"])


# --------------------------------------------------------------------------
# a8: selection (Sec. 3), per head and layer-flat (AdaKV, Appendix A.1)
# --------------------------------------------------------------------------

def brute_topk(S, k):
    # full sort: larger score first, smaller position first among equals
    return np.sort(np.lexsort((np.arange(len(S)), -np.asarray(S)))[:k])


@pytest.mark.parametrize("seed", range(6))
def test_select_unit_matches_full_sort(ora, seed):
    r = np.random.default_rng(seed)
    T, w = int(r.integers(3, 60)), int(r.integers(1, 3))
    P = T - w
    S = r.integers(0, 5, size=P).astype(np.float64)  # many exact ties
    b = int(r.integers(w, T + 3))
    idx = ora.select_unit(S, T, w, b)
    if b >= T:
        np.testing.assert_array_equal(idx, np.arange(T))
        return
    k = b - w
    assert len(idx) == b
    np.testing.assert_array_equal(idx[:k], brute_topk(S, k))
    np.testing.assert_array_equal(idx[k:], np.arange(P, T))
    assert np.all(np.diff(idx) > 0)


def test_select_rejects_budget_below_window(ora):
    with pytest.raises(ValueError):
        ora.select_unit(np.zeros(10), 12, 2, 1)


def test_select_nan_ranks_last(ora):
    S = np.array([0.1, np.nan, 0.3, 0.2, np.nan])
    idx = ora.select_unit(S, 6, 1, 4)
    np.testing.assert_array_equal(idx, [0, 2, 3, 5])


@pytest.mark.parametrize("seed", range(5))
def test_select_flat_matches_brute_force(ora, seed):
    r = np.random.default_rng(100 + seed)
    H, T, w = int(r.integers(1, 5)), int(r.integers(4, 40)), int(r.integers(1, 3))
    P = T - w
    S = r.integers(0, 6, size=(H, P)).astype(np.float64)
    b = int(r.integers(w, T))
    idx, counts = ora.select_flat(S, T, w, b)
    assert counts.sum() == H * b and len(idx) == H * b
    flat = S.reshape(-1)
    chosen = set(np.lexsort((np.arange(H * P), -flat))[:H * (b - w)].tolist())
    o = 0
    for h in range(H):
        mine = [i for i in range(P) if h * P + i in chosen]
        got = idx[o:o + counts[h]]
        np.testing.assert_array_equal(got, mine + list(range(P, T)))
        o += counts[h]


def test_select_drivers_layouts(ora):
    L, Hkv, w = 2, 3, 2
    cu = [0, 10, 25]
    r = np.random.default_rng(7)
    S = r.standard_normal((L, Hkv, 25 - 2 * w))
    bud = [5, 30]   # second sequence keeps everything (b >= T)
    idx, counts, offsets = ora.select(S, L, Hkv, cu, w, bud, ora.PER_HEAD)
    assert len(idx) == L * Hkv * (5 + 15)
    for l in range(L):
        for h in range(Hkv):
            for s, (T, b) in enumerate([(10, 5), (15, 30)]):
                o = offsets[l, h, s]
                assert counts[l, h, s] == min(b, T)
                ref = ora.select_unit(S[l, h, cu[s] - s * w: cu[s] - s * w + T - w], T, w, b)
                np.testing.assert_array_equal(idx[o:o + counts[l, h, s]], ref)
    idx2, c2, o2 = ora.select(S, L, Hkv, cu, w, bud, ora.LAYER_FLAT)
    for l in range(L):
        for s, (T, b) in enumerate([(10, 5), (15, 30)]):
            Sh = S[l, :, cu[s] - s * w: cu[s] - s * w + T - w]
            ref, rc = ora.select_flat(Sh, T, w, b)
            start = o2[l, 0, s]
            np.testing.assert_array_equal(c2[l, :, s], rc)
            np.testing.assert_array_equal(idx2[start:start + rc.sum()], ref)


def test_compact_is_exact_gather(ora):
    wl = W.custom(3, L=1, Hq=2, Hkv=2, D=8, w=2, seqlens=[12, 9], dtype="bf16", group=4)
    r = np.random.default_rng(0)
    S = r.standard_normal((1, 2, 21 - 4))
    idx, counts, offsets = ora.select(S, 1, 2, wl.cu_seqlens, 2, [5, 4])
    Kc, Vc = ora.compact(wl.K, wl.V, 1, 2, wl.cu_seqlens, 8, idx, counts, offsets)
    for h in range(2):
        for s in range(2):
            o, n = offsets[0, h, s], counts[0, h, s]
            rows = wl.K[0, h, wl.cu_seqlens[s] + idx[o:o + n]]
            np.testing.assert_array_equal(Kc[o:o + n], rows)
            np.testing.assert_array_equal(Vc[o:o + n], wl.V[0, h, wl.cu_seqlens[s] + idx[o:o + n]])


# --------------------------------------------------------------------------
# Input decode: every bf16 configuration reaches the oracle as bit patterns
# --------------------------------------------------------------------------

def test_bf16_keys_decode_to_their_values(ora):
    # bf16 is the upper half of an IEEE binary32: 0x3f80 = 1, 0x4000 = 2,
    # 0x4040 = 3, 0xbf80 = -1, 0x3f00 = 0.5, 0x4120 = 10 (exact values).  With
    # identical window queries of zero the attention is uniform, so only the
    # anchors depend on the keys: kbar is the exact column mean of the values.
    bits = np.array([[0x3f80, 0x4000], [0x4040, 0xbf80], [0x3f00, 0x4120], [0x4000, 0x3f80]], np.uint16)
    vals = np.array([[1.0, 2.0], [3.0, -1.0], [0.5, 10.0], [2.0, 1.0]])
    Q = np.zeros((1, 1, 2), np.uint16)
    r = ora.score_unit(bits, Q, 1, ora.Params(pool_kernel=1), trace=True)
    np.testing.assert_array_equal(r["kbar"], vals.mean(axis=0))
    np.testing.assert_allclose(r["dE"], np.linalg.norm(vals - vals.mean(axis=0), axis=1), rtol=1e-15)
    # subnormal and negative-zero patterns decode exactly too
    bits2 = np.array([[0x0001, 0x8000], [0x0080, 0x0000], [0x3f80, 0x3f80]], np.uint16)
    vals2 = np.array([[2.0 ** -133, 0.0], [2.0 ** -126, 0.0], [1.0, 1.0]])
    r2 = ora.score_unit(bits2, np.zeros((1, 1, 2), np.uint16), 1, ora.Params(pool_kernel=1), trace=True)
    np.testing.assert_array_equal(r2["kbar"], vals2.mean(axis=0))


@pytest.mark.parametrize("seed", [0, 1])
def test_bf16_unit_equals_its_float32_values(ora, seed):
    # the same unit given as bf16 bit patterns and as the float32 values those
    # patterns encode (decoded here by numpy, not by the oracle) scores
    # identically, bit for bit, with the value norm too
    wl = W.custom(seed, L=1, Hq=6, Hkv=2, D=32, w=3, seqlens=[70], dtype="bf16", group=8, strength=2.0)
    for h in range(2):
        K, V, Q = wl.K[0, h], wl.V[0, h], wl.Q[0, 3 * h:3 * h + 3, 0]
        p = ora.Params(imp_mode=ora.IMP_ATTN_VNORM)
        rb = ora.score_unit(K, Q, wl.w, p, V=V)
        rf = ora.score_unit(W.bf16_bits_to_f32(K), W.bf16_bits_to_f32(Q), wl.w, p, V=W.bf16_bits_to_f32(V))
        np.testing.assert_array_equal(rb["S"], rf["S"])
        np.testing.assert_array_equal(rb["stats"], rf["stats"])
    Qd = wl.Q[0, :, 0, 0]
    O, lse = ora.decode(Qd[None, :, None], wl.K[0, 0, :9], wl.V[0, 0, :9], 1, 6, 2, 1, 32,
                        np.array([[[9], [0]]]), np.array([[[0], [9]]]))
    O2, lse2 = ora.decode(W.bf16_bits_to_f32(Qd)[None, :, None], W.bf16_bits_to_f32(wl.K[0, 0, :9]),
                          W.bf16_bits_to_f32(wl.V[0, 0, :9]), 1, 6, 2, 1, 32,
                          np.array([[[9], [0]]]), np.array([[[0], [9]]]))
    np.testing.assert_array_equal(O[0, :3], O2[0, :3])
    np.testing.assert_array_equal(lse[0, :3], lse2[0, :3])


# --------------------------------------------------------------------------
# Generator sanity (statistics of the synthetic tiny workload)
# --------------------------------------------------------------------------

def test_tiny_workload_statistics(ora):
    # offset norm 4, unit noise in D=128: base mean cosine ~ 16/(16+128) ~ 0.11
    # plus the duplicate clusters; mean distance ~ sqrt(128) * E[s] ~ 11.8.
    wl = W.tiny()
    S, st = ora.score(wl.K, wl.Q, wl.L, wl.Hq, wl.Hkv, wl.cu_seqlens, wl.D, wl.w)
    for h in range(2):
        assert 0.09 <= st[0, h, 0, S_["rC"]] <= 0.15
        assert 10.0 <= st[0, h, 0, S_["DE"]] <= 13.5
        assert 0.47 <= st[0, h, 0, S_["rE"]] <= 0.57


def test_tiny_regression_fixture(ora):
    # Regression record written by tests/golden/make_golden.py from the oracle alone.
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "tiny_oracle.json")) as f:
        g = json.load(f)
    wl = W.tiny()
    S, st = ora.score(wl.K, wl.Q, wl.L, wl.Hq, wl.Hkv, wl.cu_seqlens, wl.D, wl.w)
    idx, counts, offsets = ora.select(S, wl.L, wl.Hkv, wl.cu_seqlens, wl.w, wl.budget)
    for h, gh in enumerate(g["heads"]):
        np.testing.assert_allclose(st[0, h, 0], gh["stats"], rtol=1e-12)
        np.testing.assert_allclose(S[0, h, gh["score_positions"]], gh["scores"], rtol=1e-12)
        np.testing.assert_array_equal(idx[offsets[0, h, 0]:offsets[0, h, 0] + counts[0, h, 0]], gh["selected"])


# --------------------------------------------------------------------------
# Budgets per (layer, KV head) (PyramidKV layer schedule, SparseMM head
# budgets, Appendix A.1)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(4))
def test_select_head_budgets_matches_brute_force(ora, seed):
    r = np.random.default_rng(300 + seed)
    L, Hkv, w = int(r.integers(1, 4)), int(r.integers(1, 4)), int(r.integers(1, 3))
    lens = [int(x) for x in r.integers(w + 1, 40, size=int(r.integers(1, 4)))]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    B = len(lens)
    Ptot = int(cu[-1]) - B * w
    S = r.integers(0, 6, size=(L, Hkv, Ptot)).astype(np.float64)  # many exact ties
    bud = r.integers(w, max(lens) + 3, size=(L, Hkv)).astype(np.int32)
    bud[0, 0] = w                       # the window only
    idx, counts, offsets = ora.select(S, L, Hkv, cu, w, bud, ora.HEAD_BUDGETS)
    o = 0
    for l in range(L):
        for h in range(Hkv):
            for s, T in enumerate(lens):
                b, P = int(bud[l, h]), T - w
                n = min(b, T)
                assert offsets[l, h, s] == o and counts[l, h, s] == n
                got = idx[o:o + n]
                if b >= T:
                    np.testing.assert_array_equal(got, np.arange(T))
                else:
                    Su = S[l, h, cu[s] - s * w: cu[s] - s * w + P]
                    np.testing.assert_array_equal(got, list(brute_topk(Su, b - w)) + list(range(P, T)))
                o += n
    assert o == len(idx) == ora.index_count(L, Hkv, cu, bud, ora.HEAD_BUDGETS)


def test_select_head_budgets_rejects_budget_below_window(ora):
    with pytest.raises(ValueError):
        ora.select(np.zeros((1, 2, 8)), 1, 2, [0, 10], 2, [[3, 1]], ora.HEAD_BUDGETS)


# Schedules worked by hand from the formulas of Appendix A.1 (PyramidKV):
# b^{m-1} = total/(beta m), b^0 = 2 total/m - b^{m-1}, straight line between.
#  m=4, total=4096, beta=2:  b^3 = 512, b^0 = 1536, step 1024/3:
#                            1194.67 -> 1194, 853.33 -> 853
#  m=5, total=1000, beta=4:  b^4 = 50, b^0 = 350, step 75 (sum exactly 1000)
#  m=3, total=900, beta=1.5: b^2 = 200, b^0 = 400, step 100
#  m=3, total=100, beta=3:   b^2 = 100/9 -> 11, b^0 = 500/9 -> 55, 300/9 -> 33
#  m=1:                      the whole total
#  beta=1:                   b^{m-1} = b^0 = total/m, a flat schedule
PYRAMID_CASES = [
    (4, 4096, 2.0, [1536, 1194, 853, 512]),
    (5, 1000, 4.0, [350, 275, 200, 125, 50]),
    (3, 900, 1.5, [400, 300, 200]),
    (3, 100, 3.0, [55, 33, 11]),
    (1, 777, 3.0, [777]),
    (4, 4096, 1.0, [1024, 1024, 1024, 1024]),
]


@pytest.mark.parametrize("m,total,beta,want", PYRAMID_CASES)
def test_pyramid_schedule_worked_examples(ora, m, total, beta, want):
    assert ora.pyramid_budgets(m, total, beta) == want


@pytest.mark.parametrize("m,total,beta", [(28, 28 * 6553, 20.0), (32, 32 * 128, 20.0), (7, 1234.5, 2.5)])
def test_pyramid_schedule_properties(ora, m, total, beta):
    b = ora.pyramid_budgets(m, total, beta)
    assert len(b) == m
    # the two ends of the schedule (before rounding down)
    assert b[-1] == math.floor(total / (beta * m))
    assert abs(b[0] - (2 * total / m - total / (beta * m))) < 1
    # non-increasing for beta >= 1, the sum within m of the total, never above
    assert all(x >= y for x, y in zip(b, b[1:]))
    assert total - m < sum(b) <= total


# --------------------------------------------------------------------------
# Value-norm importance (imp_mode IMP_ATTN_VNORM; Sec. 5.2: the importance
# combines |v_i|_2 with the window-mean attention; reading: the product,
# taken after pooling)
# --------------------------------------------------------------------------

def vnorm_params(**kw):
    import oracle
    return oracle.Params(imp_mode=oracle.IMP_ATTN_VNORM, **kw)


def test_vnorm_with_unit_values_is_attention_importance(ora):
    K, Q = rand_unit(50, 60, 16, G=2, w=3)
    V = np.random.default_rng(51).standard_normal((60, 16))
    V = f32(V / np.linalg.norm(V, axis=1, keepdims=True))
    r0 = ora.score_unit(K, Q, 3)
    r1 = ora.score_unit(K, Q, 3, vnorm_params(), V=V)
    np.testing.assert_allclose(r1["S"], r0["S"], rtol=1e-6)
    np.testing.assert_allclose(r1["stats"], r0["stats"], rtol=1e-6)


def test_vnorm_closed_form_with_identical_keys(ora):
    # identical keys: a_i = mean_j 1 / (P + j + 1) for every i < P (pinned
    # above); a width-5 zero-padded pool gives a_i * (number of in-range
    # neighbours) / 5, which the value norm then multiplies
    T, D, G, w = 41, 8, 2, 3
    K = f32(np.tile(np.linspace(-1, 1, D), (T, 1)))
    Q = f32(np.random.default_rng(52).standard_normal((G, w, D)))
    V = f32(np.random.default_rng(53).standard_normal((T, D)) * 3.0)
    P = T - w
    r = ora.score_unit(K, Q, w, vnorm_params(), trace=True, V=V)
    a = np.mean([1.0 / (P + j + 1) for j in range(w)])
    inrange = np.array([sum(1 for t in range(-2, 3) if 0 <= i + t < P) for i in range(P)])
    vn = np.sqrt(np.sum(V[:P].astype(np.float64) ** 2, axis=1))
    np.testing.assert_allclose(r["imp"], a * inrange / 5.0 * vn, rtol=1e-12)
    assert r["stats"][S_["imp_mean"]] == pytest.approx(np.mean(a * inrange / 5.0 * vn), rel=1e-12)


def test_vnorm_scales_with_the_values_and_keeps_the_selection(ora):
    # lambda does not depend on V; S_imp, the rescaled diversity and S all
    # scale by c when V does (c = 2: exact in fp32)
    K, Q = rand_unit(54, 80, 16, G=2, w=2, offset=0.4)
    V = f32(np.random.default_rng(55).standard_normal((80, 16)))
    r1 = ora.score_unit(K, Q, 2, vnorm_params(), V=V)
    r2 = ora.score_unit(K, Q, 2, vnorm_params(), V=f32(2.0 * V))
    np.testing.assert_allclose(r2["S"], 2.0 * r1["S"], rtol=1e-12)
    for k in ("lambda_", "rC", "rE", "DE", "sbar_mean"):
        assert r2["stats"][S_[k]] == pytest.approx(r1["stats"][S_[k]], rel=1e-12)
    for k in ("imp_mean", "scale"):
        assert r2["stats"][S_[k]] == pytest.approx(2.0 * r1["stats"][S_[k]], rel=1e-12)
    np.testing.assert_array_equal(ora.select_unit(r1["S"], 80, 2, 20), ora.select_unit(r2["S"], 80, 2, 20))


def test_vnorm_dominant_value_row_is_kept(ora):
    # with lambda = 0 the score is S_imp; a value row 1000 times longer than
    # the others makes its key the clear first choice
    K, Q = rand_unit(56, 50, 16, G=1, w=2)
    V = f32(np.random.default_rng(57).standard_normal((50, 16)) * 0.01)
    V[17] *= 1e5
    r = ora.score_unit(K, Q, 2, vnorm_params(lambda_override=0.0), V=V)
    assert int(np.argmax(r["S"])) == 17
    np.testing.assert_array_equal(ora.select_unit(r["S"], 50, 2, 3), [17, 48, 49])


def test_vnorm_needs_values(ora):
    K, Q = rand_unit(58, 20, 8)
    with pytest.raises(ValueError):
        ora.score_unit(K, Q, 2, vnorm_params())


# --------------------------------------------------------------------------
# Alternatives of Sec. 6.3 (Table 4: winsorised min-max, MAD scaling),
# Appendix D (r_std) and Appendix B.6 (centroid over the non-window keys)
# --------------------------------------------------------------------------

def alt_params(**kw):
    import oracle
    return oracle.Params(**kw)


def test_winsor_at_zero_is_minmax(ora):
    K, Q = rand_unit(70, 90, 16, G=2, w=3, offset=0.3)
    r0 = ora.score_unit(K, Q, 3, trace=True)
    r1 = ora.score_unit(K, Q, 3, alt_params(norm_mode=ora.NORM_WINSOR, winsor_q=0.0), trace=True)
    np.testing.assert_array_equal(r1["sE"], r0["sE"])
    np.testing.assert_array_equal(r1["S"], r0["S"])


@pytest.mark.parametrize("q,T", [(0.01, 300), (0.05, 300), (0.05, 41), (0.25, 12)])
def test_winsor_matches_numpy_quantiles(ora, q, T):
    K, Q = rand_unit(71, T, 16, G=2, w=2, offset=0.2)
    P = T - 2
    r = ora.score_unit(K, Q, 2, alt_params(norm_mode=ora.NORM_WINSOR, winsor_q=q), trace=True)
    d = r["dE"][:P]
    lo, hi = np.quantile(d, [q, 1 - q])
    np.testing.assert_allclose(r["sE"], (np.clip(d, lo, hi) - lo) / (hi - lo + 1e-6), rtol=1e-12, atol=1e-15)
    # the clipped extremes map to 0 and (almost) 1
    assert r["sE"].min() == 0.0 and abs(r["sE"].max() - (hi - lo) / (hi - lo + 1e-6)) < 1e-12


@pytest.mark.parametrize("T,tau", [(200, 1.0), (57, 1.0), (58, 2.5)])
def test_mad_matches_numpy_median(ora, T, tau):
    K, Q = rand_unit(72, T, 16, G=1, w=3, offset=0.5)
    P = T - 3
    r = ora.score_unit(K, Q, 3, alt_params(norm_mode=ora.NORM_MAD, mad_tau=tau), trace=True)
    d = r["dE"][:P]
    med = np.median(d)
    mad = np.median(np.abs(d - med))
    np.testing.assert_allclose(r["sE"], 1.0 / (1.0 + np.exp(-(d - med) / (tau * mad + 1e-6))), rtol=1e-12)
    # half of the keys lie at or above the median: s_E >= 1/2 for them
    assert np.sum(r["sE"] >= 0.5) >= P // 2


def test_rstd_is_the_key_standard_deviation(ora):
    # mean_T |k - kbar|^2 is the summed per-dimension variance of the keys
    K, Q = rand_unit(73, 120, 16, G=2, w=2, scale=1.7, offset=0.8)
    tau = 4.0
    r = ora.score_unit(K, Q, 2, alt_params(redundancy=ora.RED_STD, tau=tau, beta=1.0))
    Dstd = np.sqrt(np.var(K.astype(np.float64), axis=0).sum())
    rstd = 1.0 - 1.0 / (1.0 + np.exp(-Dstd / tau))
    assert r["stats"][S_["rE"]] == pytest.approx(rstd, rel=1e-12)
    assert r["stats"][S_["lambda_"]] == pytest.approx(rstd, rel=1e-12)   # beta = 1
    # r_std lies in (0, 1/2) and D_E <= D_std (Jensen)
    assert 0.0 < rstd < 0.5 and r["stats"][S_["DE"]] <= Dstd * (1 + 1e-12)


def test_rstd_two_antipodal_keys(ora):
    # k and -k: kbar = 0, every distance is |k|, D_std = |k|
    k = np.array([3.0, 4.0, 0.0, 0.0], np.float32)
    K = np.stack([k, -k, k, -k]).astype(np.float32)
    Q = np.ones((1, 1, 4), np.float32)
    r = ora.score_unit(K, Q, 1, alt_params(redundancy=ora.RED_STD, tau=5.0))
    assert r["stats"][S_["rE"]] == pytest.approx(1.0 - 1.0 / (1.0 + np.exp(-1.0)), rel=1e-12)


def test_prefix_centroid_ignores_the_window_keys(ora):
    T, w = 70, 4
    K, Q = rand_unit(74, T, 16, G=2, w=w, offset=0.3)
    P = T - w
    pp = alt_params(centroid_scope=ora.CENTROID_PREFIX)
    r1 = ora.score_unit(K, Q, w, pp, trace=True)
    np.testing.assert_allclose(r1["kbar"], K[:P].astype(np.float64).mean(axis=0), rtol=1e-12, atol=1e-15)
    K2 = K.copy()
    K2[P:] += np.float32(5.0)        # move only the window keys
    r2 = ora.score_unit(K2, Q, w, pp, trace=True)
    np.testing.assert_array_equal(r2["kbar"], r1["kbar"])
    np.testing.assert_array_equal(r2["dE"][:P], r1["dE"][:P])
    np.testing.assert_array_equal(r2["sE"], r1["sE"])
    # with the centroid over all T keys the same move changes the distances
    a1 = ora.score_unit(K, Q, w, trace=True)
    a2 = ora.score_unit(K2, Q, w, trace=True)
    assert np.abs(a2["dE"][:P] - a1["dE"][:P]).max() > 1e-3


# --------------------------------------------------------------------------
# Decode attention over the compressed cache (the generation step, Sec. 3)
# --------------------------------------------------------------------------

def test_decode_one_row_returns_its_value(ora):
    r = np.random.default_rng(90)
    D = 16
    Q = f32(r.standard_normal((1, 1, 1, D)))
    Kc, Vc = f32(r.standard_normal((1, D))), f32(r.standard_normal((1, D)))
    O, lse = ora.decode(Q, Kc, Vc, 1, 1, 1, 1, D, [[[1]]], [[[0]]])
    np.testing.assert_allclose(O[0, 0, 0], Vc[0].astype(np.float64), rtol=1e-15)
    x = float(np.dot(Q[0, 0, 0].astype(np.float64), Kc[0].astype(np.float64)) / 4.0)
    assert lse[0, 0, 0] == pytest.approx(x, rel=1e-14)


def test_decode_identical_keys_average_the_values(ora):
    r = np.random.default_rng(91)
    D, n = 8, 13
    Kc = f32(np.tile(r.standard_normal(D), (n, 1)))
    Vc = f32(r.standard_normal((n, D)))
    Q = f32(r.standard_normal((1, 1, 1, D)))
    O, lse = ora.decode(Q, Kc, Vc, 1, 1, 1, 1, D, [[[n]]], [[[0]]])
    np.testing.assert_allclose(O[0, 0, 0], Vc.astype(np.float64).mean(axis=0), rtol=1e-13)
    x = float(np.dot(Q[0, 0, 0].astype(np.float64), Kc[0].astype(np.float64)) / np.sqrt(D))
    assert lse[0, 0, 0] == pytest.approx(x + np.log(n), rel=1e-13)


def test_decode_matches_torch_attention_and_logsumexp(ora):
    from scipy.special import logsumexp
    r = np.random.default_rng(92)
    L, Hq, Hkv, B, D = 2, 6, 2, 2, 32
    G = Hq // Hkv
    counts = r.integers(1, 40, size=(L, Hkv, B)).astype(np.int32)
    offsets = np.concatenate([[0], np.cumsum(counts.reshape(-1))[:-1]]).reshape(L, Hkv, B).astype(np.int32)
    n = int(counts.sum())
    Kc, Vc = f32(r.standard_normal((n, D)) * 2), f32(r.standard_normal((n, D)))
    Q = f32(r.standard_normal((L, Hq, B, D)))
    O, lse = ora.decode(Q, Kc, Vc, L, Hq, Hkv, B, D, counts, offsets)
    for l in range(L):
        for q in range(Hq):
            for s in range(B):
                h = q // G
                o, c = offsets[l, h, s], counts[l, h, s]
                k = torch.from_numpy(Kc[o:o + c].astype(np.float64))
                v = torch.from_numpy(Vc[o:o + c].astype(np.float64))
                qq = torch.from_numpy(Q[l, q, s].astype(np.float64))
                ref = torch.nn.functional.scaled_dot_product_attention(qq[None, None], k[None], v[None])[0, 0]
                np.testing.assert_allclose(O[l, q, s], ref.numpy(), rtol=1e-12, atol=1e-14)
                x = (k @ qq).numpy() / np.sqrt(D)
                assert lse[l, q, s] == pytest.approx(logsumexp(x), rel=1e-13)


# --------------------------------------------------------------------------
# the first sweep's results as a prefill hands them over: key sums (Eq. (1);
# Appendix A.1 mu) and window softmax statistics (Sec. 3 attention)
# --------------------------------------------------------------------------

def test_prefill_sums_of_identical_keys(ora):
    # every key is v: sum k = T v and sum k/|k| = T v/|v|; every logit of a
    # row is q.v/sqrt(D), so that is its max, and the sum of exp(logit - max)
    # counts the keys the row sees (P + j + 1 causal, all T otherwise)
    T, D, G, w = 29, 16, 3, 4
    K = f32(np.tile(np.linspace(-1.5, 2.0, D), (T, 1)))
    Q = f32(np.random.default_rng(3).standard_normal((G, w, D)))
    v = K[0].astype(np.float64)
    P, R = T - w, G * w
    for causal in (True, False):
        pre = ora.prefill_unit(K, Q, w, causal)
        assert pre.shape == (2 * D + 2 * R,)
        np.testing.assert_allclose(pre[:D], T * v, rtol=1e-13)
        np.testing.assert_allclose(pre[D:2 * D], T * v / math.sqrt(float(v @ v)), rtol=1e-13)
        for g in range(G):
            for j in range(w):
                r = g * w + j
                qv = float(Q[g, j].astype(np.float64) @ v) / math.sqrt(D)
                assert pre[2 * D + r] == pytest.approx(qv, rel=1e-12, abs=1e-12)
                assert pre[2 * D + R + r] == pytest.approx(P + j + 1 if causal else T, rel=1e-12)


def test_prefill_zero_key_adds_no_direction(ora):
    # a zero key counts as zero in sum k/|k| (its norm is floored, not divided by)
    T, D, w = 12, 8, 2
    K = f32(np.tile(np.arange(1, D + 1, dtype=np.float64), (T, 1)))
    K[5] = 0.0
    Q = f32(np.zeros((1, w, D)))
    pre = ora.prefill_unit(K, Q, w)
    v = K[0].astype(np.float64)
    np.testing.assert_allclose(pre[D:2 * D], (T - 1) * v / np.linalg.norm(v), rtol=1e-13)
    np.testing.assert_allclose(pre[:D], (T - 1) * v, rtol=1e-13)
    # zero queries: every visible logit is 0
    np.testing.assert_array_equal(pre[2 * D:2 * D + w], 0.0)
    np.testing.assert_allclose(pre[2 * D + w:], [T - w + j + 1 for j in range(w)], rtol=1e-13)


def test_prefill_window_statistics_are_a_logsumexp(ora):
    # max + log(sum) is the log-sum-exp of the row's visible logits (scipy's
    # routine), and the max term alone contributes 1 to the sum
    from scipy.special import logsumexp
    T, D, G, w = 45, 32, 2, 5
    K, Q = rand_unit(4, T, D, G, w, scale=2.0)
    P, R = T - w, G * w
    Kd = K.astype(np.float64)
    for causal in (True, False):
        pre = ora.prefill_unit(K, Q, w, causal)
        for g in range(G):
            for j in range(w):
                r = g * w + j
                x = Kd[:(P + j + 1) if causal else T] @ Q[g, j].astype(np.float64) / math.sqrt(D)
                assert pre[2 * D + r] + math.log(pre[2 * D + R + r]) == pytest.approx(logsumexp(x), rel=1e-12)
                assert 1.0 <= pre[2 * D + R + r] <= len(x)


def test_prefill_sums_are_the_score_anchors_times_T(ora):
    # the score's own centroid and mu (its trace) are these sums over T
    T, D, G, w = 60, 16, 2, 3
    K, Q = rand_unit(5, T, D, G, w, offset=0.7)
    pre = ora.prefill_unit(K, Q, w)
    tr = ora.score_unit(K, Q, w, trace=True)
    np.testing.assert_allclose(pre[:D] / T, tr["kbar"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(pre[D:2 * D] / T, tr["mu"], rtol=1e-12, atol=1e-15)
    mu = pre[D:2 * D] / T
    assert float(mu @ mu) == pytest.approx(tr["stats"][S_["mu_norm2"]], rel=1e-12)


def test_prefill_sums_driver_layout(ora):
    # the whole-tensor form takes unit (l, h, s) from the same places as the score
    wl = W.custom(6, 2, 4, 2, 16, 3, [20, 33], dtype="f32")
    pre = ora.prefill_sums(wl.K, wl.Q, wl.L, wl.Hq, wl.Hkv, wl.cu_seqlens, wl.D, wl.w)
    cu, G = wl.cu_seqlens, wl.Hq // wl.Hkv
    for l in range(wl.L):
        for h in range(wl.Hkv):
            for s in range(len(cu) - 1):
                want = ora.prefill_unit(wl.K[l, h, cu[s]:cu[s + 1]], wl.Q[l, h * G:(h + 1) * G, s], wl.w)
                np.testing.assert_array_equal(pre[l, h, s], want)
