"""Pins of the oracle's calibration to what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a closed
form (Proposition 1), an exact identity of the moments, brute force over
rank-r maps, special cases that reduce to textbook PCA, or hand-derived
values (tests/golden/hand_2x2.json).
"""
import json
import os

import numpy as np
import pytest
from scipy.optimize import minimize

import oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_2x2.json")


def _spd(rng, d, cond=1e3):
    A = rng.standard_normal((d, d))
    Qm, _ = np.linalg.qr(A)
    w = np.geomspace(1.0, 1.0 / cond, d) * rng.uniform(0.5, 2.0)
    return (Qm * w) @ Qm.T


def _calib_from_moments(Sq, Sk, r):
    """Run the oracle's calibration on samples whose moments are exactly Sq, Sk
    (zero key mean): T = 2d rows built from +/- columns of a square root."""
    d = Sq.shape[0]
    Lq = np.linalg.cholesky(Sq)
    Lk = np.linalg.cholesky(Sk)
    # rows +-sqrt(d) * L[:, i]: (1/T) sum x x^T = (1/2d) * 2 * d * L L^T = S
    q = np.concatenate([np.sqrt(d) * Lq.T, -np.sqrt(d) * Lq.T])
    k = np.concatenate([np.sqrt(d) * Lk.T, -np.sqrt(d) * Lk.T])
    return O.saki_calibrate(q, k, r)


def test_moments_are_exact_from_constructed_samples():
    rng = np.random.default_rng(0)
    Sq, Sk = _spd(rng, 6), _spd(rng, 6)
    cal = _calib_from_moments(Sq, Sk, 2)
    np.testing.assert_allclose(cal["Sigma_q"], Sq, rtol=0, atol=1e-13)
    np.testing.assert_allclose(cal["Sigma_k"], Sk, rtol=0, atol=1e-13)
    np.testing.assert_allclose(cal["mu"], 0.0, atol=1e-15)


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: c["name"])
def test_hand_derived_2x2(case):
    Sq = np.array(case["Sigma_q"])
    Sk = np.array(case["Sigma_k"])
    cal = _calib_from_moments(Sq, Sk, case["r"])
    np.testing.assert_allclose(cal["sigma"], case["sigma"], rtol=1e-14)
    np.testing.assert_allclose(cal["tail"], case["tail"], rtol=1e-13)
    np.testing.assert_allclose(cal["M"], case["M"], atol=1e-14)
    np.testing.assert_allclose(cal["B_q"], case["B_q"], atol=1e-14)
    np.testing.assert_allclose(cal["B_k"], case["B_k"], atol=1e-14)
    np.testing.assert_allclose(O.predicted_reduction(cal["sigma"], case["r"]),
                               case["predicted_reduction"], rtol=1e-14)
    if "pca_loss" in case:
        V = O.key_pca_factors(cal["Sigma_k"], case["r"])
        L = O.score_loss(V @ V.T, cal["Sq_half"], cal["Sk_half"])
        np.testing.assert_allclose(L, case["pca_loss"], rtol=1e-13)


@pytest.mark.parametrize("d,r", [(4, 1), (8, 3), (16, 5), (128, 32), (128, 16), (128, 64)])
def test_prop1_optimum_equals_tail_energy(d, r):
    rng = np.random.default_rng(d * 100 + r)
    Sq, Sk = _spd(rng, d), _spd(rng, d)
    cal = _calib_from_moments(Sq, Sk, r)
    L = O.score_loss(cal["M"], cal["Sq_half"], cal["Sk_half"])
    assert abs(L - cal["tail"]) <= 1e-11 * np.sum(cal["sigma"] ** 2)
    # the truncation is a genuine one: rank exactly r
    assert np.linalg.matrix_rank(cal["M"], tol=1e-9 * np.abs(cal["M"]).max()) == r


def test_empirical_calibration_mse_equals_loss():
    """With 1/T moments, centred keys and uncentred queries, the mean squared
    score error over ALL calibration (query, key) pairs equals L(M_r) exactly
    (Eq. 1-2 with the sample moments)."""
    spec = W.SPECS["single_head_d128"]
    inp = W.make_layer(spec)
    q, k = inp["q_cal"][0].astype(np.float64), inp["k_cal"][0].astype(np.float64)
    cal = O.saki_calibrate(q, k, 32)
    assert cal["n_clamped"] == (0, 0)
    kc = k - cal["mu"]
    E = q @ (np.eye(128) - cal["M"]) @ kc.T
    mse = np.mean(E * E)
    assert abs(mse - cal["tail"]) <= 1e-9 * cal["tail"]
    # and a dropped centring would not pass: uncentred keys give another value
    E2 = q @ (np.eye(128) - cal["M"]) @ k.T
    assert abs(np.mean(E2 * E2) - cal["tail"]) > 1e-6 * cal["tail"]


@pytest.mark.parametrize("seed", range(3))
def test_optimum_beats_pca_wsvd_and_random_maps(seed):
    rng = np.random.default_rng(seed)
    d, r = 16, 4
    Sq, Sk = _spd(rng, d, 1e2), _spd(rng, d, 1e2)
    cal = _calib_from_moments(Sq, Sk, r)
    Lopt = O.score_loss(cal["M"], cal["Sq_half"], cal["Sk_half"])
    V = O.key_pca_factors(cal["Sigma_k"], r)
    assert Lopt <= O.score_loss(V @ V.T, cal["Sq_half"], cal["Sk_half"]) + 1e-12
    for _ in range(1000):
        P = rng.standard_normal((d, r)) @ rng.standard_normal((r, d))
        assert Lopt <= O.score_loss(P, cal["Sq_half"], cal["Sk_half"]) + 1e-12
    # small perturbations of the optimal factors never improve on it
    for _ in range(200):
        Bq = cal["B_q"] + 1e-3 * rng.standard_normal(cal["B_q"].shape)
        Bk = cal["B_k"] + 1e-3 * rng.standard_normal(cal["B_k"].shape)
        assert Lopt <= O.score_loss(Bq @ Bk.T, cal["Sq_half"], cal["Sk_half"]) + 1e-12


def test_bruteforce_d4_r1_never_beats_closed_form():
    """d = 4, r = 1: search over rank-1 maps P = a b^T.  (i) b on a dense set of
    directions on the 3-sphere with the exact least-squares a(b):
    min_a L(a b^T) = ||C||^2 - ||C w||^2 / ||w||^2, w = Sigma_k^{1/2} b.
    (ii) raw (a, b) in R^8 refined by Nelder-Mead on L itself."""
    rng = np.random.default_rng(7)
    Sq, Sk = _spd(rng, 4, 30.0), _spd(rng, 4, 30.0)
    cal = _calib_from_moments(Sq, Sk, 1)
    C = cal["C"]
    closed = cal["tail"]
    b = rng.standard_normal((200000, 4))
    w = b @ cal["Sk_half"]  # Sk_half symmetric
    Cw = w @ C.T
    lb = np.sum(C * C) - np.sum(Cw * Cw, 1) / np.sum(w * w, 1)
    assert lb.min() >= closed - 1e-12 * np.sum(C * C)
    assert lb.min() <= closed * (1 + 1e-3)  # the dense search approaches it

    def f(x):
        return O.score_loss(np.outer(x[:4], x[4:]), cal["Sq_half"], cal["Sk_half"])

    best = np.inf
    for _ in range(20):
        res = minimize(f, rng.standard_normal(8), method="Nelder-Mead",
                       options={"xatol": 1e-12, "fatol": 1e-14, "maxiter": 20000,
                                "maxfev": 40000})
        best = min(best, res.fun)
        assert res.fun >= closed - 1e-12 * np.sum(C * C)
    assert best <= closed * (1 + 1e-6)


def test_rank_d_reproduces_exact_scores():
    spec = W.SPECS["single_head_d128"].with_(N=256, Q=32)
    inp = W.make_layer(spec)
    cal = O.saki_calibrate(inp["q_cal"][0], inp["k_cal"][0], 128)
    np.testing.assert_allclose(cal["M"], np.eye(128), atol=1e-9)
    q, keys = inp["queries"][0, 0], inp["keys"][0, 0]
    s_hat, *_ = O.index_scores(cal["B_q"], cal["B_k"], cal["mu"], q, keys)
    s = O.exact_scores(q, keys)
    scale = O.score_scale(np.eye(128), np.eye(128), cal["mu"], q, keys)
    assert np.max(np.abs(s_hat - s) / scale) < 1e-9
    lim = O.candidate_limits(32, 256)
    hits = O.recall_hits(O.topk_rows(s_hat, lim), O.topk_rows(s, lim))
    assert np.all(hits == 64)


def test_identity_query_moment_reduces_to_key_pca():
    """Sigma_q = I: the weighted objective is the PCA objective (Sec. 5), so M_r
    is the orthogonal projector on the top-r eigenvectors of Sigma_k."""
    rng = np.random.default_rng(3)
    d, r = 12, 5
    Sk = _spd(rng, d, 50.0)
    cal = _calib_from_moments(np.eye(d), Sk, r)
    w, V = np.linalg.eigh(Sk)
    Vr = V[:, np.argsort(-w)[:r]]
    np.testing.assert_allclose(cal["M"], Vr @ Vr.T, atol=1e-12)
    # and the symmetric case Sigma_k = I: query PCA
    Sq = _spd(rng, d, 50.0)
    cal = _calib_from_moments(Sq, np.eye(d), r)
    w, U = np.linalg.eigh(Sq)
    Ur = U[:, np.argsort(-w)[:r]]
    np.testing.assert_allclose(cal["M"], Ur @ Ur.T, atol=1e-12)


def test_factorisation_and_direct_route_agree():
    """Appendix A factorisation identity: codes reproduce q^T M_r (k - mu)."""
    spec = W.SPECS["single_head_d128"].with_(N=512, Q=64)
    inp = W.make_layer(spec)
    cal = O.saki_calibrate(inp["q_cal"][0], inp["k_cal"][0], 32)
    U, s, V = cal["U"], cal["sigma"], cal["V"]
    Mr = cal["Sq_ihalf"] @ (U[:, :32] * s[:32]) @ V[:, :32].T @ cal["Sk_ihalf"]
    np.testing.assert_allclose(cal["M"], Mr, atol=1e-10 * np.abs(Mr).max())
    q, keys = inp["queries"][0, 0], inp["keys"][0, 0]
    s1, *_ = O.index_scores(cal["B_q"], cal["B_k"], cal["mu"], q, keys)
    s2 = O.direct_scores(q, cal["M"], cal["mu"], keys)
    scale = O.score_scale(cal["B_q"], cal["B_k"], cal["mu"], q, keys)
    assert np.max(np.abs(s1 - s2) / scale) < 1e-12


def test_map_is_an_oblique_projector():
    """With full-rank (clamped) moments, U_r Lambda_r = C V_r gives
    M_r = Sigma_k^{1/2} V_r V_r^T Sigma_k^{-1/2}, so M_r^2 = M_r.  This is the
    algebra of Eq. 3; it disagrees with the paper's Remark 1 (see design notes)."""
    rng = np.random.default_rng(11)
    d, r = 32, 8
    cal = _calib_from_moments(_spd(rng, d), _spd(rng, d), r)
    M = cal["M"]
    Vr = cal["V"][:, :r]
    np.testing.assert_allclose(M @ M, M, atol=1e-9 * np.abs(M).max())
    np.testing.assert_allclose(M, cal["Sk_half"] @ Vr @ Vr.T @ cal["Sk_ihalf"],
                               atol=1e-9 * np.abs(M).max())


def test_invariant_to_moment_scale_and_root_choice():
    spec = W.SPECS["single_head_d128"]
    inp = W.make_layer(spec)
    q, k = inp["q_cal"][0].astype(np.float64), inp["k_cal"][0].astype(np.float64)
    base = O.saki_calibrate(q, k, 16)
    scaled = O.saki_calibrate(3.0 * q, 0.25 * k, 16)
    np.testing.assert_allclose(scaled["M"], base["M"], atol=1e-8 * np.abs(base["M"]).max())
    # Cholesky roots (Sigma = L L^T) instead of symmetric roots give the same map
    Lq = np.linalg.cholesky(base["Sigma_q"])
    Lk = np.linalg.cholesky(base["Sigma_k"])
    Cc = Lq.T @ Lk
    U, s, Vt = np.linalg.svd(Cc)
    Mc = np.linalg.solve(Lq.T, (U[:, :16] * s[:16]) @ Vt[:16]) @ np.linalg.inv(Lk)
    np.testing.assert_allclose(Mc, base["M"], atol=1e-7 * np.abs(base["M"]).max())
    np.testing.assert_allclose(s, base["sigma"], rtol=1e-9)


def test_clamp_keeps_rank_d_exact_on_deficient_moments():
    """T < d makes both moments singular; clamping at 1e-6 lambda_max keeps
    them invertible so r = d still yields M = I (Appendix A, reading: clamp)."""
    rng = np.random.default_rng(5)
    q = rng.standard_normal((40, 64))
    k = rng.standard_normal((40, 64)) + 0.5
    cal = O.saki_calibrate(q, k, 64)
    nq, nk = cal["n_clamped"]
    assert nq >= 64 - 40 and nk >= 64 - 39
    np.testing.assert_allclose(cal["M"], np.eye(64), atol=1e-7)


def test_constant_keys_fall_back_to_identity_moment():
    q = np.random.default_rng(1).standard_normal((64, 8))
    k = np.tile(np.arange(8.0), (64, 1))
    cal = O.saki_calibrate(q, k, 4)
    assert cal["n_clamped"][1] == 8
    np.testing.assert_array_equal(cal["mu"], np.arange(8.0))
    c = O.codes(cal["B_k"], cal["mu"], k)
    assert np.all(c == 0.0)


@pytest.mark.parametrize("layer", range(4))
def test_loss_ordering_saki_pca_wsvd(layer):
    """L(SAKI) <= L(key PCA) (a theorem: Proposition 1) and, on this generator,
    L(key PCA) <= L(weight SVD) (an empirical ordering, Table 1)."""
    spec = W.SPECS["single_head_d128"]
    inp = W.make_layer(spec, layer=layer)
    cal = O.saki_calibrate(inp["q_cal"][0], inp["k_cal"][0], 32)
    Lopt = O.score_loss(cal["M"], cal["Sq_half"], cal["Sk_half"])
    V = O.key_pca_factors(cal["Sigma_k"], 32)
    Lpca = O.score_loss(V @ V.T, cal["Sq_half"], cal["Sk_half"])
    Uw = O.weight_svd_factors(inp["W_K"][0], 32)
    Lw = O.score_loss(Uw @ Uw.T, cal["Sq_half"], cal["Sk_half"])
    assert Lopt <= Lpca <= Lw
    assert abs(Lopt - cal["tail"]) <= 1e-10 * np.sum(cal["sigma"] ** 2)


def _orthonormal(rng, n, m):
    Qm, _ = np.linalg.qr(rng.standard_normal((n, m)))
    return Qm


def test_weight_svd_of_an_exact_rank_r_projection():
    """W_K = U_r diag(s) V_r^T of exact rank r (U_r [d, r], V_r [D, r]
    orthonormal, chosen here): the weight-SVD factors span exactly U_r, so
    P = U_r U_r^T, every key k = W_K x lies in the range and is reproduced,
    sketch scores equal the exact q.k, and recall@64 is 1.  Taking any other
    singular vectors (the trailing ones, or the right ones) fails: P would
    miss the keys' range."""
    rng = np.random.default_rng(8)
    d, D, r = 128, 256, 32
    U_r = _orthonormal(rng, d, r)
    V_r = _orthonormal(rng, D, r)
    s = np.linspace(5.0, 1.0, r)
    W_K = (U_r * s) @ V_r.T
    U = O.weight_svd_factors(W_K, r)
    assert U.shape == (d, r)
    np.testing.assert_allclose(U @ U.T, U_r @ U_r.T, atol=1e-12)
    x = rng.standard_normal((2048, D))
    keys = x @ W_K.T
    mu = keys[:512].mean(0)
    P = U @ U.T
    np.testing.assert_allclose(keys @ P.T, keys, atol=1e-11 * np.abs(keys).max())
    q = rng.standard_normal((40, d))
    s_hat, *_ = O.index_scores(U, U, mu, q, keys)
    s_ex = O.exact_scores(q, keys)
    assert np.max(np.abs(s_hat - s_ex)) <= 1e-11 * np.abs(s_ex).max()
    lim = O.candidate_limits(40, 2048)
    assert np.all(O.recall_hits(O.topk_rows(s_hat, lim), O.topk_rows(s_ex, lim)) == 64)


def test_weight_svd_takes_the_leading_left_singular_vectors():
    """A full-rank W_K = U diag(s) V^T with distinct singular values chosen
    here: the factors are U's first r columns, in order, up to sign."""
    rng = np.random.default_rng(9)
    d, D, r = 64, 96, 12
    U_all = _orthonormal(rng, d, d)
    V_all = _orthonormal(rng, D, d)
    s = np.geomspace(10.0, 0.1, d)
    W_K = (U_all * s) @ V_all.T
    U = O.weight_svd_factors(W_K, r)
    np.testing.assert_allclose(np.abs(U_all[:, :r].T @ U), np.eye(r), atol=1e-10)


def test_predicted_reduction_matches_heldout_measurement():
    """Remark 2 / Appendix C on synthetic data, where query and key tokens are
    independent by construction: the predicted relative score-MSE reduction
    1 - tail / sum sigma^2 matches the reduction measured on held-out pairs,
    up to sampling error (the moments are estimated on 512 tokens)."""
    spec = W.SPECS["single_head_d128"].with_(N=4096, Q=2048)
    inp = W.make_layer(spec)
    cal = O.saki_calibrate(inp["q_cal"][0], inp["k_cal"][0], 32)
    q, keys = inp["queries"][0, 0], inp["keys"][0, 0]
    s = O.exact_scores(q, keys)
    s_hat, z, b, c = O.index_scores(cal["B_q"], cal["B_k"], cal["mu"], q, keys)
    base = s - b[:, None]  # rank-0 map: only the mean term survives
    measured = 1.0 - np.mean((s - s_hat) ** 2) / np.mean(base ** 2)
    predicted = O.predicted_reduction(cal["sigma"], 32)
    assert abs(measured - predicted) < 0.01, (measured, predicted)


def test_ablation_predicted_vs_measured_across_heads():
    """Appendix C on the 32 heads of the LLaMA-shaped layer at r = 32.  Per
    head, the reduction measured on 16,384 independent held-out (query, key)
    pairs agrees with the population reduction of the same map (computed from
    the generator's exact moments) within 4.5 standard errors of the sample,
    which pins the measurement; the predicted reduction 1 - tail / sum sigma^2
    from the 512 calibration tokens then tracks the measured one across heads
    (Pearson above 0.98, median gap below 0.002)."""
    spec = W.SPECS["llama31_8b_layer"]
    r, n = 32, 16384
    wq, wk = W.weights(spec)
    lam = W.latent_std(spec) ** 2
    xc = W.tokens(spec, "calib", spec.T)
    q_cal = W._project(xc, wq)
    k_cal = W._project(xc, wk)
    xq = W._project(W.tokens(spec, "queries", n), wq)   # independent streams: q_i and k_i
    xk = W._project(W.tokens(spec, "keys", n), wk)      # come from different tokens
    pred, meas = [], []
    for h in range(spec.H_q):
        g = h // (spec.H_q // spec.H_kv)
        cal = O.saki_calibrate(q_cal[h], k_cal[g], r)
        m, se = O.measured_reduction(xq[h], xk[g], cal["M"], cal["mu"])
        pop = O.population_reduction(cal["M"], cal["mu"], (wq[h] * lam) @ wq[h].T,
                                     (wk[g] * lam) @ wk[g].T)
        assert abs(m - pop) <= 4.5 * se, (h, m, pop, se)
        pred.append(O.predicted_reduction(cal["sigma"], r))
        meas.append(m)
    pred, meas = np.array(pred), np.array(meas)
    assert np.corrcoef(pred, meas)[0, 1] > 0.98
    assert np.median(np.abs(pred - meas)) < 0.002


def test_measured_reduction_special_cases():
    """M = I removes every error (reduction 1); M = 0 removes none (0); for
    causal pairs the sums run over j <= q_pos[i] only; population_reduction
    of the rank-d map is 1."""
    rng = np.random.default_rng(2)
    q = rng.standard_normal((50, 6))
    k = rng.standard_normal((50, 6)) + 0.3
    mu = k.mean(0)
    assert O.measured_reduction(q, k, np.eye(6), mu)[0] == 1.0
    assert abs(O.measured_reduction(q, k, np.zeros((6, 6)), mu)[0]) < 1e-15
    M = np.diag([1.0, 1.0, 0.5, 0.0, 0.0, 0.0])
    pos = np.arange(50) // 2
    kc = k - mu
    num = sum((q[i] @ (kc[j] - M @ kc[j])) ** 2 for i in range(50) for j in range(pos[i] + 1))
    den = sum((q[i] @ kc[j]) ** 2 for i in range(50) for j in range(pos[i] + 1))
    assert abs(O.measured_reduction(q, k, M, mu, q_pos=pos)[0] - (1 - num / den)) < 1e-12
    Sq, Sk = _spd(rng, 6), _spd(rng, 6)
    assert abs(O.population_reduction(np.eye(6), mu, Sq, Sk) - 1.0) < 1e-15


def _rows(S):
    """2d rows whose (1/T) sum x x^T is exactly S (zero mean)."""
    d = S.shape[0]
    L = np.linalg.cholesky(S)
    return np.concatenate([np.sqrt(d) * L.T, -np.sqrt(d) * L.T])


@pytest.mark.parametrize("seed", [0, 1])
def test_shared_group_map_minimises_the_group_loss(seed):
    """The GQA-shared map (pooled query moment) against the summed per-head
    objective of Eq. 2: it equals G times the pooled tail energy (linearity of
    the loss in Sigma_q), and no other rank-r map -- each head's own optimum,
    key PCA, random maps -- does better on the group."""
    rng = np.random.default_rng(seed)
    G, d, r = 3, 12, 3
    Sqs = [_spd(rng, d, 50.0) for _ in range(G)]
    Sk = _spd(rng, d, 50.0)
    k = _rows(Sk)
    q = np.stack([_rows(S) for S in Sqs])
    sh = O.saki_calibrate_shared(q, k, r)
    halves = [O.clamped_roots(S)[0] for S in Sqs]
    sk_half = O.clamped_roots(Sk)[0]

    def group_loss(P):
        return sum(O.score_loss(P, hq, sk_half) for hq in halves)

    Lg = group_loss(sh["M"])
    assert abs(Lg - G * sh["tail"]) <= 1e-10 * G * float(np.sum(sh["sigma"] ** 2))
    for h in range(G):
        own = O.saki_calibrate(q[h], k, r)
        assert Lg <= group_loss(own["M"]) + 1e-12
    V = O.key_pca_factors(Sk, r)
    assert Lg <= group_loss(V @ V.T) + 1e-12
    for _ in range(300):
        P = rng.standard_normal((d, r)) @ rng.standard_normal((r, d))
        assert Lg <= group_loss(P) + 1e-12


def test_shared_map_special_cases():
    """One head per group, or identical heads: the shared map is the
    per-head map."""
    rng = np.random.default_rng(5)
    d, r = 10, 4
    Sq, Sk = _spd(rng, d, 20.0), _spd(rng, d, 20.0)
    q, k = _rows(Sq), _rows(Sk)
    own = O.saki_calibrate(q, k, r)
    np.testing.assert_allclose(O.saki_calibrate_shared(q[None], k, r)["M"], own["M"], atol=1e-12)
    np.testing.assert_allclose(O.saki_calibrate_shared(np.stack([q, q, q]), k, r)["M"], own["M"],
                               atol=1e-12)


def _projector(Q):
    return Q @ Q.T


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_sap_variants_are_the_stated_projectors(seed):
    """SAP-map and SAP-svd (Sec. 6) are rank-r orthogonal projectors: SAP-map
    onto the range of M_r (found here from an SVD of M_r itself), SAP-svd the
    rank-r orthogonal projector that keeps the most of C (Ky Fan: ||C P||_F^2
    reaches the sum of the r largest squared singular values, and random
    rank-r projectors stay below it).  Neither beats Proposition 1's optimum."""
    rng = np.random.default_rng(seed)
    d, r = 16, 4
    cal = _calib_from_moments(_spd(rng, d, 1e2), _spd(rng, d, 1e2), r)
    Lopt = O.score_loss(cal["M"], cal["Sq_half"], cal["Sk_half"])
    for kind in ("map", "svd"):
        Q = O.sap_factors(cal, r, kind)
        P = _projector(Q)
        np.testing.assert_allclose(Q.T @ Q, np.eye(r), atol=1e-12)
        np.testing.assert_allclose(P, P.T, atol=1e-12)
        np.testing.assert_allclose(P @ P, P, atol=1e-12)
        assert abs(np.trace(P) - r) < 1e-10
        assert Lopt <= O.score_loss(P, cal["Sq_half"], cal["Sk_half"]) + 1e-12
    Um, _, _ = np.linalg.svd(cal["M"])
    np.testing.assert_allclose(_projector(O.sap_factors(cal, r, "map")),
                               _projector(Um[:, :r]), atol=1e-9)
    C = cal["Sq_half"] @ cal["Sk_half"]
    sig = np.linalg.svd(C, compute_uv=False)
    kept = np.sum((C @ _projector(O.sap_factors(cal, r, "svd"))) ** 2)
    assert abs(kept - np.sum(sig[:r] ** 2)) <= 1e-10 * np.sum(sig ** 2)
    for _ in range(300):
        Qr, _ = np.linalg.qr(rng.standard_normal((d, r)))
        assert np.sum((C @ _projector(Qr)) ** 2) <= kept + 1e-10


def test_sap_variants_special_cases():
    """Sigma_q = I: both spans are the top-r key eigenvectors (key PCA);
    Sigma_k = I: both are query PCA; r = d: the identity."""
    rng = np.random.default_rng(5)
    d, r = 12, 5
    Sk = _spd(rng, d, 50.0)
    cal = _calib_from_moments(np.eye(d), Sk, r)
    w, V = np.linalg.eigh(Sk)
    Pk = _projector(V[:, np.argsort(-w)[:r]])
    for kind in ("map", "svd"):
        np.testing.assert_allclose(_projector(O.sap_factors(cal, r, kind)), Pk, atol=1e-10)
    Sq = _spd(rng, d, 50.0)
    cal = _calib_from_moments(Sq, np.eye(d), r)
    w, U = np.linalg.eigh(Sq)
    Pq = _projector(U[:, np.argsort(-w)[:r]])
    for kind in ("map", "svd"):
        np.testing.assert_allclose(_projector(O.sap_factors(cal, r, kind)), Pq, atol=1e-10)
    cal = _calib_from_moments(_spd(rng, d), _spd(rng, d), d)
    for kind in ("map", "svd"):
        np.testing.assert_allclose(_projector(O.sap_factors(cal, d, kind)), np.eye(d), atol=1e-10)


@pytest.mark.parametrize("layer", [0, 1])
def test_sap_losses_on_the_generator(layer):
    """On the single-head generator the exact optimum has the lowest loss
    (Proposition 1); the order among the span variants and PCA is what Sec. 7
    reports for real heads (weighted span < raw span, raw span close to PCA),
    checked here only where it is a theorem."""
    spec = W.SPECS["single_head_d128"]
    inp = W.make_layer(spec, layer=layer)
    cal = O.saki_calibrate(inp["q_cal"][0], inp["k_cal"][0], 32)
    L = {"opt": O.score_loss(cal["M"], cal["Sq_half"], cal["Sk_half"])}
    for kind in ("map", "svd"):
        L[kind] = O.score_loss(_projector(O.sap_factors(cal, 32, kind)), cal["Sq_half"],
                               cal["Sk_half"])
    assert L["opt"] <= L["map"] and L["opt"] <= L["svd"]
