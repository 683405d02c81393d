"""Pins of the fp64 oracle against facts the paper and the mathematics fix.

None of these re-types the oracle's formulas: each checks a worked example with
an exact rational answer, a closed form, an identity computed through a
different library routine, an invariance, or a brute-force count.
"""

import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.linalg
import scipy.stats

from jacap_synth import make_case
from oracle import jacap_oracle as jo
from oracle import theory

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def frac(xs):
    return np.array([float(Fraction(x)) for x in xs])


def rel_close(a, b, tol):
    a, b = np.asarray(a, float), np.asarray(b, float)
    scale = np.maximum(np.abs(b), 1e-300)
    return np.all(np.abs(a - b) <= tol * scale + 1e-300)


def rand_unit(seed, n=40, d=6, N=12, spread=1.0):
    rng = np.random.default_rng(seed)
    Q = rng.normal(size=(N, d)) + rng.normal(size=d)
    K = spread * rng.normal(size=(n, d))
    V = rng.normal(size=(n, d))
    return Q, K, V


# ---------------------------------------------------------------------------
# Worked examples (tests/golden): exact rational answers
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as f:
        return {c["name"]: c for c in json.load(f)["cases"]}


def test_worked_uniform_attention(golden):
    c = golden["uniform_attention_d2"]
    Q, K, V = (np.array(c[k]) for k in ("queries", "keys", "values"))
    for ridge, want in c["expected"]["scores"].items():
        out = jo.score_unit(Q, K, V, tau=c["tau"], ridge=float(Fraction(ridge)))
        assert rel_close(out["alpha"], frac(c["expected"]["alpha"]), 1e-14)
        assert rel_close(out["w"], frac(c["expected"]["w"]), 1e-14)
        assert np.allclose(out["scores"], frac(want), rtol=1e-13, atol=1e-15), ridge
    out = jo.evict_unit(Q, K, V, c["expected"]["select_budget"], tau=c["tau"],
                        ridge=float(Fraction(c["expected"]["select_ridge"])))
    assert out["idx"].tolist() == c["expected"]["select_idx"]
    assert np.array_equal(out["k_out"], K[c["expected"]["select_idx"]])
    assert np.array_equal(out["v_out"], V[c["expected"]["select_idx"]])


def test_worked_two_thirds(golden):
    c = golden["two_tokens_two_thirds_d4"]
    Q, K = np.array(c["queries"]), np.array(c["keys"])
    e = c["expected"]
    out = jo.score_unit(Q, K, np.array(c["values_orthogonal"]), tau=c["tau"], ridge=1.0)
    assert rel_close(out["alpha"], frac(e["alpha"]), 1e-14)
    assert rel_close(out["w"], frac(e["w"]), 1e-13)
    assert rel_close(out["scores"], frac(e["scores_orthogonal_ridge1"]), 1e-13)
    out = jo.score_unit(Q, K, np.array(c["values_coupled"]), tau=c["tau"], ridge=1.0)
    assert rel_close(out["scores"], frac(e["scores_coupled_ridge1"]), 1e-13)


def test_worked_full_vs_diag(golden):
    c = golden["full_vs_diag_covariance_d2"]
    Q, K, V = (np.array(c[k]) for k in ("queries", "keys", "values"))
    for mode in ("full", "diag"):
        e = c["expected"][mode]
        out = jo.score_unit(Q, K, V, tau=c["tau"], ridge=1.0, cov_mode=mode)
        assert np.allclose(out["kappa"], frac(e["kappa"]), rtol=1e-14, atol=1e-15)
        assert np.allclose(out["w"], frac(e["w"]), rtol=1e-14, atol=1e-17)
        assert np.allclose(out["scores"], frac(e["scores_ridge1"]), rtol=1e-13, atol=1e-16)


def test_centre_softmax_is_not_window_average(golden):
    """Z5: one softmax at mu_Q, not the mean of the per-query softmaxes."""
    c = golden["two_tokens_two_thirds_d4"]
    Q, K = np.array(c["queries"]), np.array(c["keys"])
    out = jo.score_unit(Q, K, np.array(c["values_orthogonal"]), tau=c["tau"])
    avg = np.mean([theory.softmax(K @ q / (c["tau"] * 2.0)) for q in Q], axis=0)
    assert abs(avg[0] - 2 / 3) > 1e-5
    assert abs(out["alpha"][0] - 2 / 3) < 1e-14


# ---------------------------------------------------------------------------
# P1 softmax, P2 softmax Jacobian, P3 Lemma 1 (App. A.1)
# ---------------------------------------------------------------------------

def test_p1_centre_softmax_sums_to_one():
    for seed in range(5):
        Q, K, V = rand_unit(seed, n=300, d=16, spread=3.0)
        out = jo.score_unit(Q, K, V, tau=0.5)
        a = out["alpha"]
        assert abs(a.sum() - 1.0) < 1e-14
        assert np.all(a > 0) and np.all(a < 1)
        assert np.allclose(out["one_minus_alpha"], 1.0 - a, atol=1e-15)


def test_p2_softmax_jacobian_matches_finite_differences():
    rng = np.random.default_rng(1)
    s = rng.normal(size=7)
    h = 1e-6
    fd = np.stack([(theory.softmax(s + h * e) - theory.softmax(s - h * e)) / (2 * h)
                   for e in np.eye(7)], axis=1)
    assert np.allclose(theory.softmax_jacobian(theory.softmax(s)), fd, atol=1e-9)


def test_p3_lemma1_jacobian_matches_finite_differences():
    rng = np.random.default_rng(2)
    m, dk, do = 9, 5, 4
    K_C, U_C, mu = rng.normal(size=(m, dk)), rng.normal(size=(m, do)), rng.normal(size=dk)
    h = 1e-6
    fd = np.stack([(theory.attention_map(mu + h * e, K_C, U_C)
                    - theory.attention_map(mu - h * e, K_C, U_C)) / (2 * h)
                   for e in np.eye(dk)], axis=1)
    J = theory.lemma1_jacobian(K_C, U_C, mu)
    assert J.shape == (do, dk)
    assert np.allclose(J, fd, atol=1e-9)
    # first-order expansion (Eq. 5): the residual shrinks quadratically
    dq = rng.normal(size=dk)
    res = [np.linalg.norm(theory.attention_map(mu + t * dq, K_C, U_C)
                          - theory.attention_map(mu, K_C, U_C) - J @ (t * dq)) for t in (1e-2, 1e-3)]
    assert 50 < res[0] / res[1] < 200


def test_theorem1_is_gaussian_mutual_information():
    """Eq. 7 equals H(Y) - H(Y|q) of the linearised channel (App. A.1),
    computed with scipy's Gaussian entropy."""
    rng = np.random.default_rng(3)
    K, U = rng.normal(size=(8, 4)), rng.normal(size=(8, 3))
    mu = rng.normal(size=4)
    Lam = np.diag(rng.uniform(0.5, 2.0, size=4))
    C = [0, 2, 3, 7]
    J = theory.lemma1_jacobian(K[C], U[C], mu)
    s2 = 0.3
    hy = scipy.stats.multivariate_normal(cov=J @ Lam @ J.T + s2 * np.eye(3)).entropy()
    hyq = scipy.stats.multivariate_normal(cov=s2 * np.eye(3)).entropy()
    assert abs(theory.jacobian_capacity(C, K, U, mu, Lam, noise_var=s2) - (hy - hyq)) < 1e-12


def test_p12_linear_special_case():
    """With S_C replaced by sqrt(d_k) I the Jacobian channel is the linear
    (CapKV) channel U_C K_C (App. A.2, last paragraph); checked through
    Sylvester's determinant identity on the d_k side."""
    rng = np.random.default_rng(4)
    K, U = rng.normal(size=(10, 5)), rng.normal(size=(10, 3))
    lam = rng.uniform(0.2, 1.5, size=5)
    C = [1, 4, 5, 9]
    J = U[C].T @ (math.sqrt(5) * np.eye(4)) @ K[C] / math.sqrt(5)
    lhs = theory.gaussian_capacity(J, lam, 0.7)
    R = np.diag(np.sqrt(lam))
    rhs = 0.5 * np.linalg.slogdet(np.eye(5) + R @ J.T @ J @ R / 0.7)[1]
    assert abs(lhs - rhs) < 1e-12
    assert abs(theory.linear_capacity(C, K, U, lam, 0.7) - rhs) < 1e-12


# ---------------------------------------------------------------------------
# P4 sensitivity factor (App. A.2)
# ---------------------------------------------------------------------------

def test_p4_sensitivity_peak_and_saturation():
    a = np.linspace(0.0, 1.0, 2001)
    w = jo.importance_weights(a, 1.0 - a, np.ones_like(a), 1)   # = rho^2
    assert np.argmax(w) == 1000 and abs(w[1000] - 1 / 16) < 1e-15
    assert np.allclose(w, w[::-1], atol=1e-15)
    assert w[0] == 0.0 and w[-1] == 0.0
    # a planted key that takes almost all attention gets (almost) no weight
    rng = np.random.default_rng(5)
    n, d = 64, 8
    Q = rng.normal(size=(16, d)) * 0.3 + np.eye(d)[0]
    K = rng.normal(size=(n, d)) * 0.1
    K[7] = 400.0 * np.eye(d)[0]
    V = rng.normal(size=(n, d))
    out = jo.score_unit(Q, K, V, tau=1.0, ridge=1e-3)
    a7, r7 = out["alpha"][7], out["one_minus_alpha"][7]
    assert a7 > 0.999
    # the other tokens' mass is tiny but not zero, and the key's sensitivity
    # rho = alpha (1 - alpha) -- hence its weight -- is a vanishing fraction of
    # what the same key would get at peak sensitivity (rho = 1/4 at alpha = 1/2)
    assert 0.0 < r7 < 1e-3
    assert a7 * r7 < 1e-3 * 0.25
    assert out["w"][7] < 1e-6 * out["kappa"][7] / (16 * d)


# ---------------------------------------------------------------------------
# P5 ridge leverage closed forms, via library eigvalsh / QR
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("ridge", [0.0, 1e-3, 1.0])
def test_p5_leverage_closed_forms(ridge):
    Q, K, V = rand_unit(11, n=80, d=6, spread=2.0)
    out = jo.score_unit(Q, K, V, tau=1.0, ridge=ridge)
    w, s = out["w"], out["scores"]
    M = sum(w[i] * np.outer(V[i], V[i]) for i in range(len(w)))
    ev = scipy.linalg.eigvalsh(M)
    if ridge > 0:
        assert np.all(s >= 0) and np.all(s < 1)
        assert abs(s.sum() - np.sum(ev / (ridge + ev))) < 1e-12
    else:
        assert np.all(s >= -1e-15) and np.all(s <= 1 + 1e-12)
        assert abs(s.sum() - np.linalg.matrix_rank(M)) < 1e-10
    # ridge leverage = squared row norms of the orthonormal factor of the
    # augmented matrix [sqrt(W) V; sqrt(ridge) I] (textbook identity)
    X = np.sqrt(w)[:, None] * V
    if ridge > 0:
        X = np.vstack([X, math.sqrt(ridge) * np.eye(V.shape[1])])
    Qf, _ = np.linalg.qr(X)
    lev = (Qf[:len(w)] ** 2).sum(axis=1)
    assert np.allclose(s, lev, rtol=1e-9, atol=1e-14)


def test_p5_eigh_cross_check():
    Q, K, V = rand_unit(12, n=200, d=8, spread=2.0)
    for ridge in (0.0, 1 / 8, 1.0):
        out = jo.score_unit(Q, K, V, tau=10.0, ridge=ridge)
        alt = jo.leverage_scores_eigh(V, out["w"], out["A"])
        assert np.allclose(out["scores"], alt, rtol=1e-10, atol=0)


# ---------------------------------------------------------------------------
# P6 leave-one-out identity (matrix determinant lemma, App. B.1)
# ---------------------------------------------------------------------------

def test_p6_leave_one_out_logdet():
    Q, K, V = rand_unit(13, n=30, d=5, spread=2.0)
    out = jo.score_unit(Q, K, V, tau=1.0, ridge=0.05)
    A, w, s = out["A"], out["w"], out["scores"]
    full = np.linalg.slogdet(A)[1]
    for i in range(30):
        loo = np.linalg.slogdet(A - w[i] * np.outer(V[i], V[i]))[1]
        assert abs((full - loo) - (-math.log1p(-s[i]))) < 1e-10
    # so ranking by score is exactly ranking by each token's log-det loss
    loss = np.array([full - np.linalg.slogdet(A - w[i] * np.outer(V[i], V[i]))[1] for i in range(30)])
    assert list(np.argsort(-loss, kind="stable")[:8]) == list(np.argsort(-s, kind="stable")[:8])


# ---------------------------------------------------------------------------
# P7 orthogonal special case and P11 brute force (objective (ii), App. B.1)
# ---------------------------------------------------------------------------

def test_p7_orthogonal_values_select_the_optimum():
    rng = np.random.default_rng(14)
    for trial in range(6):
        n, d, k = 7, 8, 3
        R, _ = np.linalg.qr(rng.normal(size=(d, d)))
        V = R[:n] * rng.uniform(0.2, 3.0, size=(n, 1))     # orthogonal rows
        Q = rng.normal(size=(10, d)) + rng.normal(size=d)
        K = rng.normal(size=(n, d)) * 2
        out = jo.evict_unit(Q, K, V, k, tau=1.0, ridge=0.01)
        best, val, _ = theory.brute_force_best(
            lambda C: theory.diag_objective(C, out["w"], V, 0.01), n, k)
        assert sorted(best) == out["idx"].tolist()


def test_p11_brute_force_small(capsys):
    rng = np.random.default_rng(15)
    ratios, pct = [], []
    for trial in range(5):
        n, d, k = 12, 4, 4
        Q = rng.normal(size=(8, d)) * 0.5 + rng.normal(size=d)
        K, V = rng.normal(size=(n, d)) * 2, rng.normal(size=(n, d))
        out = jo.evict_unit(Q, K, V, k, tau=1.0, ridge=0.1)
        obj = lambda C: theory.diag_objective(C, out["w"], V, 0.1)
        best, val, allv = theory.brute_force_best(obj, n, k)
        mine = obj(out["idx"])
        assert val >= mine - 1e-12
        ratios.append(mine / val)
        pct.append((allv <= mine + 1e-15).mean())
        # Theorem 1 objective (i), literal tau=1 and configured tau: report only
        mu, lam = jo.query_statistics(Q)
        for tau in (1.0, 10.0):
            obj1 = lambda C: theory.jacobian_capacity(C, K, V, mu, lam, 0.1, tau)
            b1, v1, _ = theory.brute_force_best(obj1, n, k)
            assert v1 >= obj1(out["idx"]) - 1e-12
    with capsys.disabled():
        print(f"\n[P11] F(C_jacap)/F(C*) objective (ii): {np.round(ratios, 4)}; "
              f"percentile: {np.round(pct, 3)}")


def test_greedy_runs_and_is_feasible():
    rng = np.random.default_rng(16)
    n, d, k = 10, 3, 3
    V, w = rng.normal(size=(n, d)), rng.uniform(0.01, 1, size=n)
    obj = lambda C: theory.diag_objective(C, w, V, 0.5)
    g = theory.greedy(obj, n, k)
    _, best, _ = theory.brute_force_best(obj, n, k)
    assert len(set(g)) == k and obj(g) <= best + 1e-12
    # submodular log-det: greedy reaches at least (1 - 1/e) of the optimum
    assert obj(g) >= (1 - 1 / math.e) * best


# ---------------------------------------------------------------------------
# P8 invariances
# ---------------------------------------------------------------------------

def _rot(d, seed):
    R, _ = np.linalg.qr(np.random.default_rng(seed).normal(size=(d, d)))
    return R


@pytest.mark.parametrize("mode", ["diag", "full"])
@pytest.mark.parametrize("ridge", [0.0, 1 / 6, 1.0])
def test_p8_value_rotation_invariance(mode, ridge):
    Q, K, V = rand_unit(21, n=60, d=6, spread=2.0)
    a = jo.score_unit(Q, K, V, tau=1.0, ridge=ridge, cov_mode=mode)["scores"]
    b = jo.score_unit(Q, K, V @ _rot(6, 1), tau=1.0, ridge=ridge, cov_mode=mode)["scores"]
    assert np.allclose(a, b, rtol=1e-9, atol=1e-18)


def test_p8_query_key_rotation():
    Q, K, V = rand_unit(22, n=60, d=6, spread=2.0)
    R = _rot(6, 2)
    full = jo.score_unit(Q, K, V, tau=1.0, cov_mode="full")["scores"]
    full_r = jo.score_unit(Q @ R, K @ R, V, tau=1.0, cov_mode="full")["scores"]
    assert np.allclose(full, full_r, rtol=1e-9)
    # DIAG: invariant under signed permutations only
    P = np.eye(6)[[3, 0, 5, 1, 4, 2]] * np.array([1, -1, 1, 1, -1, -1])[:, None]
    diag = jo.score_unit(Q, K, V, tau=1.0)["scores"]
    assert np.allclose(diag, jo.score_unit(Q @ P, K @ P, V, tau=1.0)["scores"], rtol=1e-12)
    assert not np.allclose(diag, jo.score_unit(Q @ R, K @ R, V, tau=1.0)["scores"], rtol=1e-6)


def test_p8_permutations_and_scaling():
    Q, K, V = rand_unit(23, n=50, d=5, spread=2.0)
    base = jo.score_unit(Q, K, V, tau=2.0, ridge=0.3)["scores"]
    perm = np.random.default_rng(3).permutation(50)
    assert np.allclose(jo.score_unit(Q, K[perm], V[perm], tau=2.0, ridge=0.3)["scores"],
                       base[perm], rtol=1e-12)
    qperm = np.random.default_rng(4).permutation(len(Q))
    assert np.allclose(jo.score_unit(Q[qperm], K, V, tau=2.0, ridge=0.3)["scores"], base, rtol=1e-12)
    s0 = jo.score_unit(Q, K, V, tau=2.0, ridge=0.0)["scores"]
    assert np.allclose(jo.score_unit(Q, K, 7.5 * V, tau=2.0, ridge=0.0)["scores"], s0, rtol=1e-10)


def test_stats_input_form():
    """Algorithm 1 with its literal inputs (mu_Q, Lambda_Q). A window of 2d
    queries mu +- sqrt(d lambda_c) e_c has exactly mean mu and 1/N covariance
    diag(lambda), so scoring it must equal scoring (mu, lambda) directly, in
    both covariance modes; FULL with a diagonal Lambda equals DIAG; a rotation
    of K with mu -> R^T mu, Lambda -> R^T Lambda R leaves FULL scores
    unchanged; Lambda = 0 gives zero scores."""
    rng = np.random.default_rng(41)
    n, d = 70, 6
    K = rng.normal(size=(n, d)) * 1.5
    V = rng.normal(size=(n, d))
    mu = rng.normal(size=d)
    lam = rng.uniform(0.1, 2.0, size=d)
    window = np.concatenate([mu + np.sqrt(d * lam)[:, None] * np.eye(d),
                             mu - np.sqrt(d * lam)[:, None] * np.eye(d)])
    direct = jo.score_unit_from_stats(mu, lam, K, V, tau=1.5, ridge=0.4)["scores"]
    assert np.allclose(jo.score_unit(window, K, V, tau=1.5, ridge=0.4)["scores"], direct,
                       rtol=1e-12)
    assert np.allclose(jo.score_unit(window, K, V, tau=1.5, ridge=0.4, cov_mode="full")["scores"],
                       direct, rtol=1e-12)
    assert np.allclose(jo.score_unit_from_stats(mu, np.diag(lam), K, V, tau=1.5,
                                                ridge=0.4)["scores"], direct, rtol=1e-12)
    B = rng.normal(size=(d, d))
    Lam = B @ B.T / d
    R = _rot(d, 5)
    full = jo.score_unit_from_stats(mu, Lam, K, V, tau=1.5, ridge=0.4)["scores"]
    rot = jo.score_unit_from_stats(R.T @ mu, R.T @ Lam @ R, K @ R, V, tau=1.5, ridge=0.4)["scores"]
    assert np.allclose(full, rot, rtol=1e-10)
    assert not np.allclose(full, direct, rtol=1e-3)
    assert np.all(jo.score_unit_from_stats(mu, np.zeros(d), K, V)["scores"] == 0.0)


# ---------------------------------------------------------------------------
# P9 Algorithm 1 literal form, P10 large-ridge limit, FULL kappa
# ---------------------------------------------------------------------------

def test_p9_algorithm1_literal_equals_ridge_one_over_d():
    Q, K, V = rand_unit(31, n=40, d=6, spread=2.0)
    n, d = K.shape
    mu = Q.mean(axis=0)
    lam = ((Q - mu) ** 2).mean(axis=0)
    tau = 10.0
    logits = [sum(K[i, c] * mu[c] for c in range(d)) / (tau * math.sqrt(d)) for i in range(n)]
    mx = max(logits)
    ex = [math.exp(x - mx) for x in logits]
    a = [x / sum(ex) for x in ex]
    s = [a[i] ** 2 * (1 - a[i]) ** 2 * sum(lam[c] * K[i, c] ** 2 for c in range(d)) for i in range(n)]
    A = np.eye(d)
    for i in range(n):
        A += s[i] * np.outer(V[i], V[i])
    Ainv = np.linalg.inv(A)
    lit = np.array([s[i] * V[i] @ Ainv @ V[i] for i in range(n)])
    out = jo.score_unit(Q, K, V, tau=tau, ridge=1.0 / d)
    assert np.allclose(out["scores"], lit, rtol=1e-11)


def test_p10_large_ridge_limit():
    Q, K, V = rand_unit(32, n=40, d=6, spread=2.0)
    big = 1e9
    out = jo.score_unit(Q, K, V, tau=1.0, ridge=big)
    lim = out["w"] * (V * V).sum(axis=1)
    assert np.allclose(big * out["scores"], lim, rtol=1e-6)


def test_full_kappa_is_variance_of_window_logits():
    rng = np.random.default_rng(33)
    Q, K = rng.normal(size=(20, 5)) + 1.0, rng.normal(size=(30, 5))
    mu, Lam = jo.query_statistics(Q, "full")
    kap = jo.query_response(K, Lam)
    direct = np.array([np.var([(q - mu) @ k for q in Q]) for k in K])   # 1/N variance
    assert np.allclose(kap, direct, rtol=1e-12)
    np_var = np.array([np.var(Q @ k) for k in K])                       # Var(q.k)
    assert np.allclose(kap, np_var, rtol=1e-10)


# ---------------------------------------------------------------------------
# Degenerate cases (Z12) and selection semantics (Z7, Z8)
# ---------------------------------------------------------------------------

def test_single_window_query_gives_zero_scores():
    _, K, V = rand_unit(41, n=20, d=4)
    q = np.ones((1, 4))
    out = jo.evict_unit(q, K, V, 5)
    assert np.all(out["scores"] == 0.0)
    assert out["idx"].tolist() == [0, 1, 2, 3, 4]


def test_single_token_and_empty():
    Q, K, V = rand_unit(42, n=1, d=4)
    out = jo.evict_unit(Q, K, V, 3)
    assert out["alpha"][0] == 1.0 and out["scores"][0] == 0.0 and out["idx"].tolist() == [0]
    out = jo.evict_unit(Q, K[:0], V[:0], 3)
    assert out["idx"].tolist() == []


def test_singular_ridge_zero_uses_pseudo_inverse():
    Q, K, V = rand_unit(43, n=3, d=6)           # rank 3 < d at ridge 0
    out = jo.score_unit(Q, K, V, tau=1.0, ridge=0.0)
    assert out["singular"]
    assert np.allclose(out["scores"], 1.0, atol=1e-8)   # n <= d: every token is a pivot


def _rank_select(s, k):
    """Brute-force definition: i is kept iff fewer than k tokens beat it."""
    s = np.asarray(s, np.float32).astype(float)
    n = len(s)

    def beats(j, i):
        if np.isnan(s[j]) and np.isnan(s[i]):
            return j < i
        if np.isnan(s[j]):
            return False
        if np.isnan(s[i]):
            return True
        return s[j] > s[i] or (s[j] == s[i] and j < i)
    return [i for i in range(n) if sum(beats(j, i) for j in range(n) if j != i) < min(k, n)]


def test_select_matches_rank_definition():
    rng = np.random.default_rng(44)
    for trial in range(40):
        n = int(rng.integers(0, 40))
        s = rng.integers(0, 5, size=n).astype(np.float32) * 0.25
        s[rng.random(n) < 0.1] = np.nan
        s[rng.random(n) < 0.1] = -0.0
        k = int(rng.integers(0, n + 3))
        got = jo.select_top(s, k)
        assert got.tolist() == _rank_select(s, k)
        assert np.all(np.diff(got) > 0)


def test_select_decides_on_fp32():
    s64 = np.array([1.0, 1.0 + 1e-12, 0.5])          # equal after fp32 rounding
    assert jo.select_top(jo.to_fp32(s64), 1).tolist() == [0]


# ---------------------------------------------------------------------------
# Output-projection variant (u_i = W_O v_i)
# ---------------------------------------------------------------------------

def test_wo_group_projection_matches_full_output_projection():
    """Sec. 3.1 (Preliminary): the layer output is W_O applied to the concatenated per-head
    outputs. When the G heads of a KV group share one attention output y_h,
    that equals sum_h W~_h y_h with W~_h = group_output_projection(...)."""
    rng = np.random.default_rng(11)
    d, H, G, dm = 4, 3, 2, 9
    w_o = rng.normal(size=(dm, H * G * d))
    ys = rng.normal(size=(H, d))
    concat = np.concatenate([ys[h] for h in range(H) for _ in range(G)])
    full = w_o @ concat
    via_groups = sum(jo.group_output_projection(w_o, h, G, d) @ ys[h] for h in range(H))
    np.testing.assert_allclose(via_groups, full, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_wo_push_through_equals_literal_output_space_scores(seed):
    """Eq. 9 / Eq. 10 evaluated literally in output space (u_i = W~ v_i,
    A = I + sum_j w_j u_j u_j^T of size d_model) equal the d x d ridge-matrix
    form with R = (W~^T W~)^{-1}."""
    rng = np.random.default_rng(100 + seed)
    d, G, w_len, n, dm = 6, 2, 5, 17, 23
    q = rng.normal(size=(G, w_len, d)) + rng.normal(size=d)
    K = rng.normal(size=(n, d))
    V = rng.normal(size=(n, d))
    w_tilde = rng.normal(size=(dm, d)) / np.sqrt(dm)
    R = jo.output_ridge_matrix(w_tilde)
    o = jo.score_unit(q, K, V, tau=1.0, ridge=R)
    w = o["w"] * 1e3          # larger weights make the capacity term matter
    U = V @ w_tilde.T         # rows u_i = W~ v_i
    A_out = np.eye(dm) + U.T @ (w[:, None] * U)
    lit = w * np.einsum("ij,ij->i", U, np.linalg.solve(A_out, U.T).T)
    A_d = jo.capacity_matrix(V, w, R)
    got, singular = jo.leverage_scores(V, w, A_d)
    assert not singular
    np.testing.assert_allclose(got, lit, rtol=1e-10, atol=0)


def test_ridge_matrix_lambda_identity_equals_scalar_ridge():
    """R = ridge * I reproduces the scalar-ridge scores."""
    case = make_case("tiny", seq_lens=[96], head_dim=64)
    q, k, v = case.unit_arrays(0, 0, 0)
    for lam in (1.0, 0.25):
        a = jo.score_unit(q, k, v, ridge=lam)["scores"]
        b = jo.score_unit(q, k, v, ridge=lam * np.eye(64))["scores"]
        np.testing.assert_allclose(b, a, rtol=1e-12, atol=0)


# ---------------------------------------------------------------------------
# Per-query-head GQA and the protected tail
# ---------------------------------------------------------------------------

def test_per_head_with_one_head_equals_pooled():
    case = make_case("tiny", seq_lens=[80])
    q, k, v = case.unit_arrays(0, 0, 0)
    a = jo.score_unit(q, k, v, ridge=0.5)["scores"]
    b = jo.score_unit_per_head(q, k, v, ridge=0.5)["scores"]
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("mode", [jo.DIAG, jo.FULL])
def test_per_head_identical_heads_equals_pooled(mode):
    """G copies of one head's window give the pooled sample the same mean and
    1/N covariance as the single head, so both readings coincide; a wrong
    normalisation of the pooled statistics (e.g. 1/(N-1)) breaks this."""
    rng = np.random.default_rng(5)
    d, w, n, G = 8, 6, 40, 3
    q1 = rng.normal(size=(1, w, d)) + rng.normal(size=d)
    qG = np.repeat(q1, G, axis=0)
    K = rng.normal(size=(n, d)) * 2
    V = rng.normal(size=(n, d))
    a = jo.score_unit(qG, K, V, tau=1.0, ridge=0.1, cov_mode=mode)["scores"]
    b = jo.score_unit_per_head(qG, K, V, tau=1.0, ridge=0.1, cov_mode=mode)["scores"]
    np.testing.assert_allclose(b, a, rtol=1e-12, atol=0)


def test_per_head_is_mean_of_single_head_scores():
    rng = np.random.default_rng(6)
    d, w, n, G = 8, 5, 30, 4
    q = rng.normal(size=(G, w, d)) + rng.normal(size=d)
    K, V = rng.normal(size=(n, d)), rng.normal(size=(n, d))
    got = jo.score_unit_per_head(q, K, V, tau=1.0)["scores"]
    each = [jo.score_unit(q[g][None], K, V, tau=1.0)["scores"] for g in range(G)]
    np.testing.assert_allclose(got, np.mean(each, axis=0), rtol=1e-13, atol=0)


@pytest.mark.parametrize("n,budget,p", [(30, 10, 0), (30, 10, 4), (30, 10, 10), (30, 10, 25),
                                        (30, 40, 5), (12, 12, 3), (1, 1, 1)])
def test_protect_last_against_definition(n, budget, p):
    """Kept set = the last min(P, B, n) positions, plus the best of the earlier
    positions by (score desc, index asc) up to min(B, n) in total."""
    rng = np.random.default_rng(n * 100 + budget + p)
    s = rng.integers(0, 4, n).astype(np.float32)
    s[rng.random(n) < 0.2] = np.nan
    got = jo.select_top(s, budget, protect_last=p)
    b = min(budget, n)
    tail = min(p, b)
    keep = set(range(n - tail, n))
    def better(i, j):  # i ranks before j
        ki = -np.inf if np.isnan(s[i]) else s[i]
        kj = -np.inf if np.isnan(s[j]) else s[j]
        return ki > kj or (ki == kj and (i < j))
    head = [i for i in range(n - tail)]
    ranked = [i for i in head if sum(better(j, i) for j in head) < b - tail]
    keep |= set(ranked)
    assert list(got) == sorted(keep)
    assert len(got) == b


# ---------------------------------------------------------------------------
# Exact greedy log-det selection
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed", range(4))
def test_greedy_logdet_matches_brute_force_greedy(seed):
    """The rank-one-update greedy equals the plain greedy that re-evaluates
    log det for every candidate set (slogdet) at every step."""
    rng = np.random.default_rng(300 + seed)
    n, d, k, ridge = 11, 4, 6, 0.3
    U = rng.normal(size=(n, d))
    w = rng.uniform(0.1, 2.0, n)
    got = jo.greedy_logdet(U, w, ridge, k)
    obj = lambda C: jo.logdet_objective(U, w, ridge, C)
    want = theory.greedy(obj, n, k)
    assert sorted(got.tolist()) == want
    # every step's choice is the best marginal gain given the earlier picks
    for t in range(k):
        base = obj(got[:t])
        gains = [obj(list(got[:t]) + [i]) - base if i not in got[:t] else -np.inf for i in range(n)]
        assert got[t] == int(np.argmax(gains))


def test_greedy_first_pick_and_orthogonal_case():
    """First pick = argmax w_i ||u_i||^2; with orthogonal u_i the gains never
    interact, so greedy = TOP-B by w_i ||u_i||^2 (= Jacap's ranking, P7)."""
    rng = np.random.default_rng(9)
    d = 7
    U = np.eye(d) * rng.uniform(0.5, 2.0, d)[:, None]
    w = rng.uniform(0.1, 1.0, d)
    order = jo.greedy_logdet(U, w, 1.0, 4)
    x = w * (U * U).sum(axis=1)
    assert order[0] == int(np.argmax(x))
    assert sorted(order.tolist()) == sorted(np.argsort(-x)[:4].tolist())


@pytest.mark.parametrize("protect", [1, 3])
def test_greedy_protected_tail_is_forced_then_greedy(protect):
    """With a protected tail: the tail first, then the plain greedy (brute
    force over slogdet) over the earlier positions from that starting set."""
    rng = np.random.default_rng(40 + protect)
    n, d, k, ridge = 10, 3, 6, 0.5
    U = rng.normal(size=(n, d))
    w = rng.uniform(0.1, 2.0, n)
    got = jo.greedy_logdet(U, w, ridge, k, protect_last=protect)
    assert got[:protect].tolist() == list(range(n - protect, n))
    C = list(range(n - protect, n))
    for _ in range(k - protect):
        base = jo.logdet_objective(U, w, ridge, C)
        gains = [jo.logdet_objective(U, w, ridge, C + [i]) - base if i not in C and i < n - protect
                 else -np.inf for i in range(n)]
        C.append(int(np.argmax(gains)))
    assert got.tolist() == C


def test_greedy_replay_and_determinant_lemma():
    """Replay of the greedy order: every chosen gain is the best one, and
    d log(ridge) + sum log(1 + gain_t) is the log det of the chosen set (matrix
    determinant lemma); a non-greedy order is caught by the replay."""
    rng = np.random.default_rng(77)
    n, d, k, ridge = 40, 5, 12, 0.25
    U = rng.normal(size=(n, d))
    w = rng.uniform(0.05, 1.5, n)
    order = jo.greedy_logdet(U, w, ridge, k)
    chosen, best = jo.greedy_replay(U, w, ridge, order)
    np.testing.assert_allclose(chosen, best, rtol=1e-12)
    total = d * np.log(ridge) + np.log1p(chosen).sum()
    assert abs(total - jo.logdet_objective(U, w, ridge, order)) < 1e-10
    # swap the step-3 pick for the runner-up: the replay must flag that step
    bad = list(order)
    alt = [i for i in np.argsort(-w * (U * U).sum(1)) if i not in bad[:3]][1]
    bad[3] = int(alt) if alt != order[3] else int([i for i in range(n) if i not in bad[:4]][0])
    ch2, be2 = jo.greedy_replay(U, w, ridge, bad[:4])
    assert ch2[3] < be2[3]


def test_other_token_mass_of_a_dominant_token():
    """1 - bar-alpha_i, the factor of the sensitivity rho_i of Eq. 8, is the
    softmax mass of the other tokens. For a token that holds nearly all of it
    (here 1 - bar-alpha ~ 1e-13) the oracle's value must match exact rational
    arithmetic on the same fp64 exponentials to fp64 precision; formed as
    Z - e_i it would be off by ~1e-3."""
    from fractions import Fraction
    rng = np.random.default_rng(5)
    z = np.concatenate([rng.normal(10.0, 1.0, 12), [40.0], rng.normal(10.0, 1.0, 30)])
    alpha, one_minus = jo.centre_attention(z)
    e = np.exp(z - z.max())
    E = [Fraction(float(x)) for x in e]
    Zx = sum(E)
    assert one_minus[12] < 1e-11
    for i in (0, 5, 12, 42):
        exact_a = float(E[i] / Zx)
        exact_r = float((Zx - E[i]) / Zx)
        assert abs(alpha[i] - exact_a) <= 1e-14 * exact_a
        assert abs(one_minus[i] - exact_r) <= 1e-14 * exact_r
