"""Plain fp64 CPU oracle of Jacap scoring, top-B selection and KV compaction.

TEST INFRASTRUCTURE ONLY. Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import or run this module; the product path
(the HIP library and its Python binding) never does. It shares no code with
the HIP path.

It follows Algorithm 1 (Jacap) of Sec. 3.4 and the equations it is built from
(centre attention, Eq. 8 importance weight, Eq. 9 capacity matrix, Eq. 10
leverage score), step by step, in float64. Readings of points the paper leaves
open:

* ridge: A = ridge*I + sum_j w_j u_j u_j^T with w_j from Eq. 8. ridge=1 is
  Eq. 9; ridge=1/d reproduces Algorithm 1 literally (it drops the 1/d_k of
  Eq. 8); ridge=0 is the plain statistical leverage form of App. B.2.
* query statistics: sample mean and the 1/N (maximum-likelihood) covariance of
  the observation-window queries (Sec. 3.4 end: estimated from observed
  queries; App. B.2: diagonal covariance in practice).
* GQA: the G query heads sharing a KV head are pooled into one sample of
  G*w queries; the per-head alternative scores each head alone and averages.
* u_i = v_i (Sec. 3.4 end: the proxy used when W_O is not applied). The
  output-projection variant u_i = W_O v_i (Sec. 3.1, Preliminary; Sec. 3.4 end) is taken
  for the G query heads of a KV head together: their outputs are summed by
  the layer, so u_i = W~ v_i with W~ = sum_g W_O^g (the heads' column slices
  of the projection). By the push-through identity its Eq. 10 score equals
  w_i v_i^T (R + sum_j w_j v_j v_j^T)^{-1} v_i with R = (W~^T W~)^{-1}: the
  d x d ridge matrix R replaces ridge*I (see output_ridge_matrix).
* TOP-B: order by (fp32 score desc, index asc), NaN lowest, -0 == +0, and
  return the kept indices in ascending order; |C| = min(B, n). No token is
  protected by default (Algorithm 1 ranks all); an optional protected tail
  keeps the most recent positions first.
"""

from __future__ import annotations

import math

import numpy as np
import scipy.linalg

DIAG = "diag"
FULL = "full"


# ---------------------------------------------------------------------------
# Step 0: query statistics (mu_Q, Lambda_Q)
# ---------------------------------------------------------------------------

def pool_queries(q_group: np.ndarray) -> np.ndarray:
    """Stack the window queries of the G query heads of one KV head: (G, w, d) -> (G*w, d)."""
    q_group = np.asarray(q_group, dtype=np.float64)
    return q_group.reshape(-1, q_group.shape[-1])


def query_statistics(Qs: np.ndarray, cov_mode: str = DIAG):
    """Centre mu_Q and covariance Lambda_Q of the local query model q = mu_Q + dq,
    dq ~ N(0, Lambda_Q) (Sec. 3.3), estimated from the observed window queries
    (Sec. 3.4, last paragraph). DIAG returns the per-channel variances (App. B.2:
    diagonal covariance in practice); FULL returns the d x d matrix."""
    Qs = np.asarray(Qs, dtype=np.float64)
    N = Qs.shape[0]
    mu = Qs.sum(axis=0) / N
    dev = Qs - mu
    if cov_mode == DIAG:
        return mu, (dev * dev).sum(axis=0) / N
    if cov_mode == FULL:
        return mu, dev.T @ dev / N
    raise ValueError(cov_mode)


# ---------------------------------------------------------------------------
# Algorithm 1, step 1: attention at the query centre over the full pool
# ---------------------------------------------------------------------------

def centre_logits(K: np.ndarray, mu: np.ndarray, tau: float) -> np.ndarray:
    """Logits k_i^T mu_Q / (tau sqrt(d_k)) of the subset-independent centre
    attention (Sec. 3.4, definition of bar-alpha; Algorithm 1, first step)."""
    d = K.shape[1]
    return (K @ mu) / (tau * math.sqrt(d))


def centre_attention(z: np.ndarray):
    """bar-alpha = softmax(z) over every cached token, and 1 - bar-alpha.

    1 - bar-alpha_i is the softmax mass of the other tokens, sum_{j != i} e_j / Z.
    Formed as Z - e_i it cancels for a token that holds most of the mass (at
    most one token holds more than half), so for that token the other tokens'
    terms are summed directly."""
    m = z.max()
    e = np.exp(z - m)
    Z = e.sum()
    rest = Z - e
    i = int(np.argmax(e))
    if e[i] > 0.5 * Z:
        rest[i] = np.delete(e, i).sum()
    return e / Z, rest / Z


# ---------------------------------------------------------------------------
# Algorithm 1, step 2: softmax-sensitive importance weight (Eq. 8)
# ---------------------------------------------------------------------------

def query_response(K: np.ndarray, lam: np.ndarray) -> np.ndarray:
    """kappa_i = k_i^T Lambda_Q k_i (Sec. 3.4, diagonal query response)."""
    K = np.asarray(K, dtype=np.float64)
    if lam.ndim == 1:
        return (K * K) @ lam
    return np.einsum("ia,ab,ib->i", K, lam, K)


def importance_weights(alpha: np.ndarray, one_minus_alpha: np.ndarray,
                       kappa: np.ndarray, d: int) -> np.ndarray:
    """w_i = (1/d_k) rho_i^2 kappa_i with rho_i = bar-alpha_i (1 - bar-alpha_i)
    (Eq. 8; rho is the diagonal softmax sensitivity of Sec. 3.4)."""
    rho = alpha * one_minus_alpha
    return rho * rho * kappa / d


# ---------------------------------------------------------------------------
# Algorithm 1, steps 3-4: capacity matrix (Eq. 9) and leverage score (Eq. 10)
# ---------------------------------------------------------------------------

def capacity_matrix(U: np.ndarray, w: np.ndarray, ridge) -> np.ndarray:
    """A = ridge * I + sum_j w_j u_j u_j^T over the whole candidate pool (Eq. 9).
    ridge may also be a d x d symmetric positive definite matrix R, which then
    takes the place of ridge * I (the output-projection variant)."""
    U = np.asarray(U, dtype=np.float64)
    d = U.shape[1]
    R = np.asarray(ridge, dtype=np.float64)
    base = R * np.eye(d) if R.ndim == 0 else R
    return base + U.T @ (w[:, None] * U)


def group_output_projection(w_o: np.ndarray, head: int, group: int, d: int) -> np.ndarray:
    """W~ = sum_g W_O^g over the G query heads g of KV head `head`: W_O^g is the
    (d_model x d) column slice of the layer's output projection that maps
    query head g's attention output into the residual stream (Sec. 3.1, Preliminary: o =
    W_O sum_i alpha_i v_i, per head). w_o is (d_model, H_q * d)."""
    w_o = np.asarray(w_o, dtype=np.float64)
    cols = [w_o[:, (head * group + g) * d:(head * group + g + 1) * d] for g in range(group)]
    return np.sum(cols, axis=0)


def output_ridge_matrix(w_tilde: np.ndarray) -> np.ndarray:
    """R = (W~^T W~)^{-1} for u_i = W~ v_i. With U = W~ V^T, Eq. 10 in output
    space is w_i v_i^T W~^T (I + W~ M W~^T)^{-1} W~ v_i (M = sum_j w_j v_j v_j^T),
    and the push-through identity turns W~^T (I + W~ M W~^T)^{-1} W~ into
    (G^{-1} + M)^{-1} with G = W~^T W~ (full column rank). So the d x d matrix
    R = G^{-1} replaces ridge * I in Eq. 9."""
    w_tilde = np.asarray(w_tilde, dtype=np.float64)
    G = w_tilde.T @ w_tilde
    return np.linalg.inv(G)


def leverage_scores(U: np.ndarray, w: np.ndarray, A: np.ndarray):
    """score_i = w_i u_i^T A^{-1} u_i (Eq. 10), evaluated as w_i ||L^{-1} u_i||^2
    with A = L L^T. Returns (scores, singular); when A is not positive definite
    (ridge 0 and a rank-deficient weighted Gram) the Moore-Penrose inverse of A
    is used instead and singular is True."""
    U = np.asarray(U, dtype=np.float64)
    try:
        L = np.linalg.cholesky(A)
    except np.linalg.LinAlgError:
        return leverage_scores_eigh(U, w, A), True
    Y = scipy.linalg.solve_triangular(L, U.T, lower=True)
    return w * (Y * Y).sum(axis=0), False


def leverage_scores_eigh(U: np.ndarray, w: np.ndarray, A: np.ndarray,
                         rcond: float = 1e-12) -> np.ndarray:
    """The same score through the eigendecomposition A = Q diag(s) Q^T:
    w_i sum_j (q_j^T u_i)^2 / s_j, dropping s_j <= rcond * max(s) (pseudo-inverse)."""
    s, Q = np.linalg.eigh(A)
    keep = s > rcond * max(float(s.max()), 0.0)
    P = np.asarray(U, dtype=np.float64) @ Q[:, keep]
    return w * (P * P / s[keep]).sum(axis=1)


# ---------------------------------------------------------------------------
# Algorithm 1, step 5: TOP-B, then the retained cache Z_C (Sec. 3.1)
# ---------------------------------------------------------------------------

def to_fp32(scores: np.ndarray) -> np.ndarray:
    """Round fp64 scores once to fp32 (round to nearest even); selection is
    decided on these."""
    return np.asarray(scores, dtype=np.float64).astype(np.float32)


def select_top(scores32: np.ndarray, budget: int, protect_last: int = 0) -> np.ndarray:
    """Indices of the min(budget, n) best tokens by (score desc, index asc), NaN
    ranked lowest and -0 equal to +0, returned in ascending index order (int32).
    protect_last = P > 0: the last min(P, budget, n) positions are kept first
    and the ranking fills the rest of the budget from the earlier positions."""
    s = np.asarray(scores32, dtype=np.float32).astype(np.float64)
    n = s.shape[0]
    b = max(0, min(int(budget), n))
    p = min(max(int(protect_last), 0), b)
    if p > 0:
        head = select_top(s[:n - p], b - p)
        return np.concatenate([head, np.arange(n - p, n)]).astype(np.int32)
    nan = np.isnan(s)
    key = np.where(nan, 0.0, s) + 0.0        # +0.0 turns -0 into +0
    # lexsort: last key is primary -> NaN flag, then -score, then index.
    order = np.lexsort((np.arange(n), -key, nan))
    return np.sort(order[:b]).astype(np.int32)


def compact(K: np.ndarray, V: np.ndarray, idx: np.ndarray):
    """Retained cache Z_C = {(k_i, v_i)}_{i in C} (Sec. 3.1): an exact gather."""
    return K[idx], V[idx]


# ---------------------------------------------------------------------------
# One unit (sequence, layer, KV head) end to end
# ---------------------------------------------------------------------------

def score_unit(q_group, K, V, *, tau: float = 10.0, ridge=1.0,
               cov_mode: str = DIAG) -> dict:
    """Jacap scores of one KV head (Algorithm 1 steps 1-4) with every
    intermediate, in float64. q_group is (G, w, d) or (N, d); K and V are (n, d).
    ridge is a scalar or a d x d SPD matrix (see capacity_matrix)."""
    Qs = pool_queries(q_group)
    mu, lam = query_statistics(Qs, cov_mode)
    return score_unit_from_stats(mu, lam, K, V, tau=tau, ridge=ridge)


def score_unit_from_stats(mu, lam, K, V, *, tau: float = 10.0, ridge=1.0) -> dict:
    """Algorithm 1 steps 1-4 from its literal inputs: the query centre mu_Q and
    covariance Lambda_Q (a length-d vector of per-channel variances, or a d x d
    matrix), K and V (n, d). Same outputs as score_unit."""
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    mu = np.asarray(mu, dtype=np.float64)
    lam = np.asarray(lam, dtype=np.float64)
    n, d = K.shape
    out = {"mu": mu, "lam": lam, "n": n, "d": d}
    if n == 0:
        out.update(scores=np.zeros(0), w=np.zeros(0), singular=False,
                   A=capacity_matrix(np.zeros((0, d)), np.zeros(0), ridge))
        return out
    z = centre_logits(K, mu, tau)
    alpha, one_minus = centre_attention(z)
    kappa = query_response(K, lam)
    w = importance_weights(alpha, one_minus, kappa, d)
    A = capacity_matrix(V, w, ridge)
    scores, singular = leverage_scores(V, w, A)
    out.update(z=z, alpha=alpha, one_minus_alpha=one_minus, kappa=kappa, w=w,
               A=A, scores=scores, singular=singular)
    return out


def score_unit_per_head(q_group, K, V, **kw) -> dict:
    """Per-query-head GQA reading: each of the G query heads is scored alone
    (its own w window queries give mu_Q, Lambda_Q, the weights and A), and a
    token's score is the mean over the heads, summed in head order."""
    q_group = np.asarray(q_group, dtype=np.float64)
    if q_group.ndim == 2:
        q_group = q_group[None]
    heads = [score_unit(q_group[g:g + 1], K, V, **kw) for g in range(q_group.shape[0])]
    total = heads[0]["scores"].copy()
    for h in heads[1:]:
        total = total + h["scores"]
    out = dict(heads[0])
    out.update(scores=total / len(heads), heads=heads,
               singular=any(h["singular"] for h in heads))
    return out


def evict_unit(q_group, K, V, budget: int, gqa: str = "pooled", protect_last: int = 0,
               **kw) -> dict:
    """score_unit (or score_unit_per_head for gqa="per_head"), then TOP-B on
    the fp32 scores and the compacted K', V'."""
    scorer = score_unit_per_head if gqa == "per_head" else score_unit
    out = scorer(q_group, K, V, **kw)
    s32 = to_fp32(out["scores"])
    idx = select_top(s32, budget, protect_last)
    Kc, Vc = compact(np.asarray(K), np.asarray(V), idx)
    out.update(scores32=s32, idx=idx, k_out=Kc, v_out=Vc)
    return out


# ---------------------------------------------------------------------------
# Exact greedy log-det selection (a quality comparator for the TOP-B ranking)
# ---------------------------------------------------------------------------

def greedy_logdet(U: np.ndarray, w: np.ndarray, ridge: float, budget: int,
                  protect_last: int = 0) -> np.ndarray:
    """Sequential greedy maximisation of log det(ridge I + sum_{i in C} w_i u_i u_i^T)
    (App. B.1: the capacity objective Jacap's one-shot scores approximate),
    with the full-pool Eq. 8 weights. Step t adds the token with the largest
    gain w_i c_i, c_i = u_i^T A_C^{-1} u_i (its log-det increase is
    log(1 + w_i c_i)); ties go to the lowest index.
    A_C^{-1} = I / ridge - sum_t g_t g_t^T, g_t = A^{-1} u_s sqrt(w_s / (1 + w_s c_s))
    (Sherman-Morrison), so c_i <- c_i - (u_i . g_t)^2.
    protect_last = P: the last min(P, budget, n) positions are added first, in
    position order, and the search covers the earlier ones.
    Returns the chosen indices in the order they were added. Requires ridge > 0."""
    U = np.asarray(U, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, d = U.shape
    k = max(0, min(int(budget), n))
    p = min(max(int(protect_last), 0), k)
    nfree = n - p
    c = (U * U).sum(axis=1) / ridge
    taken = np.zeros(n, dtype=bool)
    taken[nfree:] = True            # protected: never candidates of the search
    G = np.zeros((0, d))
    order = []
    for t in range(k):
        if t < p:
            s = nfree + t
        else:
            gain = np.where(taken, -np.inf, w * c)
            s = int(np.argmax(gain))             # first maximum: lowest index
        us = U[s]
        h = us / ridge - G.T @ (G @ us)
        g = h * math.sqrt(w[s] / (1.0 + w[s] * c[s]))
        taken[s] = True
        order.append(s)
        c = c - (U @ g) ** 2
        G = np.vstack([G, g])
    return np.asarray(order, dtype=np.int64)


def greedy_replay(U: np.ndarray, w: np.ndarray, ridge: float, order, protect_last: int = 0):
    """Follow a given pick order and report, per step, the gain w_s c_s of the
    token it took and the best gain available then (over the untaken
    positions before the protected tail; protected steps report their own
    gain for both). An order is a valid greedy path when every chosen gain
    equals the best one. Same Sherman-Morrison bookkeeping as greedy_logdet."""
    U = np.asarray(U, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, d = U.shape
    order = [int(s) for s in order]
    p = min(max(int(protect_last), 0), len(order))
    nfree = n - p
    c = (U * U).sum(axis=1) / ridge
    taken = np.zeros(n, dtype=bool)
    taken[nfree:] = True
    G = np.zeros((0, d))
    chosen, best = [], []
    for t, s in enumerate(order):
        gain = w * c
        chosen.append(gain[s])
        best.append(gain[s] if t < p else np.where(taken, -np.inf, gain).max())
        us = U[s]
        h = us / ridge - G.T @ (G @ us)
        g = h * math.sqrt(w[s] / (1.0 + w[s] * c[s]))
        taken[s] = True
        c = c - (U @ g) ** 2
        G = np.vstack([G, g])
    return np.asarray(chosen), np.asarray(best)


def logdet_objective(U: np.ndarray, w: np.ndarray, ridge: float, C) -> float:
    """log det(ridge I + sum_{i in C} w_i u_i u_i^T)."""
    U = np.asarray(U, dtype=np.float64)
    C = np.asarray(list(C), dtype=np.int64)
    A = ridge * np.eye(U.shape[1]) + U[C].T @ (np.asarray(w)[C, None] * U[C])
    sign, val = np.linalg.slogdet(A)
    return float(val) if sign > 0 else -math.inf
