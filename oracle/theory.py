"""The paper's subset-level objects, for pinning the oracle and brute force.

TEST INFRASTRUCTURE ONLY (same rule as jacap_oracle: only tests, the smoke
check and the benchmark's CPU baseline may use it).

* retained attention map f_C(q) = U_C softmax(K_C q / sqrt(d_k)) (Sec. 3.1,
  Eq. 3);
* softmax Jacobian Diag(a) - a a^T and Lemma 1's J_C = U_C S_C K_C / sqrt(d_k)
  (Sec. 3.3, Eq. 6; App. A.1);
* Theorem 1's Jacobian capacity 1/2 logdet(I + Sigma^-1 J_C Lambda_Q J_C^T)
  (Eq. 7), and the linear (CapKV) capacity of Eq. 2;
* the diagonal-approximated objective of App. B.1,
  1/2 logdet(I + Sigma^-1 sum_{i in C} w_i u_i u_i^T), with isotropic noise;
* exhaustive search over all size-B subsets and exact sequential greedy for
  small n.

Here U holds the output directions as rows (n, d_o), matching the (n, d)
storage of V; the paper writes U as columns.
"""

from __future__ import annotations

import itertools
import math

import numpy as np


def softmax(s: np.ndarray) -> np.ndarray:
    e = np.exp(s - s.max())
    return e / e.sum()


def attention_map(q: np.ndarray, K_C: np.ndarray, U_C: np.ndarray) -> np.ndarray:
    """f_C(q) = U_C softmax(K_C q / sqrt(d_k)) (Eq. 3). K_C: (m, d_k), U_C: (m, d_o)."""
    d = K_C.shape[1]
    return U_C.T @ softmax(K_C @ q / math.sqrt(d))


def softmax_jacobian(alpha: np.ndarray) -> np.ndarray:
    """d softmax / d logits = Diag(alpha) - alpha alpha^T (App. A.1)."""
    return np.diag(alpha) - np.outer(alpha, alpha)


def lemma1_jacobian(K_C: np.ndarray, U_C: np.ndarray, mu: np.ndarray) -> np.ndarray:
    """J_C = (1/sqrt(d_k)) U_C S_C K_C with S_C the softmax Jacobian at
    alpha* = softmax(K_C mu_Q / sqrt(d_k)) (Lemma 1, Eq. 6). Shape (d_o, d_k)."""
    d = K_C.shape[1]
    a = softmax(K_C @ mu / math.sqrt(d))
    return U_C.T @ softmax_jacobian(a) @ K_C / math.sqrt(d)


def gaussian_capacity(J: np.ndarray, Lam: np.ndarray, noise_var: float) -> float:
    """1/2 logdet(I + Sigma^-1 J Lambda J^T) with Sigma = noise_var * I
    (Theorem 1, Eq. 7; the Gaussian mutual information of App. A.1)."""
    Lam = np.diag(Lam) if Lam.ndim == 1 else Lam
    M = np.eye(J.shape[0]) + J @ Lam @ J.T / noise_var
    sign, logdet = np.linalg.slogdet(M)
    return 0.5 * logdet


def jacobian_capacity(C, K, U, mu, Lam, noise_var=1.0, tau=1.0) -> float:
    """Objective (i): Theorem 1's capacity of the retained subset C, with the
    subset's own centre softmax. tau=1 is the literal theorem; other tau divide
    the centre logits as Algorithm 1 does."""
    C = list(C)
    if not C:
        return 0.0
    K_C, U_C = K[C], U[C]
    d = K.shape[1]
    a = softmax(K_C @ mu / (tau * math.sqrt(d)))
    J = U_C.T @ softmax_jacobian(a) @ K_C / math.sqrt(d)
    return gaussian_capacity(J, Lam, noise_var)


def linear_capacity(C, K, U, Lam, noise_var=1.0) -> float:
    """The linear-Gaussian (CapKV) capacity 1/2 logdet(I + Sigma^-1 U_C K_C
    Lambda K_C^T U_C^T) (Eq. 2)."""
    C = list(C)
    J = U[C].T @ K[C]
    return gaussian_capacity(J, Lam, noise_var)


def diag_objective(C, w, U, ridge) -> float:
    """Objective (ii): 1/2 logdet(I + ridge^-1 sum_{i in C} w_i u_i u_i^T)
    (App. B.1, isotropic noise absorbed into the ridge), with the full-pool w."""
    C = list(C)
    d = U.shape[1]
    M = np.eye(d) + (U[C].T * w[C]) @ U[C] / ridge
    return 0.5 * np.linalg.slogdet(M)[1]


def brute_force_best(objective, n: int, k: int):
    """Exhaustive argmax of objective(C) over all |C| = k subsets of range(n).
    Returns (best_subset, best_value, all_values)."""
    best, best_val, vals = None, -np.inf, []
    for C in itertools.combinations(range(n), k):
        v = objective(C)
        vals.append(v)
        if v > best_val:
            best, best_val = C, v
    return best, best_val, np.array(vals)


def greedy(objective, n: int, k: int):
    """Exact sequential greedy: add the token with the largest objective gain."""
    C = []
    for _ in range(k):
        rest = [i for i in range(n) if i not in C]
        gains = [objective(C + [i]) for i in rest]
        C.append(rest[int(np.argmax(gains))])
    return sorted(C)
