"""Shared helpers for the GPU parity tests: run the HIP path through the C ABI
on a synthetic case, run the fp64 oracle on chosen units, compare."""

from __future__ import annotations

import math

import numpy as np
import torch

from oracle import jacap_oracle as jo

BF16_TOL = 1e-3   # relative, bf16 inputs with fp32 accumulation
FP32_TOL = 1e-5   # relative, fp32 inputs
FLOOR = 1e-6      # relative-error floor: max(|o_i|, FLOOR * max_j |o_j|)


def tol_for(case) -> float:
    return BF16_TOL if case.workload.dtype == "bf16" else FP32_TOL


def run_gpu(case, budget, tau=10.0, ridge=1.0, cov_mode=0, stream=None, ridge_matrices=None,
            gqa="pooled", protect_last=0):
    from paper_2609_08131_amd import jacap
    rm = None
    if ridge_matrices is not None:
        rm = torch.as_tensor(np.ascontiguousarray(ridge_matrices), dtype=torch.float64).cuda()
    p = jacap.Params(budget_k=budget, temperature=tau, ridge=ridge, cov_mode=cov_mode,
                     ridge_matrix=rm,
                     gqa_mode=jacap.GQA_PER_HEAD if gqa == "per_head" else jacap.GQA_POOLED,
                     protect_last=protect_last)
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    jacap.run_evict(prob, case.q_win, case.k, case.v, stream)
    flags = jacap.read_status(prob.ws, stream)
    torch.cuda.synchronize()
    return prob, flags


def unit_list(case):
    w = case.workload
    return [(b, l, h) for b in range(case.num_seqs) for l in range(w.num_layers)
            for h in range(w.num_kv_heads)]


def unit_index(case, b, l, h):
    w = case.workload
    return (b * w.num_layers + l) * w.num_kv_heads + h


def token_slice(case, b):
    lo = int(sum(case.seq_lens[:b]))
    return lo, lo + int(case.seq_lens[b])


def oracle_unit(case, b, l, h, budget, tau=10.0, ridge=1.0, cov_mode="diag", gqa="pooled",
                protect_last=0):
    q, k, v = case.unit_arrays(b, l, h)
    return jo.evict_unit(q, k, v, budget, tau=tau, ridge=ridge, cov_mode=cov_mode, gqa=gqa,
                         protect_last=protect_last)


# Scores are returned in fp32: below its normal range (2^-126) they carry an
# absolute resolution, not a relative one, so that is the comparison's scale
# there (units whose centre softmax is saturated to ~1e-30 and beyond).
FP32_NORMAL_MIN = float(np.finfo(np.float32).tiny)


def score_errors(gpu: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Floored relative error |g - o| / max(|o|, FLOOR * max|o|, 2^-126)."""
    ref = np.asarray(ref, np.float64)
    gpu = np.asarray(gpu, np.float64)
    if ref.size == 0:
        return np.zeros(0)
    denom = np.maximum(np.abs(ref), FLOOR * np.max(np.abs(ref)))
    denom = np.maximum(denom, FP32_NORMAL_MIN)
    denom = np.where(denom > 0, denom, 1.0)
    return np.abs(gpu - ref) / denom


def gpu_unit_scores(case, prob, b, l, h) -> np.ndarray:
    lo, hi = token_slice(case, b)
    return prob.scores[l, h, lo:hi].double().cpu().numpy()


def gpu_unit_idx(case, prob, b, l, h, budget) -> np.ndarray:
    n = case.seq_lens[b]
    kk = min(budget, n)
    row = prob.idx[b, l, h].cpu().numpy()
    assert np.all(row[kk:] == -1), "padding slots must hold -1"
    return row[:kk]


def overlap(a, b) -> float:
    a, b = set(np.asarray(a).tolist()), set(np.asarray(b).tolist())
    return len(a & b) / max(1, len(b))


def trace_ridge(case, b, l, h, tau=10.0):
    """ridge = tr(M)/d, where the diversity term is neither negligible nor dominant."""
    out = oracle_unit(case, b, l, h, 1, tau=tau, ridge=1.0)
    M = out["A"] - np.eye(out["A"].shape[0])
    return float(np.trace(M) / M.shape[0])


def finite_close(a, b):
    return math.isclose(a, b, rel_tol=1e-12)
