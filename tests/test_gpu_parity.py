"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Scores: floored relative error <= 1e-3 for bf16 inputs, <= 1e-5 for fp32.
Selection: jacap_select on the oracle's fp32 scores must equal the oracle's
selection bit for bit; jacap_select on the GPU scores must equal the oracle's
select rule applied to those same scores; the overlap of the GPU selection
with the oracle's (different scores, so not required to be exact) is printed.
Compaction: K', V' rows are bit-exact gathers.
"""

import numpy as np
import pytest
import torch

from jacap_synth import make_case
from jacap_synth.cases import make_output_projection
from oracle import jacap_oracle as jo

from helpers import (gpu_unit_idx, gpu_unit_scores, oracle_unit, overlap, run_gpu, score_errors,
                     token_slice, tol_for, trace_ridge, unit_list)

pytestmark = pytest.mark.gpu

COV = {"diag": 0, "full": 1}
# A unit's scores are NaN (JACAP_FLAG_SINGULAR) only when the fp64 Cholesky of
# its fp64 Gram meets a pivot at or below 1e-10 (bf16) / 1e-8 (fp32) of its
# diagonal entry, which implies cond(A) above 1e10 / 1e8: there fp64 rounding
# alone (any evaluation order, the oracle's included) moves the scores by more
# than the tolerance.
SINGULAR_COND = {"bf16": 1e10, "fp32": 1e8}


@pytest.fixture(scope="module")
def jacap():
    from paper_2609_08131_amd import jacap as j
    return j


def check_case(case, budget, ridge, mode="diag", units=None, tau=10.0, label="", jacap=None,
               ridge_matrices=None, gqa="pooled", protect_last=0):
    units = unit_list(case) if units is None else units
    all_units = len(units) == len(unit_list(case))
    prob, flags = run_gpu(case, budget, tau=tau, ridge=ridge, cov_mode=COV[mode],
                          ridge_matrices=ridge_matrices, gqa=gqa, protect_last=protect_last)
    # SINGULAR is legitimate only at ridge 0 (rank-deficient weighted Gram)
    assert flags & ~(2 if ridge == 0.0 else 0) == 0, f"status flags {flags}"
    tol = tol_for(case)
    ref32 = torch.zeros_like(prob.scores, device="cpu")
    worst, overlaps, orc, worst_cond = 0.0, [], {}, 0.0
    for (b, l, h) in units:
        o = oracle_unit(case, b, l, h, budget, tau=tau, cov_mode=mode, gqa=gqa,
                        protect_last=protect_last,
                        ridge=ridge if ridge_matrices is None else ridge_matrices[l, h])
        orc[(b, l, h)] = o
        g = gpu_unit_scores(case, prob, b, l, h)
        if len(g) and np.isnan(g).any():
            # Only a numerically singular capacity matrix may be flagged.
            assert ridge == 0.0 and (flags & 2) and np.isnan(g).all(), (label, (b, l, h))
            for hd in o.get("heads", [o]):
                ev = np.linalg.eigvalsh(hd["A"])
                cond = np.inf if ev[0] <= 0 else ev[-1] / ev[0]
                assert hd["singular"] or cond > SINGULAR_COND[case.workload.dtype], \
                    (label, (b, l, h), cond)
        elif len(g):
            # Every unit at the stated tolerance, whatever its conditioning (the
            # ill-conditioned ones take the fp64 path on the GPU).
            assert not o["singular"] or gqa == "per_head", (label, (b, l, h), "oracle singular")
            err = score_errors(g, o["scores"])
            worst = max(worst, float(err.max()))
            for hd in o.get("heads", [o]):
                ev = np.linalg.eigvalsh(hd["A"])
                worst_cond = max(worst_cond, np.inf if ev[0] <= 0 else ev[-1] / ev[0])
            assert err.max() <= tol, (label, (b, l, h), float(err.max()), int(err.argmax()))
        idx = gpu_unit_idx(case, prob, b, l, h, budget)
        assert np.array_equal(idx, jo.select_top(g.astype(np.float32), budget, protect_last)), \
            (label, (b, l, h))
        overlaps.append(overlap(idx, o["idx"]) if len(o["idx"]) else 1.0)
        lo, hi = token_slice(case, b)
        kk = len(idx)
        if kk:
            sel = torch.as_tensor(idx.astype(np.int64), device=case.k.device) + lo
            assert torch.equal(prob.k_out[b, l, h, :kk], case.k[l, h, sel])
            assert torch.equal(prob.v_out[b, l, h, :kk], case.v[l, h, sel])
        ref32[l, h, lo:hi] = torch.from_numpy(o["scores32"])
    if all_units and jacap is not None and budget > 0:
        idx2 = torch.empty_like(prob.idx)
        jacap.select(prob.cfg, prob.batch, ref32.to(prob.scores.device), idx2)
        torch.cuda.synchronize()
        for (b, l, h), o in orc.items():
            kk = len(o["idx"])
            got = idx2[b, l, h].cpu().numpy()
            assert np.array_equal(got[:kk], o["idx"]), ("select on oracle scores", label, (b, l, h))
            assert np.all(got[kk:] == -1)
    print(f"\n[parity] {label} ridge={ridge:g} {mode}: worst rel err {worst:.3e} (tol {tol:g}, "
          f"worst cond(A) {worst_cond:.2e}); overlap with oracle selection "
          f"min {min(overlaps):.4f} mean {np.mean(overlaps):.4f}")
    return prob, worst


# ---------------------------------------------------------------------------
# 1 x 1 head, d=64, n=512, w=16, k=64, fp32 (tiny workload)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("mode", ["diag", "full"])
@pytest.mark.parametrize("ridge", ["1", "1/d", "0", "trace"])
def test_tiny_fp32(jacap, ridge, mode):
    case = make_case("tiny").to("cuda")
    d = case.workload.head_dim
    r = {"1": 1.0, "1/d": 1.0 / d, "0": 0.0}.get(ridge)
    if r is None:
        r = trace_ridge(case, 0, 0, 0)
    check_case(case, case.workload.budget_k, r, mode, label=f"tiny/{ridge}", jacap=jacap)


# ---------------------------------------------------------------------------
# Llama-3-8B-shaped layer: 8 KV heads (32 q heads), d=128, n=8192, w=32, k=512, bf16
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("ridge", ["1", "1/d", "0", "trace"])
def test_llama_layer_bf16_diag(jacap, ridge):
    case = make_case("llama8b_layer", device="cuda")
    d = case.workload.head_dim
    r = {"1": 1.0, "1/d": 1.0 / d, "0": 0.0}.get(ridge)
    if r is None:
        r = trace_ridge(case, 0, 0, 0)
    check_case(case, case.workload.budget_k, r, "diag", label=f"llama_layer/{ridge}", jacap=jacap)


@pytest.mark.parametrize("ridge", [1.0, 0.0])
def test_llama_layer_bf16_full(jacap, ridge):
    case = make_case("llama8b_layer", device="cuda")
    check_case(case, case.workload.budget_k, ridge, "full", label="llama_layer", jacap=jacap)


# ---------------------------------------------------------------------------
# Ragged batches, both dtypes and head sizes, chunk boundaries and empty seqs
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d,heads,window", [(64, 3, 7), (128, 4, 64), (128, 4, 80)])
def test_full_covariance_window_shapes_bf16(jacap, d, heads, window):
    """FULL covariance with bf16 keys: the MFMA K pass stages the pooled
    window in LDS -- N_s = 21 (a partial 16-query tile, d = 64), N_s = 256 (the
    largest it takes) -- and N_s = 320 takes the VALU path; ragged lengths
    with partial 64-token passes and an empty sequence."""
    case = make_case("ragged16", device="cuda", seq_lens=(0, 1, 17, 300, 1500), num_layers=1,
                     num_kv_heads=2, num_q_heads=2 * heads, window=window, head_dim=d,
                     dtype="bf16")
    check_case(case, 64, 1.0, "full", label=f"full d={d} N_s={heads * window}", jacap=jacap)


def _low_rank_window(case, b, l, h, rank, noise, seed):
    """Replace the pooled window of unit (b, l, h) by queries spanning `rank`
    directions plus isotropic noise of standard deviation `noise` (0: a
    Lambda_Q of rank `rank`, up to the bf16 rounding of the queries)."""
    w = case.workload
    g = w.num_q_heads // w.num_kv_heads
    gen = torch.Generator().manual_seed(seed)
    basis = torch.randn((rank, w.head_dim), generator=gen)
    coef = torch.randn((g, w.window, rank), generator=gen)
    centre = torch.randn((w.head_dim,), generator=gen)
    q = centre + coef @ basis / rank ** 0.5
    q = q + noise * torch.randn((g, w.window, w.head_dim), generator=gen)
    case.q_win[b, l, h * g:(h + 1) * g] = q.to(case.q_win.dtype)


@pytest.mark.parametrize("d,heads,window", [(128, 4, 64), (64, 4, 32), (64, 8, 32)])
def test_full_covariance_triangular_path(jacap, d, heads, window):
    """FULL covariance with bf16 keys, N_s >= 2 d and units of at least 8192
    tokens: kappa = ||X k||^2 from the factor Lambda_Q = X^T X. In the same
    launch the window tile scores the shorter units (3000 and 1 tokens; an
    empty sequence), a unit whose window spans d / 8 directions (rank-deficient
    Lambda_Q) and one with no query noise beyond bf16 rounding in d / 2 of
    them; a unit whose window spans d / 2 directions plus noise at 0.06 of
    their scale (pivot ratios ~4e-3, just above the factor's cut) stays on the
    triangular path."""
    case = make_case("ragged16", seq_lens=(9000, 0, 3000, 1, 8192), num_layers=2,
                     num_kv_heads=2, num_q_heads=2 * heads, window=window, head_dim=d,
                     dtype="bf16")
    _low_rank_window(case, 0, 1, 0, d // 8, 0.0, seed=11)
    _low_rank_window(case, 4, 0, 1, d // 2, 0.0, seed=12)
    _low_rank_window(case, 4, 1, 1, d // 2, 0.06, seed=13)
    case = case.to("cuda")
    for ridge in (1.0, 0.0):
        check_case(case, 256, ridge, "full", label=f"full-tri d={d} N_s={heads * window}",
                   jacap=jacap)


def test_full_covariance_triangular_path_per_head(jacap):
    """Per-head GQA on the FULL triangular path: every query head is a unit of
    its own with N_s = w = 128 = 2d window queries (d = 64), and the K rows of
    a KV head are read by its G query-head units together (cached loads). A
    sequence of 8200 tokens takes the triangular path, one of 500 the window
    tile, in the same launch."""
    case = make_case("ragged16", seq_lens=(8200, 500), num_layers=1, num_kv_heads=2,
                     num_q_heads=4, window=128, head_dim=64, dtype="bf16").to("cuda")
    check_case(case, 128, 1.0, "full", gqa="per_head", label="full-tri per-head d=64",
               jacap=jacap)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("bf16", 64), ("fp32", 64), ("fp32", 128)])
def test_ragged_small(jacap, dtype, d):
    lens = [0, 1, 17, 255, 256, 257, 1000, 8193]
    # drawn on the CPU so that the same inputs can be reproduced off the GPU
    case = make_case("ragged16", seq_lens=lens, num_layers=2, num_kv_heads=2,
                     num_q_heads=4, head_dim=d, window=8, dtype=dtype).to("cuda")
    for ridge in (1.0, 0.0):
        check_case(case, 64, ridge, "diag", label=f"ragged/{dtype}/d{d}", jacap=jacap)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("fp32", 128), ("bf16", 64)])
def test_more_units_than_compute_units(jacap, dtype, d):
    """A batch of 288 units (more than the 256 compute units): the capacity
    factorisation takes its four-wave shape, two workgroups per compute
    unit, on the first pass (and on every unit of fp32 inputs); at ridge 0
    many units go on to the fp64 path. Every unit against the oracle."""
    lens = [(37 * i) % 200 + 1 for i in range(24)]
    case = make_case("ragged16", seq_lens=lens, num_layers=3, num_kv_heads=4,
                     num_q_heads=8, head_dim=d, window=8, dtype=dtype).to("cuda")
    assert case.num_seqs * 3 * 4 == 288
    for ridge in (1.0, 0.0):
        check_case(case, 32, ridge, "diag", label=f"288 units/{dtype}/d{d}", jacap=jacap)


def test_budget_edges(jacap):
    case = make_case("ragged16", device="cuda", seq_lens=[3, 40, 700], num_layers=1,
                     num_kv_heads=2, num_q_heads=2, head_dim=128, window=4)
    check_case(case, 40, 1.0, label="k=40 (>= some n)", jacap=jacap)
    check_case(case, 700, 1.0, label="k=n_max", jacap=jacap)
    prob, flags = run_gpu(case, 0, ridge=1.0)
    assert flags == 0 and prob.idx.numel() == 0


def test_window_of_one_gives_zero_scores(jacap):
    case = make_case("llama8b_layer", device="cuda", seq_lens=[3000], num_q_heads=8, window=1)
    prob, flags = run_gpu(case, 100, ridge=1.0)
    assert flags == 0
    assert torch.count_nonzero(prob.scores) == 0
    want = torch.arange(100, dtype=torch.int32, device="cuda")
    assert torch.equal(prob.idx[0, 0], want.expand(8, 100))


def test_deterministic_bitwise(jacap):
    case = make_case("llama8b_layer", device="cuda")
    a, _ = run_gpu(case, 512, ridge=0.0)
    s1, i1 = a.scores.clone(), a.idx.clone()
    jacap.run_evict(a, case.q_win, case.k, case.v)
    torch.cuda.synchronize()
    assert torch.equal(a.scores.view(torch.int32), s1.view(torch.int32))
    assert torch.equal(a.idx, i1)


# ---------------------------------------------------------------------------
# Data-dependent errors: flags and NaN scores for the affected unit only
# ---------------------------------------------------------------------------

def test_nonfinite_input_flags_unit(jacap):
    case = make_case("llama8b_layer", device="cuda", seq_lens=[2000], num_kv_heads=2, num_q_heads=4)
    case.k[0, 1, 77, 5] = float("nan")
    prob, flags = run_gpu(case, 64, ridge=1.0)
    assert flags & jacap.FLAG_NONFINITE
    assert torch.isnan(prob.scores[0, 1]).all()
    assert torch.isfinite(prob.scores[0, 0]).all()
    assert torch.equal(prob.idx[0, 0, 1], torch.arange(64, dtype=torch.int32, device="cuda"))


def test_singular_capacity_matrix_flagged(jacap):
    case = make_case("llama8b_layer", device="cuda", seq_lens=[50], num_kv_heads=1, num_q_heads=4)
    prob, flags = run_gpu(case, 10, ridge=0.0)          # 50 tokens < d = 128: rank deficient
    assert flags & jacap.FLAG_SINGULAR
    assert torch.isnan(prob.scores).all()
    prob, flags = run_gpu(case, 10, ridge=1.0)
    assert flags == 0 and torch.isfinite(prob.scores).all()


def test_inconsistent_offsets_are_bounded(jacap):
    case = make_case("ragged16", device="cuda", seq_lens=[100, 300], num_layers=1, num_kv_heads=1,
                     num_q_heads=1, head_dim=64, window=4)
    p = jacap.Params(budget_k=16)
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    prob.batch.max_seq_len = 200       # the second sequence (300) contradicts it
    jacap.run_evict(prob, case.q_win, case.k, case.v)
    flags = jacap.read_status(prob.ws)
    assert flags & jacap.FLAG_BAD_OFFSETS
    assert torch.all(prob.idx[1] == -1)
    assert torch.isfinite(prob.scores[0, 0, :100]).all()


# ---------------------------------------------------------------------------
# Selection kernel alone: ties, NaN, -0, budgets around n
# ---------------------------------------------------------------------------

def test_select_ties_nan_negzero(jacap):
    case = make_case("ragged16", device="cuda", seq_lens=[1, 33, 1000, 5000], num_layers=1,
                     num_kv_heads=3, num_q_heads=3, head_dim=64, window=2)
    rng = np.random.default_rng(0)
    # 600, 999, 3000, 4990 keep more than half of some units (the complement path)
    for budget in (1, 7, 33, 600, 999, 2048, 3000, 4990):
        p = jacap.Params(budget_k=budget)
        prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
        s = (rng.integers(0, 6, size=prob.scores.shape).astype(np.float32) * 0.5)
        s[rng.random(s.shape) < 0.05] = np.nan
        s[rng.random(s.shape) < 0.05] = -0.0
        s[rng.random(s.shape) < 0.02] = -1.5
        s[rng.random(s.shape) < 0.01] = np.inf
        scores = torch.from_numpy(s).cuda()
        jacap.select(prob.cfg, prob.batch, scores, prob.idx)
        torch.cuda.synchronize()
        for b in range(4):
            lo, hi = token_slice(case, b)
            for h in range(3):
                want = jo.select_top(s[0, h, lo:hi], budget)
                got = prob.idx[b, 0, h].cpu().numpy()
                assert np.array_equal(got[:len(want)], want), (budget, b, h)
                assert np.all(got[len(want):] == -1)


@pytest.mark.gpu
def test_select_large_units_both_paths(jacap):
    """Large units exercise the sampled fast path (spread-out, sorted and
    NaN/-0/inf mixes) and the general radix path (heavy ties, budget n - 1);
    the kept positions must equal the oracle's ranking bit for bit."""
    lens = [8193, 20000, 131072]
    case = make_case("ragged16", device="cuda", seq_lens=lens, num_layers=1,
                     num_kv_heads=4, num_q_heads=4, head_dim=64, window=2)
    rng = np.random.default_rng(7)
    T = sum(lens)
    kinds = {
        0: lambda n: np.exp(rng.normal(0.0, 5.0, n)),
        1: lambda n: np.sort(np.exp(rng.normal(0.0, 3.0, n))),
        2: lambda n: rng.integers(0, 5, n).astype(np.float64),
        3: lambda n: np.exp(rng.normal(0.0, 3.0, n)),
    }
    # 16384 and 125000 keep more than half (selection of the evicted tokens)
    for budget in (1, 1024, 2048, 16384, 20000, 125000):
        p = jacap.Params(budget_k=budget)
        prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
        s = np.zeros((1, 4, T), np.float32)
        for b, n in enumerate(lens):
            lo, hi = token_slice(case, b)
            for h in range(4):
                x = kinds[h](n).astype(np.float32)
                if h == 3:
                    x[rng.random(n) < 0.1] = np.nan
                    x[rng.random(n) < 0.05] = -0.0
                    x[rng.random(n) < 0.05] = 0.0
                    x[rng.random(n) < 0.01] = np.inf
                s[0, h, lo:hi] = x
        print(f"[select] budget {budget}", flush=True)
        jacap.select(prob.cfg, prob.batch, torch.from_numpy(s).cuda(), prob.idx)
        torch.cuda.synchronize()
        for b in range(len(lens)):
            lo, hi = token_slice(case, b)
            for h in range(4):
                want = jo.select_top(s[0, h, lo:hi], budget)
                got = prob.idx[b, 0, h].cpu().numpy()
                assert np.array_equal(got[:len(want)], want), (budget, b, h)
                assert np.all(got[len(want):] == -1)
    # budget = n - 1 on the large unit (the kept-for-sure list cannot hold it)
    n = lens[2]
    p = jacap.Params(budget_k=n - 1)
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    s = np.exp(rng.normal(0.0, 5.0, (1, 4, T))).astype(np.float32)
    jacap.select(prob.cfg, prob.batch, torch.from_numpy(s).cuda(), prob.idx)
    torch.cuda.synchronize()
    lo, hi = token_slice(case, 2)
    want = jo.select_top(s[0, 1, lo:hi], n - 1)
    assert np.array_equal(prob.idx[2, 0, 1].cpu().numpy()[:n - 1], want)


@pytest.mark.parametrize("wl,mode", [("tiny", "diag"), ("tiny", "full"),
                                     ("llama8b_layer", "diag"), ("llama8b_layer", "full")])
def test_score_from_stats(jacap, wl, mode):
    """jacap_score_from_stats (Algorithm 1 with its literal inputs) on
    statistics no window produced -- a random centre and positive variances,
    or a random positive semi-definite matrix -- against the oracle's
    Algorithm 1 from the same statistics, every unit element by element; with
    the window's own statistics (oracle, fp64) it reproduces jacap_score."""
    case = make_case(wl, device="cuda")
    w = case.workload
    B, L, H, d = case.num_seqs, w.num_layers, w.num_kv_heads, w.head_dim
    rng = np.random.default_rng(5)
    mu = rng.normal(size=(B, L, H, d))
    if mode == "diag":
        lam = rng.uniform(0.2, 2.0, size=(B, L, H, d))
    else:
        G = rng.normal(size=(B, L, H, d, d))
        lam = G @ np.swapaxes(G, -1, -2) / d
    p = jacap.Params(budget_k=w.budget_k, cov_mode=COV[mode])
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    jacap.score_from_stats(prob.cfg, prob.batch, torch.from_numpy(mu).cuda(),
                           torch.from_numpy(lam).cuda(), case.k, case.v, prob.scores, prob.ws)
    assert jacap.read_status(prob.ws) == 0
    tol = tol_for(case)
    worst = 0.0
    for (b, l, h) in unit_list(case):
        _, k, v = case.unit_arrays(b, l, h)
        o = jo.score_unit_from_stats(mu[b, l, h], lam[b, l, h], k, v)
        e = score_errors(gpu_unit_scores(case, prob, b, l, h), o["scores"])
        worst = max(worst, float(e.max()))
    assert worst <= tol, (wl, mode, worst)
    # the window's own statistics: the same scores as jacap_score
    mu_w = np.empty((B, L, H, d))
    lam_w = np.empty_like(lam)
    for (b, l, h) in unit_list(case):
        q, _, _ = case.unit_arrays(b, l, h)
        mu_w[b, l, h], lam_w[b, l, h] = jo.query_statistics(jo.pool_queries(q), mode)
    from_stats = torch.empty_like(prob.scores)
    jacap.score_from_stats(prob.cfg, prob.batch, torch.from_numpy(mu_w).cuda(),
                           torch.from_numpy(lam_w).cuda(), case.k, case.v, from_stats, prob.ws)
    jacap.score(prob.cfg, prob.batch, case.q_win, case.k, case.v, prob.scores, prob.ws)
    torch.cuda.synchronize()
    a, c = from_stats.double().cpu().numpy(), prob.scores.double().cpu().numpy()
    rel = np.abs(a - c) / np.maximum(np.abs(c), 1e-6 * np.abs(c).max())
    print(f"\n[from_stats] {wl} {mode}: worst error vs oracle {worst:.2e}; "
          f"vs jacap_score {rel.max():.2e}")
    assert rel.max() <= tol


def test_score_from_stats_nonfinite_flags_unit(jacap):
    case = make_case("tiny", device="cuda")
    d = case.workload.head_dim
    mu = torch.zeros((1, 1, 1, d), dtype=torch.float64, device="cuda")
    lam = torch.ones((1, 1, 1, d), dtype=torch.float64, device="cuda")
    lam[..., 3] = float("nan")
    p = jacap.Params(budget_k=8)
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    jacap.score_from_stats(prob.cfg, prob.batch, mu, lam, case.k, case.v, prob.scores, prob.ws)
    assert jacap.read_status(prob.ws) & jacap.FLAG_NONFINITE
    assert torch.isnan(prob.scores).all()


def test_stream_read_probe(jacap):
    """The measurement probe reads a buffer with a ragged last workgroup and
    leaves the sink alone (its XOR is not the sentinel)."""
    x = torch.arange((3 << 20) // 4 + 64, dtype=torch.int32, device="cuda")
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    jacap.stream_read(x, sink)
    torch.cuda.synchronize()
    assert int(sink[0]) == 0


@pytest.mark.gpu
def test_select_many_units_narrow_shape(jacap):
    """1024 units (4 sequences x 32 layers x 8 KV heads) take the narrow
    selection shape when no unit ranks more than 512 tokens: spread-out scores
    (sampled fast path), heavy ties (the band overflows: radix fallback),
    NaN/-0/inf mixes, budgets keeping more than half (complement path) and a
    protected tail; a budget ranking more than 512 takes the wide shape. Every
    unit must equal the oracle's ranking bit for bit."""
    lens = [1, 700, 3000, 9000]
    case = make_case("ragged16", device="cuda", seq_lens=lens, num_layers=32, num_kv_heads=8,
                     num_q_heads=8, head_dim=64, window=2)
    L, H, T = 32, 8, sum(lens)
    rng = np.random.default_rng(11)
    s = np.exp(rng.normal(0.0, 4.0, (L, H, T))).astype(np.float32)
    s[1::4] = rng.integers(0, 4, (len(range(1, L, 4)), H, T)).astype(np.float32)  # ties
    mix = s[2::4]
    mix[rng.random(mix.shape) < 0.1] = np.nan
    mix[rng.random(mix.shape) < 0.05] = -0.0
    mix[rng.random(mix.shape) < 0.05] = 0.0
    mix[rng.random(mix.shape) < 0.01] = np.inf
    s[2::4] = mix
    scores = torch.from_numpy(s).cuda()
    for budget, protect in ((1, 0), (64, 0), (300, 0), (512, 0), (8600, 0), (8999, 0),
                            (200, 50), (2048, 0)):
        p = jacap.Params(budget_k=budget, protect_last=protect)
        prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
        print(f"[select] 1024 units, budget {budget}, protect {protect}", flush=True)
        jacap.select(prob.cfg, prob.batch, scores, prob.idx)
        torch.cuda.synchronize()
        got_all = prob.idx.cpu().numpy()
        for b in range(len(lens)):
            lo, hi = token_slice(case, b)
            for layer in range(L):
                for h in range(H):
                    want = jo.select_top(s[layer, h, lo:hi], budget, protect)
                    got = got_all[b, layer, h]
                    assert np.array_equal(got[:len(want)], want), (budget, protect, b, layer, h)
                    assert np.all(got[len(want):] == -1)
        del prob


def test_select_evicted_is_the_complement(jacap):
    """jacap_select_evicted lists, per unit and ascending, exactly the positions
    that the oracle's ranking does not keep (ties, NaN, -0 and inf mixes; both
    selection shapes; budgets from 0 to beyond the longest sequence; a
    protected tail); -1 fills the rest of each list."""
    lens = [1, 700, 3000, 9000]
    case = make_case("ragged16", device="cuda", seq_lens=lens, num_layers=32, num_kv_heads=8,
                     num_q_heads=8, head_dim=64, window=2)
    L, H, T = 32, 8, sum(lens)
    rng = np.random.default_rng(12)
    s = np.exp(rng.normal(0.0, 4.0, (L, H, T))).astype(np.float32)
    s[1::4] = rng.integers(0, 4, (len(range(1, L, 4)), H, T)).astype(np.float32)  # ties
    mix = s[2::4]
    mix[rng.random(mix.shape) < 0.1] = np.nan
    mix[rng.random(mix.shape) < 0.05] = -0.0
    mix[rng.random(mix.shape) < 0.01] = np.inf
    s[2::4] = mix
    scores = torch.from_numpy(s).cuda()
    for budget, protect in ((0, 0), (1, 0), (300, 0), (512, 0), (2048, 0), (8600, 0),
                            (8999, 0), (9000, 0), (12000, 0), (200, 50), (8900, 3000)):
        p = jacap.Params(budget_k=budget, protect_last=protect)
        prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
        slots = jacap.alloc_slots(prob, lens)
        slots.fill_(-7)
        print(f"[select_evicted] 1024 units, budget {budget}, protect {protect}", flush=True)
        jacap.select_evicted(prob.cfg, prob.batch, scores, slots, prob.ws)
        torch.cuda.synchronize()
        got_all = slots.cpu().numpy()
        for b in range(len(lens)):
            lo, hi = token_slice(case, b)
            for layer in range(L):
                for h in range(H):
                    kept = jo.select_top(s[layer, h, lo:hi], budget, protect) if budget else []
                    want = np.setdiff1d(np.arange(hi - lo), kept)
                    got = got_all[b, layer, h]
                    assert np.array_equal(got[:len(want)], want), (budget, protect, b, layer, h)
                    assert np.all(got[len(want):] == -1)
        del prob, slots


def test_decode_rounds_refill_evicted_slots_in_place(jacap):
    """jacap_evict_slots: each round writes the next D tokens into the D slots
    it evicts (ascending slots, tokens in arrival order) instead of compacting
    the kept rows. The oracle runs the same chain with its own selections: the
    same slots in every round, hence the same caches."""
    R, D, B, rounds = 256, 32, 2, 3
    spec = dict(num_layers=1, num_kv_heads=2, num_q_heads=4, window=8, head_dim=64, dtype="bf16")
    L, H = spec["num_layers"], spec["num_kv_heads"]
    first = make_case("ragged16", seq_lens=[R + D] * B, **spec)
    k_cache, v_cache = first.k.clone().cuda(), first.v.clone().cuda()
    ok = {(b, l, h): (first.unit_arrays(b, l, h)[1].copy(), first.unit_arrays(b, l, h)[2].copy())
          for b in range(B) for l in range(L) for h in range(H)}
    q_win = first.q_win
    offsets = torch.tensor([i * (R + D) for i in range(B + 1)], dtype=torch.int32).cuda()
    for r in range(rounds):
        print(f"[decode in place] round {r}", flush=True)
        qc = q_win.cuda()
        prob = jacap.prepare(qc, k_cache, v_cache, offsets, [R + D] * B, jacap.Params(budget_k=R))
        slots = jacap.alloc_slots(prob, [R + D] * B)
        assert slots.shape[-1] == D
        jacap.run_evict_slots(prob, slots, qc, k_cache, v_cache)
        assert jacap.read_status(prob.ws) == 0
        torch.cuda.synchronize()
        nxt = make_case("ragged16", seq_lens=[D] * B, root=260908131 + 2000 + r, **spec)
        got_all = slots.cpu().numpy()
        for b in range(B):
            for l in range(L):
                for h in range(H):
                    qa = q_win[b, l, h * 2:(h + 1) * 2].to(torch.float64).numpy()
                    kk, vv = ok[(b, l, h)]
                    o = jo.evict_unit(qa, kk, vv, R)
                    want = np.setdiff1d(np.arange(R + D), o["idx"])
                    assert np.array_equal(got_all[b, l, h], want), (r, b, l, h)
                    _, nk, nv = nxt.unit_arrays(b, l, h)
                    kk, vv = kk.copy(), vv.copy()
                    kk[want], vv[want] = nk, nv
                    ok[(b, l, h)] = (kk, vv)
                    rows = torch.as_tensor(want + b * (R + D), device="cuda")
                    k_cache[l, h, rows] = nxt.k[l, h, b * D:(b + 1) * D].cuda()
                    v_cache[l, h, rows] = nxt.v[l, h, b * D:(b + 1) * D].cuda()
        q_win = nxt.q_win
        for (b, l, h), (kk, vv) in ok.items():
            lo = b * (R + D)
            np.testing.assert_array_equal(k_cache[l, h, lo:lo + R + D].double().cpu().numpy(), kk)
            np.testing.assert_array_equal(v_cache[l, h, lo:lo + R + D].double().cpu().numpy(), vv)
        del prob, slots


@pytest.mark.parametrize("gqa", ["pooled", "per_head"])
def test_dominant_token_keeps_its_weight(jacap, gqa):
    """At tau = 1 the planted sink takes nearly all of the centre softmax
    (1 - alpha ~ 1e-11): its weight rests on the rest of Z, which the chunk
    statistics keep apart from the maximum's own term (summed into it in fp32,
    it would vanish and the sink's score with it)."""
    case = make_case("ragged16", seq_lens=[256, 1025], num_layers=2, num_kv_heads=2,
                     num_q_heads=8, window=4, head_dim=64, dtype="bf16").to("cuda")
    check_case(case, 64, 1.0, "diag", tau=1.0, label=f"dominant token {gqa}", jacap=jacap,
               gqa=gqa)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("bf16", 64)])
def test_saturated_softmax_at_ridge_zero(jacap, dtype, d):
    """tau = 0.5: the centre softmax is saturated (1 - alpha of the sink and the
    other tokens' alpha near 1e-35), so the Eq. 8 weights fall far below fp32's
    range. At ridge 0 the leverage scores do not depend on the weights' common
    scale and stay O(1); the weight pass stores the weights times a power of
    two (the factorisation scales the ridge alike), so they must still match."""
    case = make_case("ragged16", seq_lens=[300, 4097], num_layers=1, num_kv_heads=2,
                     num_q_heads=4, window=16, head_dim=d, dtype=dtype).to("cuda")
    check_case(case, 64, 0.0, "diag", tau=0.5, label=f"saturated ridge 0 {dtype}",
               jacap=jacap)


@pytest.mark.parametrize("dtype,d,mode,gqa", [("bf16", 128, "diag", "pooled"),
                                              ("bf16", 128, "full", "per_head"),
                                              ("fp32", 64, "full", "pooled")])
def test_token_major_and_padded_layouts(jacap, dtype, d, mode, gqa):
    """The batch strides take other layouts than the default: K and V stored
    token-major ([L][T][H][d], viewed as [L][H][T][d]) and window queries with a
    padded row pitch (d + 8). Addressing only changes, so scores, selection and
    compaction must be bit-identical to the contiguous layout's."""
    case = make_case("ragged16", seq_lens=[0, 17, 300, 4100], num_layers=2, num_kv_heads=2,
                     num_q_heads=4, window=8, head_dim=d, dtype=dtype).to("cuda")
    p = jacap.Params(budget_k=64, cov_mode=COV[mode], protect_last=3,
                     gqa_mode=jacap.GQA_PER_HEAD if gqa == "per_head" else jacap.GQA_POOLED)
    ref = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    jacap.run_evict(ref, case.q_win, case.k, case.v)
    k_tm = case.k.permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
    v_tm = case.v.permute(0, 2, 1, 3).contiguous().permute(0, 2, 1, 3)
    qpad = torch.zeros(case.q_win.shape[:-1] + (d + 8,), dtype=case.q_win.dtype, device="cuda")
    qpad[..., :d] = case.q_win
    q_p = qpad[..., :d]
    assert k_tm.stride(2) == 2 * d and q_p.stride(3) == d + 8
    alt = jacap.prepare(q_p, k_tm, v_tm, case.seq_offsets, case.seq_lens, p)
    print(f"\n[layout] {dtype} d{d} {mode} {gqa}: token-major K/V, query pitch {d + 8}",
          flush=True)
    jacap.run_evict(alt, q_p, k_tm, v_tm)
    assert jacap.read_status(ref.ws) == 0 and jacap.read_status(alt.ws) == 0
    torch.cuda.synchronize()
    for b in range(len(case.seq_lens)):
        lo, hi = token_slice(case, b)
        assert torch.equal(alt.scores[:, :, lo:hi], ref.scores[:, :, lo:hi]), b
        kk = min(64, case.seq_lens[b])
        assert torch.equal(alt.k_out[b, :, :, :kk], ref.k_out[b, :, :, :kk]), b
        assert torch.equal(alt.v_out[b, :, :, :kk], ref.v_out[b, :, :, :kk]), b
    assert torch.equal(alt.idx, ref.idx)
    # retained rows written with a padded row pitch as well
    B, L, H = alt.idx.shape[:3]
    pad_k = torch.full((B, L, H, 64, d + 8), -3.0, dtype=case.k.dtype, device="cuda")
    pad_v = torch.full_like(pad_k, -3.0)
    k_o, v_o = pad_k[..., :d], pad_v[..., :d]
    jacap.set_out_strides(alt.batch, k_o)
    jacap.evict(alt.cfg, alt.batch, q_p, k_tm, v_tm, alt.scores, alt.idx, k_o, v_o, alt.ws)
    torch.cuda.synchronize()
    for b in range(len(case.seq_lens)):
        kk = min(64, case.seq_lens[b])
        assert torch.equal(k_o[b, :, :, :kk], ref.k_out[b, :, :, :kk]), b
        assert torch.equal(v_o[b, :, :, :kk], ref.v_out[b, :, :, :kk]), b
    assert torch.all(pad_k[..., d:] == -3.0) and torch.all(pad_v[..., d:] == -3.0)


@pytest.mark.parametrize("gqa", ["pooled", "per_head"])
def test_batch_without_tokens_is_a_no_op(jacap, gqa):
    """Every sequence empty: the K, V and score arrays have no elements (their
    tensors hold null data pointers), which the entry points accept; the
    selections are all padding and the greedy log det is d log(ridge)."""
    case = make_case("ragged16", seq_lens=[0, 0], num_layers=2, num_kv_heads=2, num_q_heads=4,
                     window=8, head_dim=64, dtype="bf16").to("cuda")
    assert case.k.numel() == 0
    p = jacap.Params(budget_k=16, ridge=0.5,
                     gqa_mode=jacap.GQA_PER_HEAD if gqa == "per_head" else jacap.GQA_POOLED)
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    prob.idx.fill_(7)
    jacap.run_evict(prob, case.q_win, case.k, case.v)
    jacap.score(prob.cfg, prob.batch, case.q_win, case.k, case.v, prob.scores, prob.ws)
    # compaction of an empty batch: null K, V, K' and V' are accepted and nothing is written
    jacap.compact(prob.cfg, prob.batch, prob.idx, case.k, case.v, case.k.new_empty(0),
                  case.v.new_empty(0))
    slots = jacap.alloc_slots(prob, case.seq_lens)
    slots.fill_(7)
    jacap.run_evict_slots(prob, slots, case.q_win, case.k, case.v)
    assert jacap.read_status(prob.ws) == 0
    torch.cuda.synchronize()
    assert torch.all(prob.idx == -1) and torch.all(slots == -1)
    if gqa == "pooled":
        g = jacap.prepare_greedy(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
        jacap.run_greedy(g, case.q_win, case.k, case.v)
        assert jacap.read_status(g.ws) == 0
        torch.cuda.synchronize()
        assert torch.all(g.idx == -1) and torch.all(g.order == -1)
        want = 64 * np.log(float(np.float32(0.5)))   # fp64 log of the fp32 ridge
        assert torch.allclose(g.logdet.cpu(), torch.full_like(g.logdet.cpu(), float(want)),
                              rtol=1e-12, atol=0)


def _sweep_specs(count=16, seed=2609):
    """Seeded random configurations across the supported envelope: head_dim,
    dtype, covariance, GQA group and mode, ridge, temperature, window (one
    query included), ragged lengths around the tile sizes (empty and one-token
    sequences included), budgets from 0 past every length, protected tails."""
    rng = np.random.default_rng(seed)
    lens_pool = [0, 1, 2, 15, 16, 17, 63, 255, 256, 257, 1000, 1025, 3000]
    specs = []
    for i in range(count):
        specs.append(dict(
            i=i, d=int(rng.choice([64, 128])), dtype=str(rng.choice(["bf16", "fp32"])),
            mode=str(rng.choice(["diag", "full"])), hkv=int(rng.choice([1, 2])),
            G=int(rng.choice([1, 2, 4])), gqa=str(rng.choice(["pooled", "per_head"])),
            ridge=float(rng.choice([1.0, 0.0078125, 0.05])), tau=float(rng.choice([1.0, 10.0])),
            window=int(rng.choice([1, 4, 8])),
            lens=[int(x) for x in rng.choice(lens_pool, int(rng.integers(1, 5)))],
            budget=int(rng.choice([0, 1, 16, 64, 300, 5000])),
            protect=int(rng.choice([0, 0, 3, 40]))))
    return specs


@pytest.mark.parametrize("spec", _sweep_specs() + [dict(sp, i=100 * (r + 1) + sp["i"])
                                                   for r, sd in enumerate((131, 977))
                                                   for sp in _sweep_specs(seed=sd)],
                         ids=lambda s: f"sweep{s['i']}")
def test_random_configuration_sweep(jacap, spec):
    s = spec
    print(f"\n[sweep] {s}", flush=True)
    case = make_case("ragged16", seq_lens=s["lens"], num_layers=2, num_kv_heads=s["hkv"],
                     num_q_heads=s["hkv"] * s["G"], window=s["window"], head_dim=s["d"],
                     dtype=s["dtype"]).to("cuda")
    check_case(case, s["budget"], s["ridge"], s["mode"], tau=s["tau"], label=f"sweep{s['i']}",
               jacap=jacap, gqa=s["gqa"], protect_last=s["protect"])


# ---------------------------------------------------------------------------
# Output-projection variant: u_i = W~ v_i through the ridge matrix R
# ---------------------------------------------------------------------------

def wo_ridge_matrices(case, d_model_factor=4):
    """R = (W~^T W~)^{-1} per (layer, KV head) from the seeded synthetic W_O,
    computed by the oracle in fp64 (an input of the GPU call)."""
    w = case.workload
    d, G = w.head_dim, w.num_q_heads // w.num_kv_heads
    wo = make_output_projection(w, d_model=d_model_factor * d).numpy()
    R = np.empty((w.num_layers, w.num_kv_heads, d, d))
    for layer in range(w.num_layers):
        for h in range(w.num_kv_heads):
            R[layer, h] = jo.output_ridge_matrix(jo.group_output_projection(wo[layer], h, G, d))
    return R


def _sweep2_specs(count=16):
    """A second seeded sweep, toward the edges: ridge 0 and the output-projection
    ridge matrices, temperatures 0.5 to 30, pooled windows up to 512 queries
    (the FULL MFMA K pass and the VALU one past 256), groups of 8, lengths at
    the K-pass, Gram and leverage chunk boundaries, budgets at those lengths."""
    rng = np.random.default_rng(8131)
    lens_pool = [0, 1, 1023, 1024, 1025, 2047, 4095, 4096, 4097, 6000]
    specs = []
    for i in range(count):
        specs.append(dict(
            i=i, d=int(rng.choice([64, 128])), dtype=str(rng.choice(["bf16", "fp32"])),
            mode=str(rng.choice(["diag", "full"])), hkv=int(rng.choice([1, 2])),
            G=int(rng.choice([1, 2, 4, 8])), gqa=str(rng.choice(["pooled", "per_head"])),
            ridge=str(rng.choice(["0", "1", "0.25", "wo"])),
            tau=float(rng.choice([0.5, 3.0, 10.0, 30.0])),
            window=int(rng.choice([1, 2, 16, 32, 64])),
            lens=[int(x) for x in rng.choice(lens_pool, int(rng.integers(1, 4)))],
            budget=int(rng.choice([0, 2, 100, 1023, 1024, 4096, 1 << 20])),
            protect=int(rng.choice([0, 1, 64]))))
    return specs


def _sweep3_specs(count=8):
    """A third seeded sweep over long units on the bf16 MFMA path: lengths
    around 8192, 16384 and 32768 (several K-pass, Gram and leverage chunks,
    ragged tails), both covariances and GQA modes, ridge 1, 0 and R."""
    rng = np.random.default_rng(20260908)
    lens_pool = [8191, 8192, 8193, 16385, 20000, 33000]
    specs = []
    for i in range(count):
        specs.append(dict(
            i=i, d=int(rng.choice([64, 128, 128])), dtype="bf16",
            mode=str(rng.choice(["diag", "full"])), hkv=int(rng.choice([1, 2])),
            G=int(rng.choice([1, 4])), gqa=str(rng.choice(["pooled", "per_head"])),
            ridge=str(rng.choice(["0", "1", "wo"])), tau=float(rng.choice([1.0, 10.0])),
            window=int(rng.choice([8, 32])),
            lens=[int(x) for x in rng.choice(lens_pool, int(rng.integers(1, 3)))],
            budget=int(rng.choice([256, 4096, 20000])), protect=int(rng.choice([0, 128]))))
    return specs


@pytest.mark.parametrize("spec", _sweep3_specs(), ids=lambda s: f"long{s['i']}")
def test_random_configuration_sweep_long_units(jacap, spec):
    s = spec
    print(f"\n[sweep long] {s}", flush=True)
    case = make_case("ragged16", seq_lens=s["lens"], num_layers=1, num_kv_heads=s["hkv"],
                     num_q_heads=s["hkv"] * s["G"], window=s["window"], head_dim=s["d"],
                     dtype=s["dtype"]).to("cuda")
    R = wo_ridge_matrices(case) if s["ridge"] == "wo" else None
    ridge = 1.0 if s["ridge"] == "wo" else float(s["ridge"])
    check_case(case, s["budget"], ridge, s["mode"], tau=s["tau"], label=f"long{s['i']}",
               jacap=jacap, gqa=s["gqa"], protect_last=s["protect"], ridge_matrices=R)


@pytest.mark.parametrize("spec", _sweep2_specs(), ids=lambda s: f"edge{s['i']}")
def test_random_configuration_sweep_edges(jacap, spec):
    s = spec
    print(f"\n[sweep edges] {s}", flush=True)
    case = make_case("ragged16", seq_lens=s["lens"], num_layers=1, num_kv_heads=s["hkv"],
                     num_q_heads=s["hkv"] * s["G"], window=s["window"], head_dim=s["d"],
                     dtype=s["dtype"]).to("cuda")
    R = wo_ridge_matrices(case) if s["ridge"] == "wo" else None
    ridge = 1.0 if s["ridge"] == "wo" else float(s["ridge"])
    check_case(case, s["budget"], ridge, s["mode"], tau=s["tau"], label=f"edge{s['i']}",
               jacap=jacap, gqa=s["gqa"], protect_last=s["protect"], ridge_matrices=R)



@pytest.mark.parametrize("mode", ["diag", "full"])
def test_wo_variant_tiny_fp32(jacap, mode):
    case = make_case("tiny").to("cuda")
    R = wo_ridge_matrices(case)
    check_case(case, 64, 1.0, mode, label=f"tiny W_O {mode}", jacap=jacap, ridge_matrices=R)


def test_wo_variant_llama_layer_bf16(jacap):
    case = make_case("llama8b_layer", seq_lens=[4096], device="cuda")
    R = wo_ridge_matrices(case)
    check_case(case, 512, 1.0, "diag", label="llama_layer W_O", jacap=jacap, ridge_matrices=R)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("fp32", 64)])
def test_wo_variant_ragged(jacap, dtype, d):
    case = make_case("ragged16", seq_lens=[0, 1, 17, 300, 1000, 4100], num_layers=2,
                     num_kv_heads=2, num_q_heads=4, window=8, head_dim=d, dtype=dtype).to("cuda")
    R = wo_ridge_matrices(case)
    check_case(case, 64, 1.0, "diag", label=f"ragged W_O {dtype} d{d}", jacap=jacap,
               ridge_matrices=R)


# ---------------------------------------------------------------------------
# Per-query-head GQA scoring and the protected tail
# ---------------------------------------------------------------------------

def test_per_head_gqa_llama_layer_bf16(jacap):
    case = make_case("llama8b_layer", seq_lens=[4096], device="cuda")
    check_case(case, 512, 1.0, "diag", label="llama_layer per-head GQA", jacap=jacap,
               gqa="per_head")


@pytest.mark.parametrize("dtype,d,mode,hq,hkv", [("bf16", 128, "diag", 4, 2),
                                                 ("fp32", 64, "full", 4, 2),
                                                 ("bf16", 128, "full", 4, 2),
                                                 ("bf16", 64, "diag", 6, 2),
                                                 ("bf16", 128, "diag", 8, 1)])
def test_per_head_gqa_ragged(jacap, dtype, d, mode, hq, hkv):
    """Every query head scored as a unit of its own in one pass (groups of 2, 3
    and 8 heads; the grid's padding past the last (unit, chunk) pair)."""
    case = make_case("ragged16", seq_lens=[0, 1, 17, 300, 1000, 4100], num_layers=2,
                     num_kv_heads=hkv, num_q_heads=hq, window=8, head_dim=d,
                     dtype=dtype).to("cuda")
    check_case(case, 64, 1.0, mode, label=f"ragged per-head {dtype} d{d} G{hq // hkv}",
               jacap=jacap, gqa="per_head")


@pytest.mark.parametrize("protect", [0, 7, 64, 100])
def test_protect_last_evict(jacap, protect):
    case = make_case("ragged16", seq_lens=[0, 5, 64, 300, 9000], num_layers=1, num_kv_heads=2,
                     num_q_heads=2, window=8, head_dim=64, dtype="bf16").to("cuda")
    check_case(case, 64, 1.0, "diag", label=f"protect_last {protect}", jacap=jacap,
               protect_last=protect)


# ---------------------------------------------------------------------------
# Decoding-stage eviction: evict -> append new tokens -> evict, several rounds
# ---------------------------------------------------------------------------

def test_decode_rounds_follow_the_oracle_chain(jacap):
    """A cache of R reserved + D new tokens per sequence is evicted back to R
    each round; the retained rows plus the next D tokens (and a new window)
    form the next round's cache. The GPU chain and the oracle's own chain must
    keep the same positions in every round (the caches then stay identical)."""
    R, D, B, rounds = 256, 32, 2, 3
    spec = dict(num_layers=1, num_kv_heads=2, num_q_heads=4, window=8, head_dim=64, dtype="bf16")
    L, H = spec["num_layers"], spec["num_kv_heads"]
    first = make_case("ragged16", seq_lens=[R + D] * B, **spec)
    k_cache, v_cache = first.k.clone(), first.v.clone()        # CPU tensors, packed
    ok = {(b, l, h): (first.unit_arrays(b, l, h)[1], first.unit_arrays(b, l, h)[2])
          for b in range(B) for l in range(L) for h in range(H)}
    q_win = first.q_win
    offsets = torch.tensor([i * (R + D) for i in range(B + 1)], dtype=torch.int32)
    for r in range(rounds):
        print(f"[decode] round {r}", flush=True)
        p = jacap.Params(budget_k=R)
        kc, vc, qc = k_cache.cuda(), v_cache.cuda(), q_win.cuda()
        prob = jacap.prepare(qc, kc, vc, offsets.cuda(), [R + D] * B, p)
        jacap.run_evict(prob, qc, kc, vc)
        assert jacap.read_status(prob.ws) == 0
        torch.cuda.synchronize()
        nxt = make_case("ragged16", seq_lens=[D] * B, root=260908131 + 1000 + r, **spec)
        new_k, new_v = [], []
        for b in range(B):
            for l in range(L):
                for h in range(H):
                    qa = q_win[b, l, h * 2:(h + 1) * 2].to(torch.float64).numpy()
                    kk, vv = ok[(b, l, h)]
                    o = jo.evict_unit(qa, kk, vv, R)
                    got = prob.idx[b, l, h].cpu().numpy()
                    assert np.array_equal(got, o["idx"]), (r, b, l, h)
                    _, nk, nv = nxt.unit_arrays(b, l, h)
                    ok[(b, l, h)] = (np.concatenate([o["k_out"], nk]), np.concatenate([o["v_out"], nv]))
            new_k.append(torch.cat([prob.k_out[b].cpu(), nxt.k[:, :, b * D:(b + 1) * D]], dim=2))
            new_v.append(torch.cat([prob.v_out[b].cpu(), nxt.v[:, :, b * D:(b + 1) * D]], dim=2))
        k_cache = torch.cat(new_k, dim=2).contiguous()
        v_cache = torch.cat(new_v, dim=2).contiguous()
        q_win = nxt.q_win
        # the GPU cache and the oracle cache hold the same rows
        for (b, l, h), (kk, vv) in ok.items():
            lo = b * (R + D)
            np.testing.assert_array_equal(k_cache[l, h, lo:lo + R + D].to(torch.float64).numpy(), kk)
