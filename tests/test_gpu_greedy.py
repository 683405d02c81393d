"""GPU parity of the exact greedy log-det selection (jacap_greedy) against the
fp64 oracle greedy (App. B.1).

The GPU computes its gains from its own fp32 Eq. 8 weights, the oracle from
fp64 ones, so two candidates whose gains agree to within that rounding may be
taken in either order. Per unit the test therefore checks:
* the pick order is a valid greedy path under the oracle: replayed in fp64,
  every pick's gain is within GAIN_TOL (relative) of the best gain available
  at that step (and exactly the best when no near-tie exists, which the
  prefix-agreement report shows);
* idx holds the same positions ascending, -1 padding; order is -1 padded;
* logdet equals log det(ridge I + sum_C w u u^T) of the chosen set under the
  oracle weights, to GAIN_TOL of its data-dependent part;
* the protected tail comes first, in position order.
"""

import numpy as np
import pytest
import torch

from jacap_synth import make_case
from oracle import jacap_oracle as jo

from helpers import token_slice, unit_list

pytestmark = pytest.mark.gpu

# Relative gain tolerance: the weights' own error (fp32 logits and query
# responses, fp32 storage) is ~1e-6 relative; the scores' bf16 bound is 1e-3.
GAIN_TOL = {"bf16": 1e-4, "fp32": 1e-5}


@pytest.fixture(scope="module")
def jacap():
    from paper_2609_08131_amd import jacap as j
    return j


def run_greedy(jacap, case, budget, ridge=1.0, tau=10.0, protect_last=0, cov_mode=0):
    p = jacap.Params(budget_k=budget, temperature=tau, ridge=ridge, cov_mode=cov_mode,
                     protect_last=protect_last)
    prob = jacap.prepare_greedy(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    jacap.run_greedy(prob, case.q_win, case.k, case.v)
    flags = jacap.read_status(prob.ws)
    torch.cuda.synchronize()
    return prob, flags


def check_greedy(jacap, case, budget, ridge=1.0, units=None, protect_last=0, label="",
                 cov_mode="diag", tau=10.0):
    units = unit_list(case) if units is None else units
    prob, flags = run_greedy(jacap, case, budget, ridge=ridge, tau=tau, protect_last=protect_last,
                             cov_mode={"diag": 0, "full": 1}[cov_mode])
    assert flags == 0, flags
    tol = GAIN_TOL[case.workload.dtype]
    ridge32 = float(np.float32(ridge))
    agree, worst = [], 0.0
    for (b, l, h) in units:
        n = case.seq_lens[b]
        kk = min(budget, n)
        pp = min(protect_last, kk)
        q, k, v = case.unit_arrays(b, l, h)
        o = jo.score_unit(q, k, v, tau=tau, ridge=ridge32, cov_mode=cov_mode)
        w = o["w"] if n else np.zeros(0)
        order = prob.order[b, l, h].cpu().numpy()
        idx = prob.idx[b, l, h].cpu().numpy()
        got = order[:kk]
        assert np.all(order[kk:] == -1) and np.all(idx[kk:] == -1), (label, (b, l, h))
        assert len(set(got.tolist())) == kk and np.all((got >= 0) & (got < n)), (label, (b, l, h))
        assert np.array_equal(idx[:kk], np.sort(got)), (label, (b, l, h))
        assert got[:pp].tolist() == list(range(n - pp, n)), (label, (b, l, h))
        ld = float(prob.logdet[b, l, h])
        d = case.workload.head_dim
        if kk == 0:
            assert abs(ld - d * np.log(ridge32)) <= 1e-12 * max(1.0, abs(d * np.log(ridge32)))
            agree.append(1.0)
            continue
        chosen, best = jo.greedy_replay(v, w, ridge32, got, protect_last=pp)
        rel = (best - chosen) / np.maximum(np.abs(best), 1e-300)
        worst = max(worst, float(rel.max()))
        assert rel.max() <= tol, (label, (b, l, h), float(rel.max()), int(rel.argmax()))
        ref = jo.greedy_logdet(v, w, ridge32, budget, protect_last=pp)
        same = np.nonzero(ref != got)[0]
        agree.append((same[0] if len(same) else kk) / kk)
        obj = jo.logdet_objective(v, w, ridge32, got)
        base = d * np.log(ridge32)
        assert abs(ld - obj) <= tol * abs(obj - base) + 1e-9 * max(1.0, abs(base)), \
            (label, (b, l, h), ld, obj)
    print(f"\n[greedy] {label}: worst replay gain gap {worst:.2e} (tol {tol:g}); "
          f"identical-prefix fraction min {min(agree):.3f} mean {np.mean(agree):.3f}")
    return prob


def test_greedy_tiny_fp32(jacap):
    case = make_case("tiny", device="cuda")
    prob = check_greedy(jacap, case, 64, label="tiny fp32")
    # fp32 inputs: no near-ties expected at this size; the whole order agrees
    q, k, v = case.unit_arrays(0, 0, 0)
    w = jo.score_unit(q, k, v)["w"]
    assert np.array_equal(prob.order[0, 0, 0].cpu().numpy(), jo.greedy_logdet(v, w, 1.0, 64))


@pytest.mark.parametrize("ridge", [1.0, 2.0 ** -12])
def test_greedy_llama_layer_bf16(jacap, ridge):
    """n = 8192, d = 128, B = 512, 8 KV heads; ridge 2^-12 makes the diversity
    term matter (many refreshes per pick)."""
    case = make_case("llama8b_layer", device="cuda")
    check_greedy(jacap, case, 512, ridge=ridge, label=f"llama8b_layer ridge {ridge:g}")


@pytest.mark.parametrize("protect", [0, 5, 64])
def test_greedy_ragged_protected(jacap, protect):
    """Ragged lengths with a ragged tail block, fp32 and d = 64, protected tail."""
    case = make_case("ragged16", device="cuda", seq_lens=(700, 1, 1300),
                     num_layers=1, num_kv_heads=2, head_dim=64, dtype="fp32")
    check_greedy(jacap, case, 96, ridge=0.5, protect_last=protect, label=f"ragged protect {protect}")


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("fp32", 64)])
def test_greedy_saturated_softmax(jacap, dtype, d):
    """tau = 0.5: the Eq. 8 weights (~1e-70) lie far outside fp32; they are
    stored times a per-unit power of two and A_0 = ridge I takes the same
    factor, so the gains w_i c_i, the picks and the log det are unchanged."""
    case = make_case("ragged16", device="cuda", seq_lens=(300, 2100), num_layers=1,
                     num_kv_heads=2, num_q_heads=4, window=16, head_dim=d, dtype=dtype)
    check_greedy(jacap, case, 64, ridge=1.0, tau=0.5, label=f"saturated {dtype}")


def test_greedy_budget_edges(jacap):
    """Budget >= n takes every position; budget 0 writes nothing but logdet."""
    case = make_case("ragged16", device="cuda", seq_lens=(300, 40), num_layers=1,
                     num_kv_heads=1, head_dim=128, dtype="bf16")
    check_greedy(jacap, case, 300, label="budget >= n")
    prob, flags = run_greedy(jacap, case, 0)
    assert flags == 0
    assert torch.allclose(prob.logdet.cpu(), torch.full((2, 1, 1), 0.0, dtype=torch.float64))


def test_greedy_full_covariance(jacap):
    case = make_case("ragged16", device="cuda", seq_lens=(2000,), num_layers=2,
                     num_kv_heads=2, head_dim=128, dtype="bf16")
    check_greedy(jacap, case, 128, cov_mode="full", label="full covariance")


def test_greedy_full_covariance_triangular_path(jacap):
    """FULL covariance with N_s = 2d pooled window queries and a unit of 9000
    tokens: the greedy picks run on weights whose kappa comes from the
    triangular factor of Lambda_Q (the eviction path's launches); the 700-token
    units take the window tile."""
    case = make_case("ragged16", device="cuda", seq_lens=(9000, 700), num_layers=1,
                     num_kv_heads=2, num_q_heads=8, window=32, head_dim=64, dtype="bf16")
    check_greedy(jacap, case, 96, cov_mode="full", label="full covariance, triangular path")


def test_greedy_deterministic(jacap):
    case = make_case("llama8b_layer", device="cuda")
    a, _ = run_greedy(jacap, case, 512)
    o1, l1 = a.order.clone(), a.logdet.clone()
    jacap.run_greedy(a, case.q_win, case.k, case.v)
    torch.cuda.synchronize()
    assert torch.equal(a.order, o1) and torch.equal(a.logdet, l1)


def test_greedy_prefill_units_bf16(jacap):
    """n = 32768, B = 512, three sampled units of a 32-layer cache."""
    case = make_case("prefill32k", device="cuda")
    check_greedy(jacap, case, 512, units=[(0, 0, 0), (0, 13, 5), (0, 31, 7)],
                 label="prefill32k sampled")


@pytest.mark.parametrize("ridge", [1.0, 2.0 ** -12])
def test_greedy_vs_leverage_quality_report(jacap, ridge):
    """The comparator's purpose: the log-det objective of Jacap's one-shot
    TOP-B (leverage) selection against the exact greedy's, on the same weights
    (oracle fp64), for sampled prefill32k units. Reported, not asserted beyond
    sanity: greedy is a (1 - 1/e)-approximation, not an upper bound."""
    case = make_case("prefill32k", device="cuda")
    budget = 512
    prob, flags = run_greedy(jacap, case, budget, ridge=ridge)
    assert flags == 0
    d = case.workload.head_dim
    rows = []
    for (b, l, h) in [(0, 0, 0), (0, 7, 3), (0, 15, 1), (0, 23, 6), (0, 31, 7)]:
        q, k, v = case.unit_arrays(b, l, h)
        o = jo.evict_unit(q, k, v, budget, ridge=ridge)
        base = d * np.log(ridge)
        lev = jo.logdet_objective(v, o["w"], ridge, o["idx"]) - base
        grd = float(prob.logdet[b, l, h]) - base
        gset = prob.idx[b, l, h].cpu().numpy()
        ov = len(set(gset.tolist()) & set(o["idx"].tolist())) / budget
        assert lev > 0 and grd > 0
        rows.append((lev / grd, ov))
    r = np.array(rows)
    print(f"\n[quality] prefill32k ridge {ridge:g} B={budget}: leverage/greedy log-det gain "
          f"min {r[:, 0].min():.4f} mean {r[:, 0].mean():.4f}; set overlap mean {r[:, 1].mean():.3f}")


def test_greedy_long128k_full_batch(jacap):
    """The comparator on the full long128k batch (256 units x 131072 tokens,
    B = 1024): every unit's output is a valid selection, and one sampled unit's
    pick order is replayed through the fp64 oracle."""
    case = make_case("long128k", device="cuda")
    budget = case.workload.budget_k
    prob, flags = run_greedy(jacap, case, budget)
    assert flags == 0, flags
    n = case.seq_lens[0]
    idx, order = prob.idx[0], prob.order[0]                # [L][H][B]
    assert torch.all(idx >= 0) and torch.all(idx < n)
    assert torch.all(torch.diff(idx, dim=-1) > 0)
    assert torch.equal(torch.sort(order, dim=-1).values, idx)
    assert torch.isfinite(prob.logdet).all() and (prob.logdet > 0).all()   # ridge 1: log det > 0
    l, h = 19, 5
    q, k, v = case.unit_arrays(0, l, h)
    w = jo.score_unit(q, k, v)["w"]
    got = order[l, h].cpu().numpy()
    chosen, best = jo.greedy_replay(v, w, 1.0, got)
    rel = (best - chosen) / np.abs(best)
    assert rel.max() <= GAIN_TOL["bf16"], float(rel.max())
    ref = jo.greedy_logdet(v, w, 1.0, budget)
    diff = np.nonzero(ref != got)[0]
    print(f"\n[greedy] long128k unit (0, {l}, {h}): worst replay gap {rel.max():.2e}; "
          f"identical prefix {(diff[0] if len(diff) else budget)} of {budget}", flush=True)
    del prob, case
    torch.cuda.empty_cache()


def _greedy_sweep_specs(count=8):
    """Seeded random configurations of the greedy comparator: head_dim, dtype,
    covariance, ridge > 0, temperature, ragged lengths around its 256-position
    blocks, budgets from 0 past every length, protected tails."""
    rng = np.random.default_rng(41)
    pool = [0, 1, 255, 256, 257, 700, 1500]
    return [dict(i=i, d=int(rng.choice([64, 128])), dtype=str(rng.choice(["bf16", "fp32"])),
                 mode=str(rng.choice(["diag", "full"])), ridge=float(rng.choice([1.0, 0.05, 2.0 ** -10])),
                 tau=float(rng.choice([1.0, 10.0])),
                 lens=[int(x) for x in rng.choice(pool, int(rng.integers(1, 4)))],
                 budget=int(rng.choice([0, 1, 40, 300, 2000])), protect=int(rng.choice([0, 0, 9])))
            for i in range(count)]


@pytest.mark.parametrize("spec", _greedy_sweep_specs(), ids=lambda s: f"gsweep{s['i']}")
def test_greedy_configuration_sweep(jacap, spec):
    s = spec
    print(f"\n[greedy sweep] {s}", flush=True)
    case = make_case("ragged16", device="cuda", seq_lens=s["lens"], num_layers=1,
                     num_kv_heads=2, num_q_heads=4, window=8, head_dim=s["d"], dtype=s["dtype"])
    check_greedy(jacap, case, s["budget"], ridge=s["ridge"], protect_last=s["protect"],
                 cov_mode=s["mode"], tau=s["tau"], label=f"gsweep{s['i']}")
