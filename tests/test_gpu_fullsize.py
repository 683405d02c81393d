"""Full-size workloads in the benchmark's launch configuration.

Every unit (sequence, layer, KV head) is scored in one jacap_evict call at the
real shape. For prefill32k (budgets 128 and 2048), long128k (ridge 1 and 0;
FULL covariance at ridge 1) and ragged16 every unit is checked against the fp64 oracle (run in parallel
worker processes): every score within the bf16 tolerance, jacap_select on the
oracle's fp32 scores bit-equal to the oracle's selection, the GPU selection
equal to the select rule on the GPU's own scores, and the overlap of the GPU's
selection with the oracle's reported. The other full-size runs check sampled
units against the oracle, plus properties that hold at any size on every unit:
  * ridge > 0: every score lies in [0, 1) (ridge leverage, Eq. 10 with A >= ridge I);
  * the selection is ascending, in range, with -1 padding exactly past min(k, n);
  * K', V' are exact gathers (sampled units).
"""

import gc
import time

import numpy as np
import pytest
import torch

from jacap_synth import make_case
from oracle import jacap_oracle as jo

from helpers import (BF16_TOL, gpu_unit_idx, gpu_unit_scores, oracle_unit, overlap, run_gpu,
                     score_errors, token_slice)
from oracle_pool import oracle_all_units

pytestmark = pytest.mark.gpu


def _free():
    gc.collect()
    torch.cuda.empty_cache()


def _check_all_units_properties(case, prob, budget, ridge):
    for b, n in enumerate(case.seq_lens):
        kk = min(budget, n)
        sub = prob.idx[b]                                    # [L][H][budget]
        assert torch.all(sub[..., kk:] == -1)
        v = sub[..., :kk]
        if kk:
            assert torch.all(v >= 0) and torch.all(v < n)
            assert torch.all(torch.diff(v, dim=-1) > 0)
    if ridge > 0:
        s = prob.scores
        assert torch.isfinite(s).all()
        assert (s >= 0).all() and (s < 1).all()


def _sample_units(case, count=3):
    w = case.workload
    total = case.num_seqs * w.num_layers * w.num_kv_heads
    picks = sorted(set([0, total - 1, total // 2, (7 * total) // 11][:count + 1]))
    out = []
    for u in picks:
        h = u % w.num_kv_heads
        l = (u // w.num_kv_heads) % w.num_layers
        b = u // (w.num_kv_heads * w.num_layers)
        if case.seq_lens[b] > 0:
            out.append((b, l, h))
    return out


def _check_sampled(case, prob, budget, ridge, label, mode="diag", gqa="pooled"):
    worst, ovs = 0.0, []
    for (b, l, h) in _sample_units(case):
        o = oracle_unit(case, b, l, h, budget, ridge=ridge, cov_mode=mode, gqa=gqa)
        g = gpu_unit_scores(case, prob, b, l, h)
        err = score_errors(g, o["scores"])
        worst = max(worst, float(err.max()))
        assert err.max() <= BF16_TOL, (label, (b, l, h), float(err.max()))
        idx = gpu_unit_idx(case, prob, b, l, h, budget)
        assert np.array_equal(idx, jo.select_top(g.astype(np.float32), budget))
        ovs.append(overlap(idx, o["idx"]))
        lo, _ = token_slice(case, b)
        sel = torch.as_tensor(idx.astype(np.int64), device="cuda") + lo
        assert torch.equal(prob.k_out[b, l, h, :len(idx)], case.k[l, h, sel])
        assert torch.equal(prob.v_out[b, l, h, :len(idx)], case.v[l, h, sel])
    print(f"\n[fullsize] {label} ridge={ridge:g}: worst rel err {worst:.3e}, "
          f"overlap with oracle selection {np.round(ovs, 4).tolist()}", flush=True)


def _check_every_unit(case, probs, ridge, label, select_budgets, cov_mode="diag"):
    """Every unit against the oracle. probs: {budget: GPU problem after
    jacap_evict}; the scores do not depend on the budget, so those of the
    first are compared. For the budgets in select_budgets, jacap_select runs
    on the oracle's fp32 scores and must reproduce the oracle's selection."""
    from paper_2609_08131_amd import jacap
    budgets = list(probs)
    first = probs[budgets[0]]
    gsc = first.scores.cpu()
    gidx = {bud: p.idx.cpu() for bud, p in probs.items()}
    ref32 = torch.zeros_like(gsc)
    orc_idx = {}
    worst, worst_unit, ovs = 0.0, None, {bud: [] for bud in budgets}
    t0 = time.time()
    count = 0
    for (b, l, h, s32, idx, singular) in oracle_all_units(case, budgets=budgets, ridge=ridge,
                                                          cov_mode=cov_mode):
        assert not singular, (label, (b, l, h))
        lo, hi = token_slice(case, b)
        g = gsc[l, h, lo:hi].double().numpy()
        ref32[l, h, lo:hi] = torch.from_numpy(s32)
        # the oracle's fp64 scores rounded once to fp32: within 2^-24 of them
        err = score_errors(g, s32.astype(np.float64))
        e = float(err.max()) if err.size else 0.0
        if e > worst:
            worst, worst_unit = e, (b, l, h)
        assert e <= BF16_TOL - 2.0 ** -23, (label, (b, l, h), e, int(err.argmax()))
        n = hi - lo
        for bud in budgets:
            kk = min(bud, n)
            row = gidx[bud][b, l, h].numpy()
            assert np.all(row[kk:] == -1)
            assert np.array_equal(row[:kk], jo.select_top(g.astype(np.float32), bud)), \
                (label, bud, (b, l, h))
            ovs[bud].append(overlap(row[:kk], idx[bud]) if kk else 1.0)
        for bud in select_budgets:
            orc_idx[(b, l, h, bud)] = idx[bud]
        count += 1
    w = case.workload
    assert count == case.num_seqs * w.num_layers * w.num_kv_heads
    for bud in select_budgets:
        p = probs[bud]
        idx2 = torch.empty_like(p.idx)
        jacap.select(p.cfg, p.batch, ref32.to(p.scores.device), idx2)
        torch.cuda.synchronize()
        idx2 = idx2.cpu()
        for (b, l, h, bb), o_idx in orc_idx.items():
            if bb != bud:
                continue
            kk = len(o_idx)
            got = idx2[b, l, h].numpy()
            assert np.array_equal(got[:kk], o_idx), ("select on oracle scores", label, bud, (b, l, h))
            assert np.all(got[kk:] == -1)
    ovtxt = ", ".join(f"k={bud}: min {min(v):.4f} mean {np.mean(v):.4f}" for bud, v in ovs.items())
    print(f"\n[fullsize] {label} ridge={ridge:g}: all {count} units, worst rel err {worst:.3e} "
          f"at {worst_unit}; jacap_select on the oracle's scores bit-exact at k in "
          f"{list(select_budgets)}; overlap of the GPU selection with the oracle's: {ovtxt} "
          f"(oracle {time.time() - t0:.0f} s)", flush=True)


def test_prefill32k_budget_sweep():
    case = make_case("prefill32k", device="cuda")
    probs = {}
    for budget in case.workload.budget_sweep:
        prob, flags = run_gpu(case, budget, ridge=1.0)
        assert flags == 0
        _check_all_units_properties(case, prob, budget, 1.0)
        if budget in (128, 2048):
            probs[budget] = prob
        else:
            del prob
    _check_every_unit(case, probs, 1.0, "prefill32k", select_budgets=(128, 2048))
    del probs, case
    _free()


@pytest.mark.parametrize("ridge", [1.0, 0.0])
def test_long128k(ridge):
    case = make_case("long128k", device="cuda")
    budget = case.workload.budget_k
    prob, flags = run_gpu(case, budget, ridge=ridge)
    assert flags == 0
    _check_all_units_properties(case, prob, budget, ridge)
    _check_every_unit(case, {budget: prob}, ridge, "long128k", select_budgets=(budget,))
    del prob, case
    _free()


def test_ragged16():
    case = make_case("ragged16", device="cuda")
    budget = case.workload.budget_k
    prob, flags = run_gpu(case, budget, ridge=1.0)
    assert flags == 0
    _check_all_units_properties(case, prob, budget, 1.0)
    _check_every_unit(case, {budget: prob}, 1.0, "ragged16", select_budgets=(budget,))
    del prob, case
    _free()


def test_per_head_gqa_long128k():
    """Per-head GQA at full size: the G = 4 query heads of every KV head scored
    as units of their own in one launch, sampled units against the oracle."""
    case = make_case("long128k", device="cuda")
    budget = case.workload.budget_k
    prob, flags = run_gpu(case, budget, ridge=1.0, gqa="per_head")
    assert flags == 0
    _check_all_units_properties(case, prob, budget, 1.0)
    _check_sampled(case, prob, budget, 1.0, "long128k per-head", gqa="per_head")
    del prob, case
    _free()


@pytest.mark.parametrize("wl", ["prefill32k", "long128k"])
def test_full_covariance_fullsize(wl):
    """FULL covariance at full size. prefill32k (N_s = 128 pooled window
    queries) takes the window tile: sampled units against the oracle,
    properties on all. long128k (N_s = 256 = 2 d, 131072 tokens) takes kappa
    from the triangular factor of Lambda_Q: every unit against the oracle."""
    case = make_case(wl, device="cuda")
    budget = case.workload.budget_k
    prob, flags = run_gpu(case, budget, cov_mode=1)
    assert flags == 0, flags
    _check_all_units_properties(case, prob, budget, 1.0)
    if wl == "long128k":
        _check_every_unit(case, {budget: prob}, 1.0, f"{wl} full", select_budgets=(),
                          cov_mode="full")
    else:
        _check_sampled(case, prob, budget, 1.0, f"{wl} full", mode="full")
    del prob
    del case
    _free()


def test_decode16k():
    """Decoding-stage eviction at its bench shape: 16 sequences x 32 layers x 8
    KV heads of 16512 tokens, budget 16384. The budget keeps more than half of
    every unit, so selection ranks the 128 evictions (the complement path)."""
    case = make_case("decode16k", device="cuda")
    budget = case.workload.budget_k
    prob, flags = run_gpu(case, budget)
    assert flags == 0, flags
    _check_all_units_properties(case, prob, budget, 1.0)
    _check_sampled(case, prob, budget, 1.0, "decode16k")
    del prob
    del case
    _free()


def test_single_unit_of_two_million_tokens():
    """The largest single unit exercised: 2^21 tokens (512 Gram chunks reduced
    in order, multi-million-token offsets, selection over 2M scores), every
    score against the oracle and the selection exact on the GPU's scores."""
    n = 1 << 21
    case = make_case("long128k", device="cuda", seq_lens=(n,), num_layers=1, num_kv_heads=1,
                     num_q_heads=4)
    budget = 4096
    print(f"[fullsize] single unit n={n}", flush=True)
    prob, flags = run_gpu(case, budget)
    assert flags == 0, flags
    o = oracle_unit(case, 0, 0, 0, budget)
    g = gpu_unit_scores(case, prob, 0, 0, 0)
    err = score_errors(g, o["scores"])
    idx = gpu_unit_idx(case, prob, 0, 0, 0, budget)
    assert np.array_equal(idx, jo.select_top(g.astype(np.float32), budget))
    sel = torch.as_tensor(idx.astype(np.int64), device="cuda")
    assert torch.equal(prob.k_out[0, 0, 0], case.k[0, 0, sel])
    assert torch.equal(prob.v_out[0, 0, 0], case.v[0, 0, sel])
    print(f"[fullsize] n={n}: worst rel err {err.max():.3e}; overlap with oracle selection "
          f"{overlap(idx, o['idx']):.4f}", flush=True)
    assert err.max() <= BF16_TOL
    del prob, case
    _free()


def test_greedy_at_its_length_limit():
    """jacap_greedy on one unit of 524288 tokens (its limit): a valid selection
    whose pick order replays through the fp64 oracle as greedy."""
    from paper_2609_08131_amd import jacap
    n = 524288
    case = make_case("long128k", device="cuda", seq_lens=(n,), num_layers=1, num_kv_heads=1,
                     num_q_heads=4)
    budget = 48
    p = jacap.Params(budget_k=budget)
    prob = jacap.prepare_greedy(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    jacap.run_greedy(prob, case.q_win, case.k, case.v)
    assert jacap.read_status(prob.ws) == 0
    order = prob.order[0, 0, 0].cpu().numpy()
    assert len(set(order.tolist())) == budget and order.min() >= 0 and order.max() < n
    assert np.array_equal(prob.idx[0, 0, 0].cpu().numpy(), np.sort(order))
    q, k, v = case.unit_arrays(0, 0, 0)
    w = jo.score_unit(q, k, v)["w"]
    chosen, best = jo.greedy_replay(v, w, 1.0, order)
    rel = (best - chosen) / np.abs(best)
    print(f"[greedy] n={n}: worst replay gap {rel.max():.2e}", flush=True)
    assert rel.max() <= 1e-4
    del prob, case
    _free()
