"""HIP graph capture of the eviction path, and concurrent calls on two streams.

jacap_evict only enqueues kernels on the caller's stream (no allocation, no
memset node, no host synchronisation; the per-unit flags are cleared by a
kernel), so a graph captured around it must replay the eager result bit for
bit. Every replay follows eager work on the same buffers (a fill of every
output) and a synchronisation, and is checked against the eager run.
"""

import pytest
import torch

from jacap_synth import make_case

from helpers import token_slice

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def jacap():
    from paper_2609_08131_amd import jacap as j
    return j


def _kept_rows_equal(case, prob, ref_k, ref_v, budget):
    for b, n in enumerate(case.seq_lens):
        kk = min(budget, n)
        assert torch.equal(prob.k_out[b, :, :, :kk], ref_k[b, :, :, :kk])
        assert torch.equal(prob.v_out[b, :, :, :kk], ref_v[b, :, :, :kk])


@pytest.mark.parametrize("gqa,protect", [("pooled", 0), ("per_head", 5)])
def test_evict_replays_from_a_graph(jacap, gqa, protect):
    case = make_case("ragged16", seq_lens=[0, 1, 17, 300, 1000, 4100], num_layers=2,
                     num_kv_heads=2, num_q_heads=4, window=8, head_dim=128,
                     dtype="bf16").to("cuda")
    budget = 64
    p = jacap.Params(budget_k=budget, ridge=1.0, protect_last=protect,
                     gqa_mode=jacap.GQA_PER_HEAD if gqa == "per_head" else jacap.GQA_POOLED)
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    print(f"\n[graph] {gqa} protect_last={protect}: eager run", flush=True)
    jacap.run_evict(prob, case.q_win, case.k, case.v)
    assert jacap.read_status(prob.ws) == 0
    torch.cuda.synchronize()
    ref_s, ref_i = prob.scores.clone(), prob.idx.clone()
    ref_k, ref_v = prob.k_out.clone(), prob.v_out.clone()

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            jacap.run_evict(prob, case.q_win, case.k, case.v)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    for rep in range(3):
        for t in (prob.scores, prob.k_out, prob.v_out):
            t.fill_(-7.0)
        prob.idx.fill_(-7)
        torch.cuda.synchronize()
        print(f"[graph] {gqa}: replay {rep}", flush=True)
        g.replay()
        torch.cuda.synchronize()
        assert jacap.read_status(prob.ws) == 0
        for b in range(len(case.seq_lens)):
            lo, hi = token_slice(case, b)
            torch.testing.assert_close(prob.scores[:, :, lo:hi], ref_s[:, :, lo:hi], rtol=0, atol=0,
                                       equal_nan=True)
        assert torch.equal(prob.idx, ref_i)
        _kept_rows_equal(case, prob, ref_k, ref_v, budget)
    del g


def test_greedy_replays_from_a_graph(jacap):
    case = make_case("ragged16", seq_lens=[0, 3, 300, 2100], num_layers=1, num_kv_heads=2,
                     num_q_heads=4, window=8, head_dim=64, dtype="bf16").to("cuda")
    p = jacap.Params(budget_k=48, ridge=1.0)
    prob = jacap.prepare_greedy(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    print("\n[graph] greedy: eager run", flush=True)
    jacap.run_greedy(prob, case.q_win, case.k, case.v)
    assert jacap.read_status(prob.ws) == 0
    torch.cuda.synchronize()
    ref = [t.clone() for t in (prob.idx, prob.order, prob.logdet)]

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            jacap.run_greedy(prob, case.q_win, case.k, case.v)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    for rep in range(3):
        prob.idx.fill_(-7)
        prob.order.fill_(-7)
        prob.logdet.fill_(-7.0)
        torch.cuda.synchronize()
        print(f"[graph] greedy: replay {rep}", flush=True)
        g.replay()
        torch.cuda.synchronize()
        assert jacap.read_status(prob.ws) == 0
        for t, r in zip((prob.idx, prob.order, prob.logdet), ref):
            torch.testing.assert_close(t, r, rtol=0, atol=0, equal_nan=True)
    del g


def test_concurrent_streams_with_distinct_workspaces(jacap):
    """Calls on different streams are independent when their workspaces are
    distinct: two eviction problems (different budgets, GQA modes and
    protected tails) launched back to back on two streams give the results of
    running them one after the other."""
    case = make_case("ragged16", seq_lens=[17, 300, 4100], num_layers=2, num_kv_heads=2,
                     num_q_heads=4, window=8, head_dim=128, dtype="bf16").to("cuda")
    params = [jacap.Params(budget_k=64), jacap.Params(budget_k=200, protect_last=7,
                                                       gqa_mode=jacap.GQA_PER_HEAD)]
    probs = [jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
             for p in params]
    for prob in probs:                       # one after the other, default stream
        jacap.run_evict(prob, case.q_win, case.k, case.v)
    torch.cuda.synchronize()
    ref = [(pr.scores.clone(), pr.idx.clone(), pr.k_out.clone()) for pr in probs]
    for pr in probs:
        pr.scores.fill_(-7.0)
        pr.idx.fill_(-7)
        pr.k_out.fill_(-7.0)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for rep in range(3):
        print(f"\n[streams] concurrent run {rep}", flush=True)
        for st in streams:
            st.wait_stream(torch.cuda.current_stream())
        for pr, st in zip(probs, streams):
            jacap.run_evict(pr, case.q_win, case.k, case.v, st)
        for st in streams:
            torch.cuda.current_stream().wait_stream(st)
        torch.cuda.synchronize()
        for pr, st, (s_ref, i_ref, k_ref) in zip(probs, streams, ref):
            assert jacap.read_status(pr.ws, st) == 0
            for b in range(len(case.seq_lens)):
                lo, hi = token_slice(case, b)
                assert torch.equal(pr.scores[:, :, lo:hi], s_ref[:, :, lo:hi])
                kk = min(pr.cfg.budget_k, case.seq_lens[b])
                assert torch.equal(pr.k_out[b, :, :, :kk], k_ref[b, :, :, :kk])
            assert torch.equal(pr.idx, i_ref)


def test_evict_slots_replays_from_a_graph(jacap):
    """The in-place decoding round (jacap_evict_slots) captured in a graph
    replays the eager evicted-slot lists and scores bit for bit."""
    case = make_case("ragged16", seq_lens=[288, 288, 100], num_layers=2, num_kv_heads=2,
                     num_q_heads=4, window=8, head_dim=64, dtype="bf16").to("cuda")
    p = jacap.Params(budget_k=256, gqa_mode=jacap.GQA_PER_HEAD)
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, p)
    slots = jacap.alloc_slots(prob, case.seq_lens)
    jacap.run_evict_slots(prob, slots, case.q_win, case.k, case.v)
    assert jacap.read_status(prob.ws) == 0
    torch.cuda.synchronize()
    ref_s, ref_sl = prob.scores.clone(), slots.clone()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            jacap.run_evict_slots(prob, slots, case.q_win, case.k, case.v)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for rep in range(3):
        prob.scores.fill_(-7.0)
        slots.fill_(-7)
        torch.cuda.synchronize()
        print(f"\n[graph] evict_slots: replay {rep}", flush=True)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(slots, ref_sl)
        for b in range(len(case.seq_lens)):
            lo, hi = token_slice(case, b)
            assert torch.equal(prob.scores[:, :, lo:hi], ref_s[:, :, lo:hi])
    del g
