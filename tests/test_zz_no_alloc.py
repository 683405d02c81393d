"""jacap_evict_noalloc (the library's own scratch memory instead of a caller
workspace) against jacap_evict through the C ABI: two calls in a row, the
second on a smaller input, each bit-identical to jacap_evict on the same
inputs (same kernels and launch sequence, so scores, indices and the compacted
K', V' agree exactly), its status word written to the caller's buffer, and a
problem whose workspace exceeds the scratch array rejected up front."""

import pytest
import torch

from jacap_synth import make_case

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def jacap():
    from paper_2609_08131_amd import jacap as j
    return j


def _both(jacap, case, params):
    ref = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, params)
    # rows past min(budget, n) of K', V' are left untouched: same fill for both
    ref.k_out.fill_(3.0)
    ref.v_out.fill_(3.0)
    jacap.run_evict(ref, case.q_win, case.k, case.v)
    ref_flags = jacap.read_status(ref.ws)
    got = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, params)
    got.scores.fill_(-7.0)
    got.idx.fill_(-7)
    got.k_out.fill_(3.0)
    got.v_out.fill_(3.0)
    status = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    jacap.evict_noalloc(got.cfg, got.batch, case.q_win, case.k, case.v, got.scores, got.idx,
                        got.k_out, got.v_out, status)
    torch.cuda.synchronize()
    assert int(status.item()) == ref_flags
    # bit for bit (NaN scores of a singular unit included)
    assert torch.equal(got.scores.view(torch.int32), ref.scores.view(torch.int32))
    assert torch.equal(got.idx, ref.idx)
    assert torch.equal(got.k_out, ref.k_out) and torch.equal(got.v_out, ref.v_out)
    return got


def test_noalloc_matches_evict_two_calls(jacap):
    # first call: one Llama-3-8B-shaped layer (8 KV heads x 8192 tokens, bf16)
    big = make_case("llama8b_layer", device="cuda")
    _both(jacap, big, jacap.Params(budget_k=512))
    # second call, smaller: a ragged batch at d = 64, ridge 0 (units on the fp64
    # path, and a 17-token sequence whose units are singular), per-head GQA and
    # a protected tail; the scratch still holds the first call's contents
    small = make_case("ragged16", device="cuda", seq_lens=[700, 17, 2049], num_layers=2,
                      num_kv_heads=2, num_q_heads=4, window=8, head_dim=64)
    _both(jacap, small, jacap.Params(budget_k=64, ridge=0.0, gqa_mode=jacap.GQA_PER_HEAD,
                                     protect_last=5))
    # and the first shape again after the smaller one
    _both(jacap, big, jacap.Params(budget_k=300, ridge=0.25))


def test_noalloc_rejects_problems_beyond_its_scratch(jacap):
    # 8 KV heads x 2^19 tokens: about 85 MiB of workspace
    case = make_case("llama8b_layer", device="cuda", seq_lens=[1 << 19])
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens,
                         jacap.Params(budget_k=16))
    assert prob.ws.numel() > 64 << 20
    with pytest.raises(jacap.JacapError) as e:
        jacap.evict_noalloc(prob.cfg, prob.batch, case.q_win, case.k, case.v, prob.scores,
                            prob.idx, prob.k_out, prob.v_out)
    assert e.value.code == jacap.ERR_WORKSPACE
