"""The seeded generator: determinism, layout and the planted structure."""

import numpy as np
import torch

from jacap_synth import WORKLOADS, make_case


def test_deterministic_and_shapes():
    a = make_case("tiny")
    b = make_case("tiny")
    assert torch.equal(a.k, b.k) and torch.equal(a.v, b.v) and torch.equal(a.q_win, b.q_win)
    w = WORKLOADS["tiny"]
    assert a.k.shape == (1, 1, 512, 64) and a.k.dtype == torch.float32
    assert a.q_win.shape == (1, 1, 1, 16, 64)
    assert a.seq_offsets.tolist() == [0, 512]
    c = make_case("tiny", root=7)
    assert not torch.equal(a.k, c.k)
    assert w.budget_k == 64


def test_sink_and_heavy_hitters_attract_attention():
    case = make_case("tiny")
    q, k, v = case.unit_arrays(0, 0, 0)
    mu = q.reshape(-1, 64).mean(axis=0)
    logits = k @ mu
    order = np.argsort(-logits)
    assert order[0] == 0                      # the sink (4x the query centre)
    assert set(order[1:9].tolist()) <= set(range(1, 512))
    # the 8 heavy hitters sit near the centre: cosine with mu close to 1
    cos = (k @ mu) / (np.linalg.norm(k, axis=1) * np.linalg.norm(mu))
    assert (cos > 0.9).sum() == 9


def test_bf16_rounding_and_ragged_layout():
    case = make_case("ragged16", num_layers=2, num_kv_heads=2, num_q_heads=4,
                     head_dim=64, seq_lens=[5, 0, 17])
    assert case.k.dtype == torch.bfloat16 and case.k.shape == (2, 2, 22, 64)
    assert case.seq_offsets.tolist() == [0, 5, 5, 22]
    assert case.q_win.shape == (3, 2, 4, 32, 64)
    q, k, v = case.unit_arrays(2, 1, 1)
    assert k.shape == (17, 64) and q.shape == (2, 32, 64)
    ragged = make_case("ragged16", num_layers=1, num_kv_heads=1, num_q_heads=1,
                       head_dim=64, n_heavy=2, ragged=(4, 10, 30))
    assert all(10 <= n <= 30 for n in ragged.seq_lens) and len(ragged.seq_lens) == 4
