"""Seeded synthetic KV caches and observation windows.

Recipe (applied per sequence b, layer l, KV head h; G = H_q / H_kv query heads
share the KV head):

* query centre  c_h ~ N(0, I_d); the G*w window queries are c_h + N(0, I_d);
* background keys and values ~ N(0, I_d), each with 4 outlier channels
  (chosen per tensor, without replacement) multiplied by a scale: the value
  scale is 8; the key scale is 8, or drawn once per layer from U[2, 10];
* optional key drift: the token axis is cut into segments of ``seg`` tokens and
  segment s adds a mean m_s = m_{s-1} + N(0, std^2 I) (m_0 = 0) to its keys;
* token 0 is an attention sink: k_0 = 4 c_h;
* ``n_heavy`` planted heavy hitters at distinct positions drawn uniformly from
  1..n-1: k = c_h + N(0, 0.1^2 I);
* everything is drawn in fp32 and rounded once (round-to-nearest-even) to the
  workload's storage dtype.

Layouts: K and V are [L][H_kv][T_total][d] with the sequences of a ragged batch
packed along T (``seq_offsets`` = exclusive prefix sum of the lengths, int32);
the window queries are [B][L][H_q][w][d].

Bulk arrays come from a torch generator on the requested device, so CPU and GPU
draws differ; each is deterministic for a given seed. Small draws (outlier
channels, heavy-hitter positions, per-layer scales, ragged lengths) come from
NumPy and are identical on every device.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np
import torch

ROOT_SEED = 260908131


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and distribution parameters of one synthetic workload."""

    name: str
    wid: int
    num_layers: int
    num_kv_heads: int
    num_q_heads: int
    head_dim: int
    window: int
    budget_k: int
    dtype: str                      # "fp32" or "bf16"
    seq_lens: tuple = ()            # fixed lengths (one entry per sequence)
    ragged: Optional[tuple] = None  # (num_seqs, lo, hi): lengths ~ U{lo..hi}
    n_heavy: int = 32
    k_outlier: tuple = ("fixed", 8.0)   # or ("uniform", lo, hi), per layer
    v_outlier: float = 8.0
    n_outlier: int = 4
    drift: Optional[tuple] = None   # (segment_len, std)
    budget_sweep: tuple = ()


WORKLOADS = {
    "tiny": Workload(
        name="tiny", wid=0, num_layers=1, num_kv_heads=1, num_q_heads=1,
        head_dim=64, window=16, budget_k=64, dtype="fp32", seq_lens=(512,),
        n_heavy=8),
    "llama8b_layer": Workload(
        name="llama8b_layer", wid=1, num_layers=1, num_kv_heads=8,
        num_q_heads=32, head_dim=128, window=32, budget_k=512, dtype="bf16",
        seq_lens=(8192,), n_heavy=32),
    "prefill32k": Workload(
        name="prefill32k", wid=2, num_layers=32, num_kv_heads=8,
        num_q_heads=32, head_dim=128, window=32, budget_k=512, dtype="bf16",
        seq_lens=(32768,), n_heavy=32, k_outlier=("uniform", 2.0, 10.0),
        budget_sweep=(128, 256, 512, 1024, 2048)),
    "long128k": Workload(
        name="long128k", wid=3, num_layers=32, num_kv_heads=8,
        num_q_heads=32, head_dim=128, window=64, budget_k=1024, dtype="bf16",
        seq_lens=(131072,), n_heavy=32, k_outlier=("uniform", 2.0, 10.0),
        drift=(4096, 0.5)),
    "ragged16": Workload(
        name="ragged16", wid=4, num_layers=32, num_kv_heads=8,
        num_q_heads=32, head_dim=128, window=32, budget_k=256, dtype="bf16",
        ragged=(16, 4096, 32768), n_heavy=32,
        k_outlier=("uniform", 2.0, 10.0)),
    # Decoding-stage eviction: a cache holding the reserved budget plus one
    # re-eviction interval of 128 new tokens, 16 sequences.
    "decode2k": Workload(
        name="decode2k", wid=5, num_layers=32, num_kv_heads=8,
        num_q_heads=32, head_dim=128, window=64, budget_k=2048, dtype="bf16",
        seq_lens=(2048 + 128,) * 16, n_heavy=32, k_outlier=("uniform", 2.0, 10.0)),
    "decode16k": Workload(
        name="decode16k", wid=6, num_layers=32, num_kv_heads=8,
        num_q_heads=32, head_dim=128, window=64, budget_k=16384, dtype="bf16",
        seq_lens=(16384 + 128,) * 16, n_heavy=32, k_outlier=("uniform", 2.0, 10.0)),
}
BY_ID = {w.wid: w for w in WORKLOADS.values()}


def _workload(spec) -> Workload:
    if isinstance(spec, Workload):
        return spec
    if isinstance(spec, int):
        return BY_ID[spec]
    return WORKLOADS[spec]


def unit_seed(wid: int, seq: int, layer: int, root: int = ROOT_SEED) -> np.random.SeedSequence:
    """SeedSequence for one (workload, sequence, layer) slab of the cache."""
    return np.random.SeedSequence(root, spawn_key=(int(wid), int(seq), int(layer)))


def _torch_seed(ss: np.random.SeedSequence) -> int:
    return int(ss.generate_state(1, np.uint64)[0] & np.uint64((1 << 62) - 1))


def _storage_dtype(name: str) -> torch.dtype:
    return {"fp32": torch.float32, "bf16": torch.bfloat16}[name]


@dataclasses.dataclass
class Case:
    """One synthetic batch: window queries, keys, values and ragged offsets."""

    workload: Workload
    q_win: torch.Tensor        # [B][L][H_q][w][d]
    k: torch.Tensor            # [L][H_kv][T_total][d]
    v: torch.Tensor            # [L][H_kv][T_total][d]
    seq_lens: list
    seq_offsets: torch.Tensor  # int32 [B+1], same device as k

    @property
    def num_seqs(self) -> int:
        return len(self.seq_lens)

    @property
    def total_tokens(self) -> int:
        return int(sum(self.seq_lens))

    @property
    def max_seq_len(self) -> int:
        return int(max(self.seq_lens)) if self.seq_lens else 0

    def to(self, device) -> "Case":
        """The same case with every tensor moved to `device` (values unchanged)."""
        return Case(workload=self.workload, q_win=self.q_win.to(device), k=self.k.to(device),
                    v=self.v.to(device), seq_lens=list(self.seq_lens),
                    seq_offsets=self.seq_offsets.to(device))

    def unit_arrays(self, b: int, layer: int, head: int):
        """Host fp64 copies (exact widening) of one unit's Q window, K and V."""
        w = self.workload
        g = w.num_q_heads // w.num_kv_heads
        lo = int(sum(self.seq_lens[:b]))
        hi = lo + int(self.seq_lens[b])
        q = self.q_win[b, layer, head * g:(head + 1) * g]
        k = self.k[layer, head, lo:hi]
        v = self.v[layer, head, lo:hi]
        to = lambda t: t.detach().to("cpu", torch.float64).numpy()
        return to(q), to(k), to(v)


def draw_seq_lens(wl: Workload, root: int = ROOT_SEED) -> list:
    if wl.ragged is None:
        return [int(x) for x in wl.seq_lens]
    nseq, lo, hi = wl.ragged
    rng = np.random.default_rng(np.random.SeedSequence(root, spawn_key=(wl.wid, 1 << 20)))
    return [int(x) for x in rng.integers(lo, hi + 1, size=nseq)]


def make_case(spec="tiny", *, device="cpu", root: int = ROOT_SEED,
              seq_lens: Optional[Sequence[int]] = None, **overrides) -> Case:
    """Build a seeded synthetic case.

    ``spec`` names a workload (or passes a ``Workload``); ``overrides`` replace
    any of its fields (e.g. ``head_dim=128, dtype="bf16"``) for tests;
    ``seq_lens`` replaces the sequence lengths.
    """
    wl = _workload(spec)
    if overrides:
        wl = dataclasses.replace(wl, **overrides)
    lens = list(seq_lens) if seq_lens is not None else draw_seq_lens(wl, root)
    L, H, Hq, d, w = wl.num_layers, wl.num_kv_heads, wl.num_q_heads, wl.head_dim, wl.window
    if Hq % H != 0:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    G = Hq // H
    B = len(lens)
    T = int(sum(lens))
    dt = _storage_dtype(wl.dtype)
    dev = torch.device(device)

    k_all = torch.empty((L, H, T, d), dtype=dt, device=dev)
    v_all = torch.empty((L, H, T, d), dtype=dt, device=dev)
    q_all = torch.empty((B, L, Hq, w, d), dtype=dt, device=dev)

    off = 0
    for b, n in enumerate(lens):
        for layer in range(L):
            ss = unit_seed(wl.wid, b, layer, root)
            np_ss, torch_ss = ss.spawn(2)
            rng = np.random.default_rng(np_ss)
            gen = torch.Generator(device=dev)
            gen.manual_seed(_torch_seed(torch_ss))
            if wl.k_outlier[0] == "fixed":
                k_scale = float(wl.k_outlier[1])
            else:
                k_scale = float(rng.uniform(wl.k_outlier[1], wl.k_outlier[2]))
            centre = torch.randn((H, d), generator=gen, device=dev)
            q = centre[:, None, None, :] + torch.randn((H, G, w, d), generator=gen, device=dev)
            q_all[b, layer] = q.reshape(Hq, w, d).to(dt)
            if n == 0:
                continue
            kk = torch.randn((H, n, d), generator=gen, device=dev)
            vv = torch.randn((H, n, d), generator=gen, device=dev)
            for h in range(H):
                kch = rng.choice(d, size=min(wl.n_outlier, d), replace=False)
                vch = rng.choice(d, size=min(wl.n_outlier, d), replace=False)
                kk[h, :, torch.as_tensor(kch, device=dev)] *= k_scale
                vv[h, :, torch.as_tensor(vch, device=dev)] *= wl.v_outlier
            if wl.drift is not None:
                seg, std = wl.drift
                nseg = (n + seg - 1) // seg
                steps = std * torch.randn((H, nseg, d), generator=gen, device=dev)
                steps[:, 0] = 0.0
                means = torch.cumsum(steps, dim=1)
                seg_of = torch.arange(n, device=dev) // seg
                kk += means[:, seg_of, :]
            kk[:, 0] = 4.0 * centre
            n_hh = min(wl.n_heavy, n - 1)
            if n_hh > 0:
                noise = 0.1 * torch.randn((H, n_hh, d), generator=gen, device=dev)
                for h in range(H):
                    pos = 1 + rng.choice(n - 1, size=n_hh, replace=False)
                    kk[h, torch.as_tensor(pos, device=dev)] = centre[h] + noise[h]
            k_all[layer, :, off:off + n] = kk.to(dt)
            v_all[layer, :, off:off + n] = vv.to(dt)
        off += n

    offsets = torch.tensor(np.concatenate([[0], np.cumsum(lens)]).astype(np.int32), device=dev)
    return Case(workload=wl, q_win=q_all, k=k_all, v=v_all, seq_lens=lens, seq_offsets=offsets)


def make_output_projection(spec="tiny", *, d_model: int = 256, device="cpu",
                           root: int = ROOT_SEED, **overrides) -> torch.Tensor:
    """Seeded synthetic output projections W_O, one per layer: fp32
    [L][d_model][H_q * d] with entries N(0, 1/d_model) (a random stand-in for a
    trained projection; no checkpoint is available)."""
    wl = _workload(spec)
    if overrides:
        wl = dataclasses.replace(wl, **overrides)
    out = torch.empty((wl.num_layers, d_model, wl.num_q_heads * wl.head_dim),
                      dtype=torch.float32, device=device)
    for layer in range(wl.num_layers):
        ss = np.random.SeedSequence(root, spawn_key=(wl.wid, 1 << 21, layer))
        gen = torch.Generator(device=device)
        gen.manual_seed(_torch_seed(ss))
        out[layer] = torch.randn((d_model, wl.num_q_heads * wl.head_dim), generator=gen,
                                 device=device) / math.sqrt(d_model)
    return out
