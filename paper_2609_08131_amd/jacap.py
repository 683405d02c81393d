"""Python binding of libjacap.so (ctypes; argument marshalling only).

Every function here converts torch tensors to raw device pointers and calls
the C entry point of the same name; all computation happens in the HIP
kernels of libjacap.so. If the library is missing the import of this module
fails loudly (there is no fallback path).

Layouts follow include/jacap.h: K, V [L][H_kv][T_total][d] (any strides with
d contiguous), window queries [B][L][H_q][w][d], scores [L][H_kv][T_total]
fp32, idx [B][L][H_kv][budget] int32, K', V' [B][L][H_kv][budget][d].
"""

from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libjacap.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)
COV_DIAG, COV_FULL = 0, 1
RIDGE_SCALAR, RIDGE_MATRIX = 0, 1   # enum jacap_ridge_mode
GQA_POOLED, GQA_PER_HEAD = 0, 1     # enum jacap_gqa_mode
DTYPE_FP32, DTYPE_BF16 = 0, 1
FLAG_NONFINITE, FLAG_SINGULAR, FLAG_BAD_OFFSETS = 1, 2, 4

_TORCH_DTYPE = {DTYPE_FP32: torch.float32, DTYPE_BF16: torch.bfloat16}
_DTYPE_CODE = {torch.float32: DTYPE_FP32, torch.bfloat16: DTYPE_BF16}


class JacapError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} failed: {status_string(code)} ({code})")
        self.code = code


class Config(ctypes.Structure):
    _fields_ = [
        ("num_layers", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("budget_k", ctypes.c_int32),
        ("temperature", ctypes.c_float),
        ("ridge", ctypes.c_float),
        ("cov_mode", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("ridge_mode", ctypes.c_int32),
        ("gqa_mode", ctypes.c_int32),
        ("protect_last", ctypes.c_int32),
    ]


class Batch(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32),
        ("max_seq_len", ctypes.c_int32),
        ("total_tokens", ctypes.c_int64),
        ("seq_offsets", ctypes.c_void_p),
        ("k_stride_layer", ctypes.c_int64), ("k_stride_head", ctypes.c_int64),
        ("k_stride_token", ctypes.c_int64),
        ("v_stride_layer", ctypes.c_int64), ("v_stride_head", ctypes.c_int64),
        ("v_stride_token", ctypes.c_int64),
        ("q_stride_seq", ctypes.c_int64), ("q_stride_layer", ctypes.c_int64),
        ("q_stride_head", ctypes.c_int64), ("q_stride_pos", ctypes.c_int64),
        ("out_stride_seq", ctypes.c_int64), ("out_stride_layer", ctypes.c_int64),
        ("out_stride_head", ctypes.c_int64), ("out_stride_row", ctypes.c_int64),
        ("ridge_mat", ctypes.c_void_p),
    ]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"libjacap.so not found at {LIB_PATH}; build it with "
            "`python -m paper_2609_08131_amd.build` (there is no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    P, C, B = ctypes.c_void_p, ctypes.POINTER(Config), ctypes.POINTER(Batch)
    sz = ctypes.c_size_t
    sigs = {
        "jacap_workspace_size": [C, B, ctypes.POINTER(sz)],
        "jacap_score": [C, B, P, P, P, P, P, sz, P],
        "jacap_score_from_stats": [C, B, P, P, P, P, P, P, sz, P],
        "jacap_select": [C, B, P, P, P, sz, P],
        "jacap_compact": [C, B, P, P, P, P, P, P],
        "jacap_evict": [C, B, P, P, P, P, P, P, P, P, sz, P],
        "jacap_select_evicted": [C, B, P, P, ctypes.c_int32, P, sz, P],
        "jacap_evict_slots": [C, B, P, P, P, P, P, ctypes.c_int32, P, sz, P],
        "jacap_read_status": [P, P, ctypes.POINTER(ctypes.c_uint32)],
        "jacap_greedy_workspace_size": [C, B, ctypes.POINTER(sz)],
        "jacap_greedy": [C, B, P, P, P, P, P, P, P, sz, P],
        "jacap_stream_read": [P, sz, P, P],
        "jacap_evict_noalloc": [C, B, P, P, P, P, P, P, P, P, P],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.jacap_status_string.argtypes = [ctypes.c_int]
    lib.jacap_status_string.restype = ctypes.c_char_p
    lib.jacap_timing_start.argtypes = [ctypes.c_uint32]
    lib.jacap_timing_start.restype = ctypes.c_int
    lib.jacap_timing_stop.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)]
    lib.jacap_timing_stop.restype = ctypes.c_int
    lib.jacap_phase_name.argtypes = [ctypes.c_int32]
    lib.jacap_phase_name.restype = ctypes.c_char_p
    return lib


_lib = _load()
EXPORTED = ("jacap_workspace_size", "jacap_score", "jacap_score_from_stats", "jacap_select",
            "jacap_compact", "jacap_evict", "jacap_read_status", "jacap_status_string",
            "jacap_timing_start", "jacap_timing_stop", "jacap_phase_name",
            "jacap_greedy_workspace_size", "jacap_greedy", "jacap_stream_read",
            "jacap_select_evicted", "jacap_evict_slots", "jacap_evict_noalloc")
NUM_PHASES = 13   # enum jacap_phase


def status_string(code: int) -> str:
    return _lib.jacap_status_string(int(code)).decode()


def _check(fn: str, code: int) -> None:
    if code != OK:
        raise JacapError(fn, code)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


# ---------------------------------------------------------------------------
# Descriptors
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Params:
    """Method parameters (see jacap_config in include/jacap.h)."""

    budget_k: int
    temperature: float = 10.0
    ridge: float = 1.0
    cov_mode: int = COV_DIAG
    # Output-projection variant: device float64 [L][H_kv][d][d] matrices R that
    # replace ridge * I (see include/jacap.h); None = scalar ridge.
    ridge_matrix: Optional[torch.Tensor] = None
    gqa_mode: int = GQA_POOLED
    protect_last: int = 0       # most recent positions of each sequence always kept


def make_config(q_win: torch.Tensor, k: torch.Tensor, p: Params) -> Config:
    B, L, Hq, w, d = q_win.shape
    Lk, H, T, dk = k.shape
    if Lk != L or dk != d:
        raise ValueError("q_win and k disagree on layers or head_dim")
    if k.dtype not in _DTYPE_CODE or q_win.dtype != k.dtype:
        raise ValueError("q_win, k, v must share a dtype: float32 or bfloat16")
    return Config(L, H, Hq, d, w, int(p.budget_k), float(p.temperature), float(p.ridge),
                  int(p.cov_mode), _DTYPE_CODE[k.dtype],
                  RIDGE_SCALAR if p.ridge_matrix is None else RIDGE_MATRIX,
                  int(p.gqa_mode), int(p.protect_last))


def make_batch(seq_offsets: torch.Tensor, seq_lens, q_win: torch.Tensor, k: torch.Tensor,
               v: torch.Tensor, out: Optional[torch.Tensor] = None) -> Batch:
    """seq_lens: host list of the sequence lengths (for max_seq_len / total)."""
    if seq_offsets.dtype != torch.int32 or not seq_offsets.is_cuda:
        raise ValueError("seq_offsets must be a device int32 tensor")
    b = Batch()
    b.num_seqs = len(seq_lens)
    b.max_seq_len = int(max(seq_lens)) if len(seq_lens) else 0
    b.total_tokens = int(sum(seq_lens))
    b.seq_offsets = seq_offsets.data_ptr()
    for name, t in (("k", k), ("v", v)):
        if t.stride(-1) != 1:
            raise ValueError(f"{name}: head_dim must be contiguous")
        setattr(b, f"{name}_stride_layer", t.stride(0))
        setattr(b, f"{name}_stride_head", t.stride(1))
        setattr(b, f"{name}_stride_token", t.stride(2))
    if q_win.stride(-1) != 1:
        raise ValueError("q_win: head_dim must be contiguous")
    b.q_stride_seq, b.q_stride_layer, b.q_stride_head, b.q_stride_pos = q_win.stride()[:4]
    if out is not None:
        b.out_stride_seq, b.out_stride_layer, b.out_stride_head, b.out_stride_row = out.stride()[:4]
    else:
        d = k.shape[-1]
        # dense [B][L][H][budget][d] is filled in by allocate_outputs users
        b.out_stride_row = d
    return b


def set_ridge_matrix(b: Batch, r: torch.Tensor, shape) -> None:
    """Point the batch at the ridge matrices R (device float64 [L][H_kv][d][d])."""
    L, H, d = shape
    if r.dtype != torch.float64 or not r.is_cuda or tuple(r.shape) != (L, H, d, d) \
            or not r.is_contiguous():
        raise ValueError("ridge_matrix must be a contiguous device float64 [L][H_kv][d][d] tensor")
    b.ridge_mat = r.data_ptr()


def set_out_strides(b: Batch, out: torch.Tensor) -> None:
    b.out_stride_seq, b.out_stride_layer, b.out_stride_head, b.out_stride_row = out.stride()[:4]


# ---------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def workspace_size(cfg: Config, batch: Batch) -> int:
    n = ctypes.c_size_t(0)
    _check("jacap_workspace_size", _lib.jacap_workspace_size(ctypes.byref(cfg), ctypes.byref(batch), ctypes.byref(n)))
    return int(n.value)


def alloc_workspace(cfg: Config, batch: Batch, device=None) -> torch.Tensor:
    nbytes = workspace_size(cfg, batch)
    # torch's caching allocator returns 512-byte aligned blocks
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device or "cuda")
    assert ws.data_ptr() % 256 == 0
    return ws


def score(cfg, batch, q_win, k, v, scores, ws, stream=None) -> None:
    _check("jacap_score", _lib.jacap_score(
        ctypes.byref(cfg), ctypes.byref(batch), _ptr(q_win), _ptr(k), _ptr(v), _ptr(scores),
        _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream)))


def score_from_stats(cfg, batch, mu, lam, k, v, scores, ws, stream=None) -> None:
    """jacap_score_from_stats: mu float64 [U][d]; lam float64 [U][d] (DIAG) or
    [U][d][d] (FULL), U in unit order (seq, layer, kv head)."""
    _check("jacap_score_from_stats", _lib.jacap_score_from_stats(
        ctypes.byref(cfg), ctypes.byref(batch), _ptr(mu), _ptr(lam), _ptr(k), _ptr(v),
        _ptr(scores), _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream)))


def stream_read(src: torch.Tensor, sink: torch.Tensor, stream=None) -> None:
    """jacap_stream_read over every byte of the contiguous device tensor src
    (a measurement probe; sink: a device tensor of at least 4 bytes)."""
    assert src.is_contiguous()
    _check("jacap_stream_read", _lib.jacap_stream_read(
        _ptr(src), src.numel() * src.element_size(), _ptr(sink), _stream(stream)))


def select(cfg, batch, scores, idx, ws=None, stream=None) -> None:
    _check("jacap_select", _lib.jacap_select(
        ctypes.byref(cfg), ctypes.byref(batch), _ptr(scores), _ptr(idx), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))


def compact(cfg, batch, idx, k, v, k_out, v_out, stream=None) -> None:
    _check("jacap_compact", _lib.jacap_compact(
        ctypes.byref(cfg), ctypes.byref(batch), _ptr(idx), _ptr(k), _ptr(v), _ptr(k_out),
        _ptr(v_out), _stream(stream)))


def evict(cfg, batch, q_win, k, v, scores, idx, k_out, v_out, ws, stream=None) -> None:
    _check("jacap_evict", _lib.jacap_evict(
        ctypes.byref(cfg), ctypes.byref(batch), _ptr(q_win), _ptr(k), _ptr(v), _ptr(scores),
        _ptr(idx), _ptr(k_out), _ptr(v_out), _ptr(ws), ws.numel(), _stream(stream)))


def evict_noalloc(cfg, batch, q_win, k, v, scores, idx, k_out, v_out, status=None,
                  stream=None) -> None:
    """jacap_evict with the library's own scratch memory (no workspace);
    status: optional int32 device tensor of one element receiving the flags."""
    _check("jacap_evict_noalloc", _lib.jacap_evict_noalloc(
        ctypes.byref(cfg), ctypes.byref(batch), _ptr(q_win), _ptr(k), _ptr(v), _ptr(scores),
        _ptr(idx), _ptr(k_out), _ptr(v_out), _ptr(status), _stream(stream)))


def select_evicted(cfg, batch, scores, slots, ws, stream=None) -> None:
    """slots: int32 [B][L][H][slot_cap] (the last dimension is the capacity)."""
    _check("jacap_select_evicted", _lib.jacap_select_evicted(
        ctypes.byref(cfg), ctypes.byref(batch), _ptr(scores), _ptr(slots),
        int(slots.shape[-1]), _ptr(ws), ws.numel(), _stream(stream)))


def evict_slots(cfg, batch, q_win, k, v, scores, slots, ws, stream=None) -> None:
    _check("jacap_evict_slots", _lib.jacap_evict_slots(
        ctypes.byref(cfg), ctypes.byref(batch), _ptr(q_win), _ptr(k), _ptr(v), _ptr(scores),
        _ptr(slots), int(slots.shape[-1]), _ptr(ws), ws.numel(), _stream(stream)))


def greedy_workspace_size(cfg: Config, batch: Batch) -> int:
    n = ctypes.c_size_t(0)
    _check("jacap_greedy_workspace_size", _lib.jacap_greedy_workspace_size(
        ctypes.byref(cfg), ctypes.byref(batch), ctypes.byref(n)))
    return int(n.value)


def greedy(cfg, batch, q_win, k, v, idx, order, logdet, ws, stream=None) -> None:
    _check("jacap_greedy", _lib.jacap_greedy(
        ctypes.byref(cfg), ctypes.byref(batch), _ptr(q_win), _ptr(k), _ptr(v), _ptr(idx),
        _ptr(order), _ptr(logdet), _ptr(ws), ws.numel() if ws is not None else 0,
        _stream(stream)))


def read_status(ws: torch.Tensor, stream=None) -> int:
    f = ctypes.c_uint32(0)
    _check("jacap_read_status", _lib.jacap_read_status(_ptr(ws), _stream(stream), ctypes.byref(f)))
    return int(f.value)


# ---------------------------------------------------------------------------
# Convenience: allocate outputs and run the whole path on torch tensors
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Problem:
    """Descriptors and output buffers for one batch (allocated once, reusable)."""

    cfg: Config
    batch: Batch
    scores: torch.Tensor
    idx: torch.Tensor
    k_out: torch.Tensor
    v_out: torch.Tensor
    ws: torch.Tensor


def prepare(q_win, k, v, seq_offsets, seq_lens, params: Params) -> Problem:
    cfg = make_config(q_win, k, params)
    B = len(seq_lens)
    L, H, T, d = k.shape
    dev = k.device
    kb = max(int(params.budget_k), 0)
    scores = torch.empty((L, H, T), dtype=torch.float32, device=dev)
    idx = torch.empty((B, L, H, max(kb, 1)), dtype=torch.int32, device=dev)[..., :kb]
    k_out = torch.empty((B, L, H, max(kb, 1), d), dtype=k.dtype, device=dev)
    v_out = torch.empty_like(k_out)
    batch = make_batch(seq_offsets, seq_lens, q_win, k, v, out=k_out)
    if params.ridge_matrix is not None:
        set_ridge_matrix(batch, params.ridge_matrix, (L, H, d))
    ws = alloc_workspace(cfg, batch, dev)
    return Problem(cfg, batch, scores, idx, k_out[..., :kb, :], v_out[..., :kb, :], ws)


def run_evict(prob: Problem, q_win, k, v, stream=None) -> None:
    evict(prob.cfg, prob.batch, q_win, k, v, prob.scores, prob.idx, prob.k_out, prob.v_out,
          prob.ws, stream)


def alloc_slots(prob: Problem, seq_lens) -> torch.Tensor:
    """int32 [B][L][H][max(0, max_seq_len - budget)] for select_evicted / evict_slots."""
    B, L, H = prob.idx.shape[:3]
    cap = max(0, int(prob.batch.max_seq_len) - int(prob.cfg.budget_k))
    return torch.empty((B, L, H, max(cap, 1)), dtype=torch.int32, device=prob.scores.device)


def run_evict_slots(prob: Problem, slots, q_win, k, v, stream=None) -> None:
    evict_slots(prob.cfg, prob.batch, q_win, k, v, prob.scores, slots, prob.ws, stream)


@dataclasses.dataclass
class GreedyProblem:
    """Descriptors, outputs and workspace of jacap_greedy for one batch."""

    cfg: Config
    batch: Batch
    idx: torch.Tensor       # int32 [B][L][H][budget], ascending, -1 padding
    order: torch.Tensor     # int32 [B][L][H][budget], pick order, -1 padding
    logdet: torch.Tensor    # float64 [B][L][H]
    ws: torch.Tensor


def prepare_greedy(q_win, k, v, seq_offsets, seq_lens, params: Params) -> GreedyProblem:
    cfg = make_config(q_win, k, params)
    B = len(seq_lens)
    L, H, T, d = k.shape
    dev = k.device
    kb = max(int(params.budget_k), 0)
    idx = torch.empty((B, L, H, max(kb, 1)), dtype=torch.int32, device=dev)[..., :kb]
    order = torch.empty_like(idx)
    logdet = torch.empty((B, L, H), dtype=torch.float64, device=dev)
    batch = make_batch(seq_offsets, seq_lens, q_win, k, v)
    nbytes = greedy_workspace_size(cfg, batch)
    ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
    assert ws.data_ptr() % 256 == 0
    return GreedyProblem(cfg, batch, idx, order, logdet, ws)


def run_greedy(prob: GreedyProblem, q_win, k, v, stream=None) -> None:
    greedy(prob.cfg, prob.batch, q_win, k, v, prob.idx, prob.order, prob.logdet, prob.ws, stream)


# ---------------------------------------------------------------------------
# Per-phase GPU timing (jacap_timing_start / jacap_timing_stop)
# ---------------------------------------------------------------------------
def phase_name(phase: int) -> str:
    return _lib.jacap_phase_name(int(phase)).decode()


PHASES = tuple(phase_name(p) for p in range(NUM_PHASES))


def timing_start(phases=None) -> None:
    """Start recording the named phases (all when None); clears old records."""
    names = PHASES if phases is None else phases
    mask = 0
    for n in names:
        mask |= 1 << PHASES.index(n)
    _check("jacap_timing_start", _lib.jacap_timing_start(mask))


def timing_stop() -> dict:
    """Stop recording; {phase: (summed GPU ms, recorded calls)} for recorded phases."""
    ms = (ctypes.c_double * NUM_PHASES)()
    calls = (ctypes.c_int32 * NUM_PHASES)()
    _check("jacap_timing_stop", _lib.jacap_timing_stop(ms, calls))
    return {PHASES[p]: (ms[p], calls[p]) for p in range(NUM_PHASES) if calls[p] > 0}
