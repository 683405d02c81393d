"""Benchmark of the Jacap eviction pass (score + select + compact) on one MI355X.

One step = jacap_evict over the whole synthetic batch (every layer and KV
head): window statistics, centre attention, Eq. 8 weights, weighted Gram,
Cholesky, leverage scores, top-B selection and K/V compaction. Inputs are
resident in HBM before timing starts.

Prints one JSON line:
  value        cached tokens scored+selected per second (full-model tokens:
               one token = its K/V rows in every layer and KV head)
  roofline     the dominant phase's algorithmic HBM bytes per launch / its
               average GPU duration, timed with HIP events that the library
               records around that phase on the launch stream inside the
               timed region; "traffic" is its measured HBM bytes per launch
               (rocprofv3 FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of
               known size) when the recorded counters match the current
               kernel source, else null. roofline.pass is the whole pass:
               K and V bytes read once per step / ms_per_step against the
               same peak (also the top-level step_frac)
  cpu_baseline the fp64 oracle timed on this host on a bounded sample
"""

from __future__ import annotations

import argparse
import hashlib
import json
import re
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "cached tokens scored+selected/sec per GPU; achieved HBM GB/s vs peak"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="long128k")
    ap.add_argument("--budget", type=int, default=None)
    ap.add_argument("--ridge", type=float, default=1.0)
    ap.add_argument("--tau", type=float, default=10.0)
    ap.add_argument("--cov", choices=("diag", "full"), default="diag",
                    help="query covariance: per-channel variances (default) or the full matrix")
    ap.add_argument("--gqa", choices=("pooled", "per_head"), default="pooled",
                    help="GQA reading: the group's queries pooled (default) or each head alone")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="time budget of the oracle CPU baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mode", choices=("evict", "greedy"), default="evict",
                    help="evict: the Jacap pass (the headline line); greedy: the exact "
                         "greedy log-det selection (jacap_greedy), a quality comparator")
    ap.add_argument("--inplace", action="store_true",
                    help="evicted-slot lists instead of the compacted cache "
                         "(jacap_evict_slots: a decoding round whose cache is refilled in place)")
    ap.add_argument("--flush", action="store_true",
                    help="before every step (outside its timed events) read a 1 GiB buffer "
                         "with the default cache policy, so that inputs smaller than the "
                         "256 MB MALL are not measured cache-warm")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 1 GiB elementwise copy (torch.neg; the "
                         "reference kernel for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    return ap.parse_args()


COPY_BYTES = 1 << 30
FLUSH_BYTES = 1 << 30
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
# Source files whose kernels each phase launches (a change voids recorded counters).
# Source file, kernel (the DIAG bf16 one on long128k) and launch function of
# each phase.
PHASE_SOURCES = {
    "qstats": ("k_stats.hip", "qstats_kernel", "launch_qstats"),
    "kpass": ("k_stats.hip", "kpass_quad_kernel", "launch_kpass"),
    # FULL covariance on the triangular path: the K pass and the factor of Lambda_Q
    "kpass_tri": ("k_stats.hip", "kpass_tri_kernel", "launch_kpass"),
    "qfactor": ("k_factor.hip", "qfactor_kernel", "launch_qfactor"),
    "weights": ("k_stats.hip", "softmax_weights_kernel", "launch_softmax_weights"),
    "gram": ("k_gram.hip", "gram_mfma_kernel", "launch_gram"),
    "gram_reduce": ("k_gram.hip", "gram_reduce_kernel", "launch_gram_reduce"),
    "factor": ("k_factor.hip", "factor_kernel", "launch_factor"),
    "leverage": ("k_leverage.hip", "leverage_mfma_kernel", "launch_leverage"),
    "select": ("k_select.hip", "select_kernel", "launch_select"),
    "compact": ("k_select.hip", "compact_kernel", "launch_compact"),
    "greedy_init": ("k_greedy.hip", "greedy_init_kernel", "launch_greedy"),
    "greedy": ("k_greedy.hip", "greedy_kernel", "launch_greedy"),
}


def _top_level_functions(text):
    """{name: source text} of the function definitions at namespace scope of
    a HIP source file (with their template line), by brace matching."""
    # comments and string literals blanked, offsets kept
    text = re.sub(r"//[^\n]*|/\*.*?\*/|\"(?:\\.|[^\"\\])*\"",
                  lambda m: re.sub(r"[^\n]", " ", m.group(0)), text, flags=re.S)
    out, i, n = {}, 0, len(text)
    while i < n:
        ch = text[i]
        if ch == "{":
            start = max(text.rfind(";", 0, i), text.rfind("}", 0, i), text.rfind("{", 0, i)) + 1
            head = "\n".join(l for l in text[start:i].split("\n")
                             if not l.lstrip().startswith("#")).strip()
            if re.match(r"(namespace\b|extern\s+\S+$)", head):
                i += 1  # namespace scope: its contents are scanned in place
                continue
            j, d = i, 0
            while j < n:
                d += text[j] == "{"
                d -= text[j] == "}"
                if d == 0:
                    break
                j += 1
            m = re.search(r"(\w+)\s*\((?:[^()]|\([^()]*\))*\)[^()]*$", head)
            if m and not re.match(r"(struct|class|union|enum)\b", head.split("\n")[-1].strip()):
                out[m.group(1)] = out.get(m.group(1), "") + text[start:j + 1]
            i = j + 1
            continue
        i += 1
    return out


def source_sha(phase):
    """Hash of what the phase's kernel and launch come from: the shared
    internal header, the workspace layout (chunk sizes), the launch function,
    and the kernel's own definition with, transitively, the file's functions
    it names (edits elsewhere in the file leave it unchanged)."""
    entry = PHASE_SOURCES.get(phase)
    if entry is None:
        return None
    fname, kernel, launch = entry
    csrc = os.path.join(ROOT, "paper_2609_08131_amd", "csrc")
    with open(os.path.join(csrc, fname)) as fh:
        funcs = _top_level_functions(fh.read())
    with open(os.path.join(csrc, "jacap_host.hip")) as fh:
        host = _top_level_functions(fh.read())
    with open(os.path.join(csrc, "jacap_internal.hpp")) as fh:
        parts = [fh.read(), host.get("layout", ""), funcs.get(launch, "")]
    seen, todo = set(), [kernel]
    while todo:
        name = todo.pop()
        if name in seen or name not in funcs:
            continue
        seen.add(name)
        parts.append(funcs[name])
        todo.extend(f for f in funcs if f not in seen and re.search(r"\b%s\b" % f, funcs[name]))
    return hashlib.sha256("\n".join(parts).encode()).hexdigest()[:16]


def traffic_key(phase, cov, gqa, w, case):
    """The counter record of `phase`'s kernel in this configuration: FULL
    covariance with bf16 keys, 2 d <= N_s <= 256 window queries per scored
    unit and a sequence of at least 8192 tokens runs the triangular K pass."""
    ns = w.window if gqa == "per_head" else (w.num_q_heads // w.num_kv_heads) * w.window
    if phase == "kpass" and cov == "full":
        tri = (w.dtype == "bf16" and 2 * w.head_dim <= ns <= 256 and
               max(case.seq_lens) >= 8192)
        return "kpass_tri" if tri else "kpass_full"
    return phase


def recorded_traffic(phase, workload):
    """HBM bytes per launch of `phase` from the committed counter summary, if
    it was taken on this workload with the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh).get(phase)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("workload") != workload or rec.get("source_sha") != source_sha(phase):
        return None
    return rec.get("hbm_bytes_per_launch")


def phase_bytes(phase, case, budget, prob):
    """Algorithmic HBM bytes of one launch of `phase` over the whole batch:
    every input read once and every output written once."""
    w = case.workload
    e = case.k.element_size()
    d = w.head_dim
    entries = case.total_tokens * w.num_layers * w.num_kv_heads
    units = case.num_seqs * w.num_layers * w.num_kv_heads
    nb = d // 16
    npair = nb * (nb + 1) // 2
    kept = sum(min(budget, n) for n in case.seq_lens) * w.num_layers * w.num_kv_heads
    return {
        "qstats": case.q_win.numel() * e,
        "kpass": entries * (d * e + 8),                    # K rows; z, kappa out
        "weights": entries * 12,                            # z, kappa in; w out
        "gram": entries * (d * e + 4),                      # V rows, w
        "leverage": entries * (d * e + 8),                  # V rows, w; score out
        "select": entries * 4 + units * budget * 4,         # scores in; idx out
        "compact": 2 * kept * d * e * 2,                    # K, V rows in and out
        "gram_reduce": None, "factor": units * npair * 256 * 8,  # each unit's Gram (fp64 size)
        "refine": None, "init": None,
        "greedy_init": entries * (d * e + 4 + 12),          # V rows, w; c, stamp out
        "greedy": None,
    }.get(phase)


def greedy_flops(case, budget):
    """Least fp64 work of the greedy picks: per pick, A^{-1} u (d^2 FMA) and the
    rank-one downdate (d^2 FMA), 4 d^2 flops; refreshes of stale bounds add
    2 d^2 each and are not counted."""
    w = case.workload
    picks = sum(min(budget, n) for n in case.seq_lens) * w.num_layers * w.num_kv_heads
    return 4.0 * w.head_dim ** 2 * picks


def ensure_built():
    lib = os.path.join(ROOT, "paper_2609_08131_amd", "libjacap.so")
    if not os.path.exists(lib):
        from paper_2609_08131_amd import build
        build.build()


def cpu_baseline(case, budget, tau, ridge, seconds, cov="diag", gqa="pooled"):
    """Time the fp64 oracle on as many units (sequence, layer, KV head) of the
    same workload as fit in `seconds`; scale to full-model tokens/s."""
    from oracle import jacap_oracle as jo
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        cores = max([i.get("num_threads", 1) for i in info] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    w = case.workload
    units = [(b, l, h) for b in range(case.num_seqs) for l in range(w.num_layers)
             for h in range(w.num_kv_heads)]
    rng = np.random.default_rng(0)
    order = rng.permutation(len(units))
    done_tokens, done_units = 0, 0
    t_total = 0.0
    for i in order:
        b, l, h = units[i]
        q, k, v = case.unit_arrays(b, l, h)          # host copy, not timed
        t0 = time.perf_counter()
        jo.evict_unit(q, k, v, budget, tau=tau, ridge=ridge, cov_mode=cov, gqa=gqa)
        t_total += time.perf_counter() - t0
        done_tokens += k.shape[0]
        done_units += 1
        if t_total >= seconds:
            break
    entries_per_s = done_tokens / t_total
    tokens_per_s = entries_per_s / (w.num_layers * w.num_kv_heads)
    return {"value": tokens_per_s, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{done_units} of {len(units)} units (seq, layer, kv head) of {w.name}, "
                      f"{done_tokens} token-entries in {t_total:.1f} s; tokens/s = "
                      f"entries/s / (layers*kv_heads)",
            "entries_per_s": entries_per_s, "cpu_model": cpu_model()}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def read_probe(jacap, src, stream, reps=5):
    """GB/s of the library's streaming-read probe over the whole tensor src
    (one untimed pass, then `reps` timed ones, HIP events on `stream`)."""
    sink = torch.zeros(4, dtype=torch.int32, device=src.device)
    jacap.stream_read(src, sink, stream)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record(stream)
    for _ in range(reps):
        jacap.stream_read(src, sink, stream)
    e.record(stream)
    torch.cuda.synchronize()
    nbytes = src.numel() * src.element_size()
    return nbytes, nbytes * reps / (s.elapsed_time(e) * 1e-3) / 1e9


PEAK_FP64_TFLOPS = 78.6   # MI355X vector fp64


def main_greedy(args):
    """jacap_greedy on the workload: Eq. 8 weights, the initial pass and the
    sequential greedy picks (one workgroup per unit)."""
    from jacap_synth import make_case
    from paper_2609_08131_amd import jacap

    torch.cuda.set_device(0)
    case = make_case(args.workload, device="cuda")
    w = case.workload
    budget = args.budget if args.budget is not None else w.budget_k
    params = jacap.Params(budget_k=budget, temperature=args.tau, ridge=args.ridge,
                          cov_mode={"diag": jacap.COV_DIAG, "full": jacap.COV_FULL}[args.cov])
    prob = jacap.prepare_greedy(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, params)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        jacap.run_greedy(prob, case.q_win, case.k, case.v, stream)
    flags = jacap.read_status(prob.ws, stream)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    jacap.timing_start()
    for s, e in ev:
        s.record(stream)
        jacap.run_greedy(prob, case.q_win, case.k, case.v, stream)
        e.record(stream)
    torch.cuda.synchronize()
    per_phase = {k: ms / n for k, (ms, n) in jacap.timing_stop().items()}
    times = np.array([s.elapsed_time(e) for s, e in ev])
    ms = float(times.mean())
    g_ms = per_phase["greedy"]
    flops = greedy_flops(case, budget)
    units = case.num_seqs * w.num_layers * w.num_kv_heads
    # one workgroup per unit: at most min(units, 256) compute units are busy
    peak = PEAK_FP64_TFLOPS * min(units, 256) / 256
    achieved = flops / (g_ms * 1e-3) / 1e12
    init_bytes = phase_bytes("greedy_init", case, budget, prob)
    out = {
        "metric": "cached tokens greedily selected/sec per GPU (exact greedy log-det comparator)",
        "value": case.total_tokens / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic", "status_flags": flags,
        "config": {"workload": w.name, "mode": "greedy", "num_seqs": case.num_seqs,
                   "layers": w.num_layers, "kv_heads": w.num_kv_heads, "head_dim": w.head_dim,
                   "tokens": case.total_tokens, "budget_k": budget, "ridge": args.ridge},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": None, "kernel": "greedy",
                     "kernel_ms": g_ms, "flops_per_launch": flops,
                     "note": "fp64 work of the picks only; sequential in the picks"},
        "greedy_init_gbs": init_bytes / (per_phase["greedy_init"] * 1e-3) / 1e9,
        "phases_ms": {k: round(v, 4) for k, v in per_phase.items()},
    }
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    ensure_built()
    if args.mode == "greedy":
        return main_greedy(args)
    from jacap_synth import make_case
    from paper_2609_08131_amd import jacap

    torch.cuda.set_device(0)
    case = make_case(args.workload, device="cuda")
    w = case.workload
    budget = args.budget if args.budget is not None else w.budget_k
    params = jacap.Params(budget_k=budget, temperature=args.tau, ridge=args.ridge,
                          cov_mode={"diag": jacap.COV_DIAG, "full": jacap.COV_FULL}[args.cov],
                          gqa_mode={"pooled": jacap.GQA_POOLED,
                                    "per_head": jacap.GQA_PER_HEAD}[args.gqa])
    prob = jacap.prepare(case.q_win, case.k, case.v, case.seq_offsets, case.seq_lens, params)
    stream = torch.cuda.current_stream()
    if args.inplace:
        slots = jacap.alloc_slots(prob, case.seq_lens)
        run = lambda: jacap.run_evict_slots(prob, slots, case.q_win, case.k, case.v, stream)
    else:
        run = lambda: jacap.run_evict(prob, case.q_win, case.k, case.v, stream)
    torch.cuda.synchronize()

    if args.copy_calibration:
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)   # one elementwise kernel: reads and writes 1 GiB
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        run()
    flags = jacap.read_status(prob.ws, stream)
    torch.cuda.synchronize()

    # Which phase dominates: two untimed steps with every phase recorded.
    jacap.timing_start()
    for _ in range(2):
        run()
    per_phase = {k: ms / n for k, (ms, n) in jacap.timing_stop().items()}
    dominant = max(per_phase, key=per_phase.get)

    # Timed region: K steps; the library records the dominant phase only.
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    flush_buf = torch.ones(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda") if args.flush else None
    flush_sink = torch.zeros((), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    jacap.timing_start([dominant])
    t_wall = time.perf_counter()
    for s, e in ev:
        if flush_buf is not None:
            torch.sum(flush_buf, dim=0, out=flush_sink)   # evicts the MALL; outside the events
        s.record(stream)
        run()
        e.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    dom_ms, dom_calls = jacap.timing_stop()[dominant]
    dom_avg = dom_ms / dom_calls
    times = np.array([s.elapsed_time(e) for s, e in ev])   # ms
    ms = float(times.mean())

    esize = case.k.element_size()
    d = w.head_dim
    entries = case.total_tokens * w.num_layers * w.num_kv_heads
    step_bytes = 2 * entries * d * esize                   # K and V read once
    tokens_per_s = case.total_tokens / (ms * 1e-3)
    dom_bytes = phase_bytes(dominant, case, budget, prob)
    achieved = dom_bytes / (dom_avg * 1e-3) / 1e9 if dom_bytes else None
    traffic = recorded_traffic(traffic_key(dominant, args.cov, args.gqa, w, case), w.name)
    # measured ceiling for streaming reads: the probe over the K cache
    probe_bytes, probe_gbs = read_probe(jacap, case.k, stream)

    out = {
        "metric": METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "ms_per_step_min": float(times.min()),
        "ms_per_step_median": float(np.median(times)),
        "wall_s": wall,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "entries_per_s": entries / (ms * 1e-3),
        "status_flags": flags,
        "config": {
            "workload": w.name, "num_seqs": case.num_seqs, "layers": w.num_layers,
            "kv_heads": w.num_kv_heads, "q_heads": w.num_q_heads, "head_dim": d,
            "tokens": case.total_tokens, "window": w.window, "budget_k": budget,
            "tau": args.tau, "ridge": args.ridge, "cov_mode": args.cov, "gqa": args.gqa,
            "inplace": args.inplace,
            "cache": "flushed before every step" if args.flush else (
                "warm (inputs fit in the 256 MB MALL)" if step_bytes < (256 << 20) else
                "cold (inputs exceed the MALL)"),
        },
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": achieved / PEAK_HBM_GBS if achieved else None, "traffic": traffic,
            "kernel": dominant, "kernel_ms": dom_avg, "kernel_launches": dom_calls,
            "alg_bytes_per_launch": dom_bytes,
            "traffic_over_alg": traffic / dom_bytes if traffic and dom_bytes else None,
            "frac_of_probe": achieved / probe_gbs if achieved else None,
            "pass": {"achieved": step_bytes / (ms * 1e-3) / 1e9, "peak": PEAK_HBM_GBS,
                     "frac": step_bytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                     "bytes_per_step": step_bytes,
                     "note": "score+select+compact pass: K and V bytes read once / step time"},
        },
        "read_probe": {"gbs": probe_gbs, "bytes": probe_bytes,
                       "kind": "jacap_stream_read over the K cache: non-temporal 16-byte "
                               "loads, whole lines per wave instruction, 1 MiB per workgroup"},
        "phases_ms": {k: round(v, 4) for k, v in per_phase.items()},
        "step_hbm_gbs": step_bytes / (ms * 1e-3) / 1e9,
        "step_frac": step_bytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
    }
    if not args.no_cpu_baseline:
        cb = cpu_baseline(case, budget, args.tau, args.ridge, args.cpu_seconds, args.cov, args.gqa)
        cb["gpu_speedup"] = tokens_per_s / cb["value"]
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
