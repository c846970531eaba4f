#!/usr/bin/env python3
"""Benchmark of the Hypic GDN hot path on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
segment build (o, S_seg, P_hat, log_decay for every segment and head), Eq. (6)
composition of the batch's segments in order behind the prefix state
(emitting the state entering each segment) and the seam rescan of every
segment's first w tokens from that state.  The headline workload is the
long-context RAG shape: 32 segments of 4096 bf16 tokens, 16 q/k heads shared by
32 v heads, d_k = d_v = 128, alpha ~ U(0.9, 1), composed behind the state of a
1024-token prefix, seam w = 8 (the paper's default window).  value = tokens / s
over the K timed steps, inputs resident in HBM.

Also reported (each a sub-key of the one JSON line):
  roofline      the build scan kernel: algorithmic FLOP per launch (the chunk
                products of every v-head, the K K^T and Q K^T Gram counted once
                per q/k head) over the median of its launch durations (HIP
                events on the launch stream around the build inside every timed
                step), against the dense bf16 matrix-core peak;
  layer_bf16    the 16-head, 8 x 2048-token layer workload, same step;
  agentic       64 ragged segments (log-uniform 128..16384 tokens), seam w = 32;
  compose_burst serve-time burst: 256 requests x U{8..64} segments of a
                512-entry float32 pool, then a w = 64 seam per listed segment;
                compositions / s, the composition kernel's HBM roofline;
  families, kda, adjacent   the Tab. 1 transition families, the KDA row and the
                reuse-time steps;
  cpu_baseline  the float64 oracle on the host cores on a bounded sample of the
                headline workload, and its compositions / s on burst requests.

Before each timed loop the leg warms up by time: its warm-up steps, then batches
of builds until two consecutive batch times agree within 1 % (the clocks have
settled), whatever --warmup says.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""

import argparse
import gc
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

from paper_2607_01299_amd import workloads as W  # noqa: E402

METRIC = "segment-build tokens/s + MFMA util; compositions/s + HBM GB/s (1 MI355X)"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
HEADLINE_CFG = 3
HEADLINE_SEAM_W = 8   # the paper's seam window (Sec. 6)
AGENTIC_SEAM_W = 32


# Algorithmic work of the chunked scan per (token, v-head) at chunk C:
#   2C(3 d_k + 2 d_v)   K K^T, Q K^T, W, U, (Q K^T . Gamma) Vn
#   6 d_k d_v           W' S0, Q S0, K^T Vn
#   4 d_k^2             W P0, K^T X (operator path)
def flop_per_token_head(d_k, d_v, chunk):
    return 2 * chunk * (3 * d_k + 2 * d_v) + 6 * d_k * d_v + 4 * d_k * d_k


def gram_flop_per_token(d_k, chunk):
    """K K^T and Q K^T per token of one q/k head: shared by the v-heads of a
    grouped-head (GVA) group, so counted once per q/k head."""
    return 4 * chunk * d_k


def build_flop(T, h_qk, h_v, d_k, d_v, chunk):
    """Algorithmic FLOP of one build launch over T tokens."""
    per_v = flop_per_token_head(d_k, d_v, chunk) - gram_flop_per_token(d_k, chunk)
    return float(T) * (h_v * per_v + h_qk * gram_flop_per_token(d_k, chunk))


CSRC = os.path.join(HERE, "paper_2607_01299_amd", "csrc")
TRAFFIC_FILE = os.path.join(HERE, "profiles", "hbm_traffic.json")
MFMA_FILE = os.path.join(HERE, "profiles", "mfma_counters.json")
KERNEL_SOURCES = {
    "scan_bf16": ["scan_bf16.hip", "frag32.hpp", "mfma.hpp", "scan.hpp"],
    "compose": ["compose.hip", "mfma.hpp", "scan.hpp"],
    "family_scalar_build": ["gated_pipe.hip", "frag32.hpp", "mfma.hpp", "family.hpp", "scan.hpp"],
    "family_diagonal_build": ["gated_pipe.hip", "frag32.hpp", "mfma.hpp", "family.hpp", "scan.hpp"],
    "family_scalar_compose": ["family.hip", "mfma.hpp", "family.hpp", "scan.hpp", "frag_common.hpp"],
    "family_diagonal_compose": ["family.hip", "mfma.hpp", "family.hpp", "scan.hpp", "frag_common.hpp"],
    "kda_build": ["kda.hip", "kda.hpp", "scan.hpp", "mfma.hpp", "frag_common.hpp"],
}
FAMILY_WORKLOAD = W.CONFIG_NAMES[2] + "; gates from workloads.family_gate (softplus)"
FAMILY_BURST_WORKLOAD = W.CONFIG_NAMES[5] + " (family tuples)"
KDA_WORKLOAD = W.CONFIG_NAMES[2] + "; per-channel gates from workloads.family_gate (diagonal, softplus)"


def _code_only(src):
    """Source text without comments, blank lines or indentation."""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    return "\n".join(ln.strip() for ln in src.splitlines() if ln.strip())


def kernel_source_sha256(kernel):
    """Hash of a kernel's code (comments and layout ignored), so a counter
    record stays valid across comment-only edits and lapses on any code change."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(CSRC, name), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def _record(path, kernel, workload):
    """The committed counter record of `kernel` (a KERNEL_SOURCES key) on
    `workload`, or None when there is none or the kernel's code changed since."""
    try:
        with open(path) as f:
            recs = json.load(f)
    except (OSError, ValueError):
        return None
    for key, rec in recs.items():
        if rec.get("source", key) != kernel or rec.get("workload") != workload:
            continue
        if rec.get("src_sha256") != kernel_source_sha256(kernel):
            return None
        return rec
    return None


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    passes (scaled by a plain copy of known size), or None."""
    rec = _record(TRAFFIC_FILE, kernel, workload)
    if rec is None:
        return None
    return float(rec["fetch_bytes_per_launch"]) + float(rec["write_bytes_per_launch"])


def measured_mfma(kernel, workload):
    """Matrix-core counters of a kernel from the committed rocprofv3 passes
    (MfmaUtil: MFMA-busy cycles over active cycles x SIMDs; bf16 MFMA ops x 512),
    or None."""
    rec = _record(MFMA_FILE, kernel, workload)
    if rec is None:
        return None
    out = {"mfma_busy_frac": float(rec["mfma_util_pct"]) / 100.0}
    if rec.get("mfma_bf16_flop_per_launch") is not None:
        out["mfma_flop_per_launch"] = float(rec["mfma_bf16_flop_per_launch"])
        out["mfma_over_algorithmic"] = float(rec["counted_over_algorithmic"])
    return out


def copy_calibration(torch, nbytes=1 << 30, reps=3):
    """A plain device-to-device copy of known size, for scaling HBM counters."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}))


def compose_bytes_per_head_step(d_k, d_v, write_incoming=True):
    # read P_hat_i and S_i and log_decay_i; optionally write the incoming state
    return 4 * (d_k * d_k + d_k * d_v * (2 if write_incoming else 1)) + 4


def hbm_roofline(alg_bytes, ms, kernel, workload, record_key=None):
    """HBM roofline of one launch: `frac` from the counted HBM bytes when a
    record of the current kernel code exists (never above the bytes the
    counters saw), else from the algorithmic bytes; both fractions reported."""
    traffic = measured_traffic(record_key or kernel, workload) if kernel else None
    alg_gbs = alg_bytes / (ms * 1e-3) / 1e9
    out = {"bound": "hbm", "peak": PEAK_HBM_GBS, "unit": "GB/s", "traffic": traffic,
           "bytes_per_launch": alg_bytes, "achieved_algorithmic": alg_gbs,
           "frac_algorithmic": alg_gbs / PEAK_HBM_GBS}
    counted = alg_bytes if traffic is None else min(alg_bytes, traffic)
    out["achieved"] = counted / (ms * 1e-3) / 1e9
    out["frac"] = out["achieved"] / PEAK_HBM_GBS
    if traffic is None and out["frac"] > 1.0:
        # more algorithmic bytes than HBM can deliver in this time: caches serve
        # re-reads, and without a counter record of this kernel code the HBM
        # share is unknown
        out["achieved"] = out["frac"] = None
        out["note_frac"] = ("algorithmic bytes above the HBM peak (re-reads served by the "
                            "caches); no counter record of the current kernel code")
    return out


# ---------------------------------------------------------------------------
# CPU baseline: the oracle, run before the GPU is touched
# ---------------------------------------------------------------------------

_CPU = {}  # the workloads, inherited by the forked workers (read only)


def _oracle_build_pair(pair):
    import oracle
    seg, head = pair
    w = _CPU["build"]
    lo, hi = int(w["cu_seqlens"][seg]), int(w["cu_seqlens"][seg + 1])
    sl = slice(lo, hi)
    oracle.build_segments(w["q"][sl], w["k"][sl], w["v"][sl], w["beta"][sl],
                          w["log_alpha"][sl], [0, hi - lo], seg_head_pairs=[(0, head)])
    return hi - lo


def _oracle_burst_pair(pair):
    """One (request, head) of the burst: Eq. (6) over the request's segments and
    the w = 64 seam of each from its incoming state.  Returns the number of
    head-steps."""
    import oracle
    r, h = pair
    p = _CPU["pool"]
    off = p["req_offsets"]
    lo, hi = int(off[r]), int(off[r + 1])
    ids = p["seg_ids"][lo:hi]
    _, S_inc = oracle.compose(p["P_hat"], p["log_decay"], p["S_seg"], ids, [0, hi - lo],
                              req_head_pairs=[(0, h)])
    t = p["tokens"]
    oracle.seam(t["q"], t["k"], t["v"], t["beta"], t["log_alpha"], p["tok_start"][lo:hi],
                p["tok_len"][lo:hi], p["w"], S_inc,
                entry_head_pairs=[(e, h) for e in range(hi - lo)])
    return hi - lo


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(build_w, pool_w, build_s=12.0, burst_s=6.0):
    """The oracle on the host cores: (segment, head) builds of the headline
    workload (state and operator, float64 token recurrence), and (request,
    head) pairs of the burst (Eq. (6) composition plus the w = 64 seams), each
    for about `build_s` / `burst_s` seconds of wall time.  Worker processes are
    forked with the workloads in memory, one BLAS thread each."""
    import multiprocessing as mp
    affinity = len(os.sched_getaffinity(0))
    # a one-GPU host share is 16 cores, whatever the affinity mask shows
    workers = max(1, min(affinity, 16))
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = "1"
    _CPU["build"] = build_w
    _CPU["pool"] = pool_w
    n_seg = len(build_w["cu_seqlens"]) - 1
    h_v = int(build_w["v"].shape[1])
    distinct = [(s, h) for h in range(h_v) for s in range(n_seg)]
    ctx = mp.get_context("fork")
    with ctx.Pool(workers) as pool:
        # one round to time a pair, then rounds sized to the wall-time budget
        t0 = time.perf_counter()
        toks = pool.map(_oracle_build_pair, distinct[:workers])
        per_round = time.perf_counter() - t0
        rounds = max(1, int(build_s / max(per_round, 1e-3)))
        pairs = [distinct[(workers + i) % len(distinct)] for i in range(rounds * workers)]
        t0 = time.perf_counter()
        toks = pool.map(_oracle_build_pair, pairs)
        dt = time.perf_counter() - t0
        n_req = len(pool_w["req_offsets"]) - 1
        h_b = int(pool_w["S_seg"].shape[1])
        bursts = [(r, h) for r in range(n_req) for h in range(h_b)]
        t0 = time.perf_counter()
        head_steps = sum(pool.map(_oracle_burst_pair, bursts[:workers]))
        per_round = time.perf_counter() - t0
        rounds = max(1, int(burst_s / max(per_round, 1e-3)))
        sample = [bursts[(workers + i) % len(bursts)] for i in range(rounds * workers)]
        t0 = time.perf_counter()
        head_steps = sum(pool.map(_oracle_burst_pair, sample))
        dt_burst = time.perf_counter() - t0
    token_heads = float(sum(toks))
    return {
        "value": token_heads / dt / h_v,
        "unit": "tokens/s",
        "cores": workers,
        "kind": "oracle",
        "sample": "%d (segment, head) builds of %d tokens of the headline workload (state and "
                  "operator, float64 token recurrence; its %d distinct pairs, cycled) on %d "
                  "processes, %.1f s; tokens/s = token-heads/s / %d v-heads"
                  % (len(pairs), int(toks[0]), len(distinct), workers, dt, h_v),
        "cpu_model": cpu_model(),
        "affinity_cores": affinity,
        "compositions_per_s": head_steps / h_b / dt_burst,
        "compositions_sample": "%d (request, head) pairs of the burst (%d head-steps: float64 "
                               "Eq. (6) and the w = 64 seam of each listed segment) on %d "
                               "processes, %.1f s; compositions/s = head-steps/s / %d heads"
                               % (len(sample), head_steps, workers, dt_burst, h_b),
    }


# ---------------------------------------------------------------------------
# GPU legs
# ---------------------------------------------------------------------------

def _to_dev(w, torch):
    dt = torch.bfloat16 if w["dtype"] == W.BF16 else torch.float32
    q = torch.from_numpy(w["q"]).cuda().to(dt).contiguous()
    k = torch.from_numpy(w["k"]).cuda().to(dt).contiguous()
    v = torch.from_numpy(w["v"]).cuda().to(dt).contiguous()
    beta = torch.from_numpy(w["beta"]).cuda().contiguous()
    la = torch.from_numpy(w["log_alpha"]).cuda().contiguous()
    return q, k, v, beta, la


def _events_ms(torch, stream, fn, reps):
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def settle(torch, stream, step, warmup, batch=10, min_s=0.3, max_s=8.0, tol=0.01):
    """Warm up by time: `warmup` steps, then batches of `batch` steps until two
    consecutive batch times agree within `tol` (after at least `min_s` seconds,
    at most `max_s`).  Returns (seconds, steps)."""
    t0 = time.perf_counter()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    n, prev = warmup, None
    while True:
        ms = _events_ms(torch, stream, step, batch)
        n += batch
        el = time.perf_counter() - t0
        if el > max_s or (el > min_s and prev is not None and abs(ms - prev) <= tol * prev):
            return el, n
        prev = ms


def _gpu_prefix_state(torch, w):
    """The state after the workload's prefix tokens, built on the GPU (untimed
    set-up; the parity tests check the same state against the oracle)."""
    from paper_2607_01299_amd import ops
    p = w["prefix"]
    dt = torch.bfloat16 if w["dtype"] == W.BF16 else torch.float32
    q, k, v = [torch.from_numpy(p[key]).cuda().to(dt).contiguous() for key in ("q", "k", "v")]
    beta = torch.from_numpy(p["beta"]).cuda().contiguous()
    la = torch.from_numpy(p["log_alpha"]).cuda().contiguous()
    res = ops.build_segment(q, k, v, beta, la, [0, q.shape[0]], want_operator=False,
                            want_o=False)
    torch.cuda.synchronize()
    return res["S_seg"]


def bench_step(torch, w, steps, warmup, seam_w):
    """One workload's step (build, composition behind its prefix, seams): K timed
    steps with events around each launch on the pipeline's stream."""
    from paper_2607_01299_amd.pipeline import SegmentPipeline
    cfg = int(w["cfg"])
    q, k, v, beta, la = _to_dev(w, torch)
    S_prefix = _gpu_prefix_state(torch, w) if "prefix" in w else None
    pipe = SegmentPipeline(q, k, v, beta, la, w["cu_seqlens"], chunk=w["chunk"], seam_w=seam_w,
                           S_prefix=S_prefix)
    stream = pipe.stream
    warm_s, warm_n = settle(torch, stream, pipe.run, warmup)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(stream)
        pipe.build()
        ev[i][1].record(stream)
        pipe.compose()
        ev[i][2].record(stream)
        pipe.seam()
        ev[i][3].record(stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    build = [e[0].elapsed_time(e[1]) for e in ev]
    comp = [e[1].elapsed_time(e[2]) for e in ev]
    seam = [e[2].elapsed_time(e[3]) for e in ev]
    stepms = [e[0].elapsed_time(e[3]) for e in ev]
    # the same step replayed as one HIP graph, for reference
    pipe.capture()
    for _ in range(3):
        pipe.replay()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(steps):
        pipe.replay()
    torch.cuda.synchronize()
    dt_graph = time.perf_counter() - t1
    T = int(w["cu_seqlens"][-1])
    h_qk, h_v = int(w["q"].shape[1]), int(w["v"].shape[1])
    d_k, d_v = int(w["d_k"]), int(w["d_v"])
    flop = build_flop(T, h_qk, h_v, d_k, d_v, w["chunk"])
    build_ms = float(np.median(build))
    achieved = flop / (build_ms * 1e-3) / 1e12
    name = W.CONFIG_NAMES[cfg]
    n_comp = len(w["lengths"])
    comp_ms = float(np.median(comp))
    comp_bytes = float(compose_bytes_per_head_step(d_k, d_v, write_incoming=False)) * n_comp * h_v
    out = {
        "ms_per_step": dt / steps * 1e3,
        "ms_per_step_median": float(np.median(stepms)),
        "ms_per_step_graph": dt_graph / steps * 1e3,
        "tokens": T,
        "tokens_per_s": T / (dt / steps),
        "build_ms": build_ms,
        "build_ms_mean": float(np.mean(build)),
        "compose_us": comp_ms * 1e3,
        "seam_us": float(np.median(seam)) * 1e3,
        "warmup_s": warm_s,
        "warmup_steps": warm_n,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": measured_traffic("scan_bf16", name),
                     "counter": measured_mfma("scan_bf16", name),
                     "kernel": "scan_bf16_kernel (segment build)",
                     "flop_per_launch": flop,
                     "timing": "median of %d launch durations (HIP events inside the timed steps)"
                               % steps},
        "compose_roofline": {"bound": "latency (one chained request)",
                             "achieved_algorithmic": comp_bytes / (comp_ms * 1e-3) / 1e9,
                             "unit": "GB/s", "bytes_per_launch": comp_bytes,
                             "kernel": "compose_kernel"},
        "config": {"workload": name, "segments": len(w["lengths"]), "tokens": T, "h_qk": h_qk,
                   "h_v": h_v, "d_k": d_k, "d_v": d_v, "chunk": w["chunk"], "seam_w": seam_w,
                   "prefix_tokens": (int(w["prefix"]["q"].shape[0]) if "prefix" in w else 0),
                   "seed": w["seed"]},
    }
    del pipe
    return out


def bench_compose_burst(torch, steps, warmup):
    from paper_2607_01299_amd.pipeline import ComposeBurst, SeamAdvanceBurst
    p = W.pool_workload()
    dev = "cuda"
    P = torch.from_numpy(p["P_hat"]).to(dev)
    g = torch.from_numpy(p["log_decay"]).to(dev)
    S = torch.from_numpy(p["S_seg"]).to(dev)
    t = p["tokens"]
    toks = (torch.from_numpy(t["q"]).to(dev).to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["k"]).to(dev).to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["v"]).to(dev).to(torch.bfloat16).contiguous(),
            torch.from_numpy(t["beta"]).to(dev), torch.from_numpy(t["log_alpha"]).to(dev))
    burst = ComposeBurst(P, g, S, p["seg_ids"], p["req_offsets"], toks, p["tok_start"],
                         p["tok_len"], p["w"])
    stream = burst.stream
    settle(torch, stream, burst.run, warmup, batch=3, min_s=0.3)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(stream)
        burst.compose()
        ev[i][1].record(stream)
        burst.seam()
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    comp_ms = float(np.median([e[0].elapsed_time(e[1]) for e in ev]))
    seam_ms = float(np.median([e[1].elapsed_time(e[2]) for e in ev]))
    nnz, h_v = burst.nnz, burst.h_v
    name = W.CONFIG_NAMES[5]
    # the composition's own bytes: P_hat_i, S_i and log_decay_i read per
    # head-step (131,076 B at d = 128); this launch also writes the incoming
    # state that the separate seam launch reads
    alg = float(compose_bytes_per_head_step(burst.d_k, burst.d_v, False)) * nnz * h_v
    alg_inc = float(compose_bytes_per_head_step(burst.d_k, burst.d_v, True)) * nnz * h_v
    roof = hbm_roofline(alg, comp_ms, None, name)
    traffic = measured_traffic("compose", name)
    roof.update({"traffic": traffic, "kernel": "compose_kernel",
                 "bytes_per_launch_with_incoming": alg_inc,
                 "frac_with_incoming": alg_inc / (comp_ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                 "counter": measured_mfma("compose", name),
                 "note": "frac counts the 131,076 B per head-step the composition needs; "
                         "frac_with_incoming adds the incoming-state write the separate seam "
                         "launch reads"})
    two_launch = {"ms_per_burst": dt / steps * 1e3, "compositions_per_s": nnz / (dt / steps),
                  "compose_ms": comp_ms, "seam_ms": seam_ms, "roofline": roof,
                  "note": "compose_kernel writing the incoming states, then the seam launch"}
    # the composition alone (S_out, no incoming states: the launch a caller
    # that needs no seam makes), the same kernel
    states_ms = _events_ms(torch, stream, burst.compose_states, max(steps // 2, 4))
    states_roof = hbm_roofline(alg, states_ms, None, name)
    states_roof["kernel"] = "compose_kernel (S_incoming = NULL)"
    two_launch["compose_states_only"] = {
        "ms": states_ms, "compositions_per_s": nnz / (states_ms * 1e-3), "roofline": states_roof,
        "note": "Eq. (6) to S_out without the incoming-state writes; frac by the composition's "
                "131,076 B per head-step"}
    # the same burst in one pass (hypic_compose_and_rescan): each (request,
    # head) keeps its state on chip; the seam of each entry from its incoming
    # state, then Eq. (4)
    one = SeamAdvanceBurst(P, g, S, p["seg_ids"], p["req_offsets"], toks, p["tok_start_pool"],
                           p["seam_len_pool"], p["w"], advance=False)
    settle(torch, one.stream, one.run, 1, batch=3, min_s=0.3)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(one.stream)
        one.run()
        ev[i][1].record(one.stream)
    torch.cuda.synchronize()
    dt1 = time.perf_counter() - t0
    one_ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del one
    seam_bytes = float(p["w"] * (2 * 2 * burst.d_k + 2 * burst.d_v + 8 + 2 * burst.d_v))
    one_roof = hbm_roofline(alg, one_ms, None, name)
    one_roof.update({"kernel": "scan_bf16_kernel (composition with seams, one pass)",
                     "bytes_per_launch_with_seams": alg + seam_bytes * nnz * h_v,
                     "frac_with_seams": (alg + seam_bytes * nnz * h_v) / (one_ms * 1e-3) / 1e9
                                        / PEAK_HBM_GBS,
                     "note": "frac counts the 131,076 B per head-step the composition needs; "
                             "frac_with_seams adds each seam's tokens read and outputs written"})
    # the same requests with seams that advance the state (Sec. 4.3): the pool
    # tuples read as tail tuples, each entry's 64 tokens as its seam
    adv = SeamAdvanceBurst(P, g, S, p["seg_ids"], p["req_offsets"], toks, p["tok_start_pool"],
                           p["seam_len_pool"], p["w"])
    adv.run()
    adv1_ms = _events_ms(torch, adv.stream, adv.run, max(steps // 2, 2))
    del adv
    adv = SeamAdvanceBurst(P, g, S, p["seg_ids"], p["req_offsets"], toks, p["tok_start_pool"],
                           p["seam_len_pool"], p["w"], lanes=2)
    adv.run()
    adv_ms = _events_ms(torch, adv.stream, adv.run, max(steps // 2, 2))
    del adv
    return {
        "compositions_per_s": nnz / (dt1 / steps),
        "requests_per_s": burst.n_req / (dt1 / steps),
        "ms_per_burst": dt1 / steps * 1e3,
        "ms_per_burst_median": one_ms,
        "roofline": one_roof,
        "two_launch": two_launch,
        "seam_advance": {"ms_per_burst": min(adv_ms, adv1_ms),
                         "compositions_per_s": nnz / (min(adv_ms, adv1_ms) * 1e-3),
                         "ms_per_burst_one_call": adv1_ms, "ms_per_burst_two_lanes": adv_ms,
                         "note": "seams run from the running state, then tail tuples (Sec. 4.3), "
                                 "one pass"},
        "config": {"workload": name, "requests": burst.n_req,
                   "compositions": nnz, "pool": int(p["n_pool"]), "h_v": h_v,
                   "d_k": burst.d_k, "d_v": burst.d_v, "seam_w": p["w"], "seed": p["seed"]},
    }


def family_build_bytes(family, T, h_qk, h_v, d_k, d_v, n_seg):
    """Algorithmic HBM bytes of one family build launch: q, k, v read and o
    written in bf16, the gates read in float32, S_seg and log_decay written."""
    g = 1 if family == "scalar" else d_k
    return (T * (2 * h_qk * d_k * 2 + 2 * h_v * d_v * 2 + h_v * g * 4)
            + n_seg * h_v * (d_k * d_v * 4 + g * 4))


def family_compose_bytes_per_head_step(family, d_k, d_v):
    # read S_i and log_decay_i, write the incoming state
    return 2 * 4 * d_k * d_v + 4 * (1 if family == "scalar" else d_k)


def bench_families(torch, steps, warmup, seam_w):
    """Scalar and diagonal families (Tab. 1) on the layer workload: the whole
    family step (build, composition of the batch in order, seams) and the
    build kernel's HBM roofline; then a serve-time burst over a pool of family
    tuples with the burst's request lists."""
    from paper_2607_01299_amd.pipeline import FamilyComposeBurst, FamilyPipeline
    w = W.segment_workload(2)
    q, k, v, _, _ = _to_dev(w, torch)
    T = int(w["cu_seqlens"][-1])
    h_qk, h_v, d_k, d_v = int(w["q"].shape[1]), int(w["v"].shape[1]), w["d_k"], w["d_v"]
    n_seg = len(w["lengths"])
    p = W.pool_workload()
    S_pool = torch.from_numpy(p["S_seg"]).cuda()
    out = {}
    for family in ("scalar", "diagonal"):
        gate = torch.from_numpy(W.family_gate(family, T, h_v, d_k, w["seed"] + 1000)).cuda()
        pipe = FamilyPipeline(family, q, k, v, gate, w["cu_seqlens"], seam_w=seam_w)
        settle(torch, pipe.stream, pipe.run, warmup)
        t0 = time.perf_counter()
        for _ in range(steps):
            pipe.run()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / steps
        build_ms = _events_ms(torch, pipe.stream, pipe.build, steps)
        byts = float(family_build_bytes(family, T, h_qk, h_v, d_k, d_v, n_seg))
        # pool of family tuples: the burst's states, per-channel or scalar
        # log-decays ~ U(-3, 0)
        rng = np.random.default_rng(p["seed"] + 7)
        ld_shape = (p["n_pool"], h_v) if family == "scalar" else (p["n_pool"], h_v, d_k)
        ld = torch.from_numpy(rng.uniform(-3.0, 0.0, size=ld_shape).astype(np.float32)).cuda()
        burst = FamilyComposeBurst(family, ld, S_pool, p["seg_ids"], p["req_offsets"])
        burst.compose()
        comp_ms = _events_ms(torch, burst.stream, burst.compose, max(steps // 2, 3))
        cbytes = float(family_compose_bytes_per_head_step(family, d_k, d_v)) * burst.nnz * h_v
        croof = hbm_roofline(cbytes, comp_ms, "family_%s_compose" % family,
                             FAMILY_BURST_WORKLOAD)
        croof.update({"kernel": "family_compose_kernel",
                      "note": "frac counts the HBM bytes the FETCH/WRITE counters saw; pool "
                              "re-reads served by L2 and the memory-side cache are the gap "
                              "to frac_algorithmic"})
        broof = hbm_roofline(byts, build_ms, "family_%s_build" % family, FAMILY_WORKLOAD)
        broof["kernel"] = ("scalar_pipe_kernel (build)" if family == "scalar"
                           else "diag_pipe_kernel (build)")
        out[family] = {
            "tokens_per_s": T / dt,
            "ms_per_step": dt * 1e3,
            "build_ms": build_ms,
            "roofline": broof,
            "compose_burst": {"compositions_per_s": burst.nnz / (comp_ms * 1e-3),
                              "compose_ms": comp_ms, "roofline": croof},
        }
        del pipe, burst
    return {"workload": FAMILY_WORKLOAD, "burst_workload": FAMILY_BURST_WORKLOAD, **out}


def kda_flops(d_k, d_v, chunk):
    """Algorithmic FLOPs per (token, v-head) of the chunked KDA build, split
    into the state columns (the Gram K K^T and the A tiles, Y = (K . e^B) S0, N,
    Q S0, A N, K^T N) and the operator columns (Y and N of P_hat, K^T N_P).
    The total equals the GDN count of flop_per_token_head."""
    state = 2 * chunk * (2 * d_k + 2 * d_v) + 6 * d_k * d_v
    operator = 2 * chunk * d_k + 4 * d_k * d_k
    return state, operator


def bench_kda(torch, steps, warmup):
    """KDA row of Tab. 1 on the layer workload (16 heads, d = 128, 8 x 2048 bf16
    tokens, per-channel gates from the diagonal-family generator): the build with
    its operator, timed with HIP events over back-to-back launches.  Every
    product runs on the bf16 matrix cores (the operator columns and the
    intra-chunk scores as three split passes), so the roofline peak is the bf16
    one, as for the GDN build."""
    from paper_2607_01299_amd.pipeline import KdaPipeline
    w = W.segment_workload(2)
    q, k, v, beta, _ = _to_dev(w, torch)
    T = int(w["cu_seqlens"][-1])
    h_v, d_k, d_v = int(w["v"].shape[1]), w["d_k"], w["d_v"]
    gate = torch.from_numpy(W.family_gate("diagonal", T, h_v, d_k, w["seed"] + 2000)).cuda()
    pipe = KdaPipeline(q, k, v, beta, gate, w["cu_seqlens"])
    settle(torch, pipe.stream, pipe.build, warmup)
    ms = _events_ms(torch, pipe.stream, pipe.build, steps)
    f_state, f_op = kda_flops(d_k, d_v, 64)
    flop = float(f_state + f_op) * T * h_v
    achieved = flop / (ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS
    return {"workload": KDA_WORKLOAD,
            "tokens_per_s": T / (ms * 1e-3), "build_ms": ms,
            "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                         "frac": achieved / peak,
                         "traffic": measured_traffic("kda_build", KDA_WORKLOAD),
                         "kernel": "kda_scan_kernel (state and operator launches)",
                         "flop_per_launch": flop,
                         "flop_split": {"state": float(f_state) * T * h_v,
                                        "operator": float(f_op) * T * h_v}}}


def bench_adjacent(torch, steps):
    """The reuse-time steps next to the cache, each an HBM stream: the Eq. (7)
    state shift over the 512-entry serve-time pool, the Eq. (8) re-rotation of
    32 x 4096 cached bf16 keys (16 heads, d = 128) and the width-4 causal conv
    over the q, k, v channels (6144) of 8 x 2048 bf16 tokens.  Inputs are drawn
    on the device (timing only)."""
    from paper_2607_01299_amd import ops
    g = torch.Generator(device="cuda").manual_seed(W.SEED_BASE + 9)
    out = {}

    def leg(name, fn, byts, workload):
        fn()
        ms = _events_ms(torch, torch.cuda.current_stream(), fn, steps)
        roof = hbm_roofline(byts, ms, None, workload)
        out[name] = {"ms": ms, "workload": workload, "roofline": roof}

    S = torch.randn((512, 16, 128, 128), device="cuda", generator=g)
    S_out = torch.empty_like(S)
    delta = torch.arange(512, dtype=torch.int32, device="cuda") * 1024
    leg("rope_shift_state", lambda: ops.rope_shift_state(S, delta, out=S_out),
        2.0 * S.numel() * 4, "512 x 16 heads x 128 x 128 float32 states")
    del S, S_out
    k = torch.randn((32 * 4096, 16, 128), device="cuda", generator=g).to(torch.bfloat16)
    k_out = torch.empty_like(k)
    cu = W.cu_from_lengths([4096] * 32)
    cu_d = torch.from_numpy(cu).cuda()
    dl = torch.arange(32, dtype=torch.int32, device="cuda") * 4096
    leg("rope_rerotate_keys", lambda: ops.rope_rerotate_keys(k, cu, dl, out=k_out,
                                                             cu_seqlens_dev=cu_d),
        2.0 * k.numel() * 2, "32 x 4096 tokens x 16 heads x 128 bf16 keys")
    del k, k_out
    x = torch.randn((8 * 2048, 6144), device="cuda", generator=g).to(torch.bfloat16)
    wt = torch.randn((6144, 4), device="cuda", generator=g) * 0.5
    cu = W.cu_from_lengths([2048] * 8)
    cu_d = torch.from_numpy(cu).cuda()
    leg("causal_conv", lambda: ops.causal_conv(x, wt, cu, cu_seqlens_dev=cu_d),
        2.0 * x.numel() * 2 + wt.numel() * 4 + 2 * 8 * 3 * 6144 * 4,
        "8 x 2048 tokens x 6144 bf16 channels, width 4, SiLU")
    return out


def _say(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=HEADLINE_CFG, choices=[2, 3, 4],
                    help="workload of the headline step (default: the long-context RAG shape)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--headline-only", action="store_true",
                    help="only the headline step (profiling)")
    ap.add_argument("--no-burst", action="store_true")
    ap.add_argument("--no-families", action="store_true",
                    help="skip the family, KDA and reuse-time-step legs")
    ap.add_argument("--families-only", action="store_true",
                    help="run only the family and reuse-time-step legs (profiling)")
    ap.add_argument("--no-segments", action="store_true",
                    help="run only the burst (profiling)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 1 GiB device copy (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(segments would shard across GPUs with no exchange). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        import torch
        copy_calibration(torch)
        return

    seam_w = {3: HEADLINE_SEAM_W, 2: HEADLINE_SEAM_W, 4: AGENTIC_SEAM_W}[args.config]
    head_w = None
    if not (args.families_only or args.no_segments):
        head_w = W.segment_workload(args.config)
        _say("headline workload drawn: %s" % W.CONFIG_NAMES[args.config])
    cpu = None
    if not args.no_cpu_baseline and head_w is not None and not args.headline_only:
        cpu = cpu_baseline(head_w, W.pool_workload())
        _say("cpu baseline done: %.1f tokens/s, %.1f compositions/s"
             % (cpu["value"], cpu["compositions_per_s"]))

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_2607_01299_amd import _lib
    _lib.load()
    # Python's cyclic collector stays off in the GPU legs, as timeit keeps it
    # off: a full collection of the interpreter's objects stalls the host for
    # 40-60 ms, and one such pause inside a timed loop of short launches lets
    # the queue drain
    gc.collect()
    gc.freeze()
    gc.disable()
    if args.families_only:
        print(json.dumps({"families": bench_families(torch, max(args.steps, 100), args.warmup,
                                                     HEADLINE_SEAM_W),
                          "kda": bench_kda(torch, max(args.steps, 100), args.warmup),
                          "adjacent": bench_adjacent(torch, max(args.steps, 100))}))
        return
    if args.no_segments:
        burst = bench_compose_burst(torch, max(args.steps // 2, 3), max(args.warmup // 2, 1))
        print(json.dumps({"compose_burst": burst}))
        return

    seg = bench_step(torch, head_w, args.steps, args.warmup, seam_w)
    _say("headline step done: %.3f ms/step, build %.3f ms" % (seg["ms_per_step"],
                                                                seg["build_ms"]))
    del head_w
    subs = {}
    if not args.headline_only:
        for cfg, key, sw in ((2, "layer_bf16", HEADLINE_SEAM_W), (4, "agentic", AGENTIC_SEAM_W)):
            if cfg == args.config:
                continue
            wl = W.segment_workload(cfg)
            subs[key] = bench_step(torch, wl, max(args.steps, 50), args.warmup, sw)
            del wl
            _say("%s step done: %.3f ms/step" % (key, subs[key]["ms_per_step"]))
        if not args.no_burst:
            subs["compose_burst"] = bench_compose_burst(torch, max(args.steps // 2, 6),
                                                        max(args.warmup // 2, 1))
            _say("burst done: %.2f ms" % subs["compose_burst"]["ms_per_burst"])
        if not args.no_families:
            subs["families"] = bench_families(torch, max(args.steps, 100), args.warmup,
                                              HEADLINE_SEAM_W)
            subs["kda"] = bench_kda(torch, max(args.steps, 100), args.warmup)
            subs["adjacent"] = bench_adjacent(torch, max(args.steps, 100))
    value = seg["tokens"] / (seg["ms_per_step"] * 1e-3)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": seg["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded generators; the paper's datasets are not used)",
        "config": seg["config"],
        "roofline": seg["roofline"],
        "cpu_baseline": cpu,
    }
    for key in ("ms_per_step_median", "ms_per_step_graph", "build_ms", "build_ms_mean",
                "compose_us", "seam_us", "compose_roofline", "warmup_s", "warmup_steps"):
        out[key] = seg[key]
    out.update(subs)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
