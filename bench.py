#!/usr/bin/env python3
"""Benchmark of the Hypic GDN hot path on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
segment build (o, S_seg, P_hat, log_decay for every segment and head), Eq. (6)
composition of the batch's segments in order (emitting the state entering
each segment) and the seam rescan of every segment's first w tokens from that
state.  ms_per_step_graph reports the same step replayed as one HIP graph.  Default workload: 16 heads, d_k = d_v = 128, 8 independent segments of
2048 bf16 tokens, chunk 64, seam w = 8.  value = tokens / s over the timed
steps, inputs resident in HBM.

Also reported:
  roofline      the build scan kernel: algorithmic FLOP per launch over its
                average duration (HIP events on the launch stream around
                back-to-back builds after the timed steps; build_ms_in_step is
                the same call bracketed inside each step) vs the dense bf16
                matrix-core peak;
  compose_burst serve-time burst: 256 requests x U{8..64} segments of a
                512-entry float32 pool (16 heads, 128 x 128), then a w = 64
                seam per listed segment; compositions / s and the composition
                kernel's algorithmic HBM bandwidth;
  cpu_baseline  the float64 oracle on the host cores on a bounded sample.

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

# Algorithmic work of the chunked scan per (token, v-head) at chunk C:
#   2C(3 d_k + 2 d_v)   K K^T, Q K^T, W, U, (Q K^T . Gamma) Vn
#   6 d_k d_v           W' S0, Q S0, K^T Vn
#   4 d_k^2             W P0, K^T X (operator path)
def flop_per_token_head(d_k, d_v, chunk):
    return 2 * chunk * (3 * d_k + 2 * d_v) + 6 * d_k * d_v + 4 * d_k * d_k


CSRC = os.path.join(HERE, "paper_2607_01299_amd", "csrc")
TRAFFIC_FILE = os.path.join(HERE, "profiles", "hbm_traffic.json")
KERNEL_SOURCES = {
    "scan_bf16": ["scan_bf16.hip", "mfma.hpp", "scan.hpp"],
    "compose": ["compose.hip", "mfma.hpp", "scan.hpp"],
    "family_scalar_build": ["family.hip", "mfma.hpp", "family.hpp", "scan.hpp", "frag_common.hpp"],
    "family_diagonal_build": ["family.hip", "mfma.hpp", "family.hpp", "scan.hpp", "frag_common.hpp"],
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
    """Hash of a kernel's code (comments and layout ignored), so the HBM counter
    record stays valid across comment-only edits and lapses on any code change."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(CSRC, name), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    passes (scaled by a plain copy of known size), or None when the kernel's
    sources changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("workload") != workload:
        return None
    if rec.get("src_sha256") != kernel_source_sha256(kernel):
        return None
    return float(rec["fetch_bytes_per_launch"]) + float(rec["write_bytes_per_launch"])


MFMA_FILE = os.path.join(HERE, "profiles", "mfma_counters.json")


def measured_mfma(kernel, workload):
    """Matrix-core counters of a kernel from the committed rocprofv3 passes
    (MfmaUtil: MFMA-busy cycles over active cycles x SIMDs; bf16 MFMA ops x 512),
    or None when the kernel's sources changed since they were taken."""
    try:
        with open(MFMA_FILE) as f:
            rec = json.load(f).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("workload") != workload:
        return None
    if rec.get("src_sha256") != kernel_source_sha256(kernel):
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
    # read P_hat_i and S_i, write the incoming state, read log_decay_i
    return 4 * (d_k * d_k + d_k * d_v * (2 if write_incoming else 1)) + 4


# ---------------------------------------------------------------------------
# CPU baseline: the oracle, run before the GPU is touched
# ---------------------------------------------------------------------------

def _oracle_pair(args):
    cfg, seg, head = args
    import oracle
    w = _CACHE.get(cfg)
    lo, hi = int(w["cu_seqlens"][seg]), int(w["cu_seqlens"][seg + 1])
    sl = slice(lo, hi)
    oracle.build_segments(w["q"][sl], w["k"][sl], w["v"][sl], w["beta"][sl],
                          w["log_alpha"][sl], [0, hi - lo], seg_head_pairs=[(0, head)])
    return hi - lo


_CACHE = {}


def _worker_init(cfg):
    _CACHE[cfg] = W.segment_workload(cfg)


def cpu_baseline(cfg, h_v, pairs_per_worker=100):
    import multiprocessing as mp
    workers = min(len(os.sched_getaffinity(0)), 16)
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = "1"
    wl = W.segment_workload(cfg)
    n_seg = len(wl["cu_seqlens"]) - 1
    distinct = [(cfg, s, h) for h in range(h_v) for s in range(n_seg)]
    # 10-20 s of wall time on 16 cores: the distinct pairs, cycled
    pairs = [distinct[i % len(distinct)] for i in range(workers * pairs_per_worker)]
    ctx = mp.get_context("spawn")
    with ctx.Pool(workers, initializer=_worker_init, initargs=(cfg,)) as pool:
        pool.map(_oracle_pair, pairs[:workers])           # warm the workers
        t0 = time.perf_counter()
        toks = pool.map(_oracle_pair, pairs)
        dt = time.perf_counter() - t0
    token_heads = float(sum(toks))
    return {
        "value": token_heads / dt / h_v,
        "unit": "tokens/s",
        "cores": workers,
        "kind": "oracle",
        "sample": "%d (segment, head) builds of %d tokens (S and operator, float64 token "
                  "recurrence; the workload's %d distinct pairs, cycled) on %d processes, "
                  "%.1f s; tokens/s = token-heads/s / %d heads"
                  % (len(pairs), int(toks[0]), len(distinct), workers, dt, h_v),
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


def bench_segments(torch, cfg, steps, warmup, seam_w):
    from paper_2607_01299_amd.pipeline import SegmentPipeline
    w = W.segment_workload(cfg)
    q, k, v, beta, la = _to_dev(w, torch)
    pipe = SegmentPipeline(q, k, v, beta, la, w["cu_seqlens"], chunk=w["chunk"], seam_w=seam_w)
    for _ in range(warmup):
        pipe.run()
    torch.cuda.synchronize()
    stream = pipe.stream
    # eager steps, with the build bracketed by events inside each step
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(stream)
        pipe.build()
        ev[i][1].record(stream)
        pipe.compose()
        pipe.seam()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    build_in_step_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    # the same step replayed as one HIP graph, for reference (the launches of
    # an eager step already queue back to back, so the graph does not shorten it)
    pipe.capture()
    for _ in range(max(warmup, 1)):
        pipe.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        pipe.replay()
    torch.cuda.synchronize()
    dt_graph = time.perf_counter() - t0
    # the build kernel's average launch duration: `steps` launches back to back
    # between one pair of events on the launch stream (amortises the markers)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        pipe.build()
    e1.record(stream)
    torch.cuda.synchronize()
    build_ms = e0.elapsed_time(e1) / steps
    T = int(w["cu_seqlens"][-1])
    h_v, d_k, d_v = w["v"].shape[1], w["d_k"], w["d_v"]
    flop = float(flop_per_token_head(d_k, d_v, w["chunk"])) * T * h_v
    achieved = flop / (build_ms * 1e-3) / 1e12
    return {
        "ms_per_step": dt / steps * 1e3,
        "ms_per_step_graph": dt_graph / steps * 1e3,
        "tokens": T,
        "build_ms": build_ms,
        "build_ms_in_step": build_in_step_ms,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": measured_traffic("scan_bf16", W.CONFIG_NAMES[cfg]),
                     "counter": measured_mfma("scan_bf16", W.CONFIG_NAMES[cfg]),
                     "kernel": "scan_bf16_kernel (segment build)",
                     "flop_per_launch": flop},
        "config": {"workload": W.CONFIG_NAMES[cfg], "segments": len(w["lengths"]),
                   "tokens": T, "h_qk": int(w["q"].shape[1]), "h_v": int(h_v), "d_k": d_k,
                   "d_v": d_v, "chunk": w["chunk"], "seam_w": seam_w, "seed": w["seed"]},
    }


def bench_compose_burst(torch, steps, warmup):
    from paper_2607_01299_amd.pipeline import ComposeBurst
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
    for _ in range(warmup):
        burst.run()
    torch.cuda.synchronize()
    stream = burst.stream
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        ev[i][0].record(stream)
        burst.compose()
        ev[i][1].record(stream)
        burst.seam()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    comp_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    nnz, h_v = burst.nnz, burst.h_v
    byts = float(compose_bytes_per_head_step(burst.d_k, burst.d_v)) * nnz * h_v
    gbs = byts / (comp_ms * 1e-3) / 1e9
    # the same requests with seams that advance the state (Sec. 4.3): the pool
    # tuples read as tail tuples, each entry's 64 tokens as its seam
    from paper_2607_01299_amd.pipeline import SeamAdvanceBurst
    adv = SeamAdvanceBurst(P, g, S, p["seg_ids"], p["req_offsets"], toks, p["tok_start_pool"],
                           p["seam_len_pool"], p["w"])
    adv.run()
    adv1_ms = _events_ms(torch, adv.stream, adv.run, max(steps // 2, 2))
    del adv
    # the same burst over two lanes (half the requests each, on two streams), so
    # that one lane's seam steps overlap the other's compositions
    adv = SeamAdvanceBurst(P, g, S, p["seg_ids"], p["req_offsets"], toks, p["tok_start_pool"],
                           p["seam_len_pool"], p["w"], lanes=2)
    adv.run()
    adv_ms = _events_ms(torch, adv.stream, adv.run, max(steps // 2, 2))
    del adv
    return {
        "compositions_per_s": nnz / (dt / steps),
        "requests_per_s": burst.n_req / (dt / steps),
        "ms_per_burst": dt / steps * 1e3,
        "compose_ms": comp_ms,
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": gbs / PEAK_HBM_GBS,
                     "traffic": measured_traffic("compose", W.CONFIG_NAMES[5]),
                     "counter": measured_mfma("compose", W.CONFIG_NAMES[5]),
                     "kernel": "compose_kernel", "bytes_per_launch": byts},
        "seam_advance": {"ms_per_burst": adv_ms, "compositions_per_s": nnz / (adv_ms * 1e-3),
                         "lanes": 2, "ms_per_burst_one_call": adv1_ms,
                         "note": "seams run from the running state, then tail tuples (Sec. 4.3)"},
        "config": {"workload": W.CONFIG_NAMES[5], "requests": burst.n_req,
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


def _events_ms(torch, stream, fn, reps):
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def bench_families(torch, steps, warmup, seam_w):
    """Scalar and diagonal families (Tab. 1) on the bench workload: the whole
    family step (build, composition of the batch in order, seams) and the
    build kernel's HBM roofline; then a serve-time burst over a pool of family
    tuples with the configuration-5 request lists."""
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
        for _ in range(warmup):
            pipe.run()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            pipe.run()
        torch.cuda.synchronize()
        dt = (time.perf_counter() - t0) / steps
        build_ms = _events_ms(torch, pipe.stream, pipe.build, steps)
        byts = float(family_build_bytes(family, T, h_qk, h_v, d_k, d_v, n_seg))
        gbs = byts / (build_ms * 1e-3) / 1e9
        # pool of family tuples: the configuration-5 states, per-channel or
        # scalar log-decays ~ U(-3, 0)
        rng = np.random.default_rng(p["seed"] + 7)
        ld_shape = (p["n_pool"], h_v) if family == "scalar" else (p["n_pool"], h_v, d_k)
        ld = torch.from_numpy(rng.uniform(-3.0, 0.0, size=ld_shape).astype(np.float32)).cuda()
        burst = FamilyComposeBurst(family, ld, S_pool, p["seg_ids"], p["req_offsets"])
        burst.compose()
        comp_ms = _events_ms(torch, burst.stream, burst.compose, max(steps // 2, 3))
        cbytes = float(family_compose_bytes_per_head_step(family, d_k, d_v)) * burst.nnz * h_v
        cgbs = cbytes / (comp_ms * 1e-3) / 1e9
        out[family] = {
            "tokens_per_s": T / dt,
            "ms_per_step": dt * 1e3,
            "build_ms": build_ms,
            "roofline": {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": gbs / PEAK_HBM_GBS,
                         "traffic": measured_traffic("family_%s_build" % family, FAMILY_WORKLOAD),
                         "kernel": ("family_pipe_kernel (build)" if family == "scalar"
                                    else "family_scan_kernel (build)"),
                         "bytes_per_launch": byts},
            "compose_burst": {"compositions_per_s": burst.nnz / (comp_ms * 1e-3),
                              "compose_ms": comp_ms,
                              "roofline": {"bound": "hbm", "achieved": cgbs,
                                           "peak": PEAK_HBM_GBS, "unit": "GB/s",
                                           "frac": cgbs / PEAK_HBM_GBS,
                                           "traffic": measured_traffic(
                                               "family_%s_compose" % family,
                                               FAMILY_BURST_WORKLOAD),
                                           "kernel": "family_compose_kernel",
                                           "bytes_per_launch": cbytes}},
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
    """KDA row of Tab. 1 on the bench workload (16 heads, d = 128, 8 x 2048 bf16
    tokens, per-channel gates from the diagonal-family generator): the build with
    its operator, timed with HIP events over back-to-back launches.  Every
    product runs on the bf16 matrix cores (the operator columns as three split
    passes), so the roofline peak is the bf16 one, as for the GDN build."""
    from paper_2607_01299_amd.pipeline import KdaPipeline
    w = W.segment_workload(2)
    q, k, v, beta, _ = _to_dev(w, torch)
    T = int(w["cu_seqlens"][-1])
    h_v, d_k, d_v = int(w["v"].shape[1]), w["d_k"], w["d_v"]
    gate = torch.from_numpy(W.family_gate("diagonal", T, h_v, d_k, w["seed"] + 2000)).cuda()
    pipe = KdaPipeline(q, k, v, beta, gate, w["cu_seqlens"])
    for _ in range(warmup):
        pipe.build()
    torch.cuda.synchronize()
    ms = _events_ms(torch, pipe.stream, pipe.build, steps)
    f_state, f_op = kda_flops(d_k, d_v, 64)
    flop = float(f_state + f_op) * T * h_v
    achieved = flop / (ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS
    return {"workload": KDA_WORKLOAD,
            "tokens_per_s": T / (ms * 1e-3), "build_ms": ms,
            "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                         "frac": achieved / peak,
                         # both launches of one build
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
        gbs = byts / (ms * 1e-3) / 1e9
        out[name] = {"ms": ms, "workload": workload,
                     "roofline": {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS,
                                  "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS, "traffic": None,
                                  "bytes_per_launch": byts}}

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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # 200 timed steps after 50 warm-up steps: about 50 ms of GPU work, enough
    # for the clocks to settle (5 + 20 steps read the build about 15 % slower)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--config", type=int, default=2, choices=[2, 3, 4])
    ap.add_argument("--seam-w", type=int, default=8)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-burst", action="store_true")
    ap.add_argument("--no-families", action="store_true",
                    help="skip the scalar / diagonal family and reuse-time-step legs")
    ap.add_argument("--families-only", action="store_true",
                    help="run only the family and reuse-time-step legs (profiling)")
    ap.add_argument("--no-segments", action="store_true",
                    help="skip the segment step (profiling the burst alone)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain 1 GiB device copy (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(segments shard across GPUs with no exchange; see the design notes). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        import torch
        copy_calibration(torch)
        return
    cpu = None
    if not args.no_cpu_baseline and not args.no_segments and not args.families_only:
        wl = W.segment_workload(args.config)
        cpu = cpu_baseline(args.config, int(wl["v"].shape[1]))
        print("[bench] cpu baseline done: %.1f tokens/s" % cpu["value"], file=sys.stderr,
              flush=True)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_2607_01299_amd import _lib
    _lib.load()
    # Python's cyclic collector stays off in the GPU legs, as timeit keeps it
    # off: a full collection of the interpreter's objects stalls the host for
    # 40-60 ms, and one such pause inside a timed loop of short launches lets
    # the queue drain (the conv leg read 0.297 ms per call for an 88 us kernel)
    gc.collect()
    gc.freeze()
    gc.disable()
    if args.families_only:
        print(json.dumps({"families": bench_families(torch, args.steps, args.warmup,
                                                     args.seam_w),
                          "kda": bench_kda(torch, args.steps, args.warmup),
                          "adjacent": bench_adjacent(torch, args.steps)}))
        return
    if args.no_segments:
        burst = bench_compose_burst(torch, max(args.steps // 2, 3), max(args.warmup // 2, 1))
        print(json.dumps({"compose_burst": burst}))
        return

    seg = bench_segments(torch, args.config, args.steps, args.warmup, args.seam_w)
    print("[bench] segment step done: %.3f ms/step" % seg["ms_per_step"], file=sys.stderr,
          flush=True)
    burst = None if args.no_burst else bench_compose_burst(torch, max(args.steps // 2, 3),
                                                           max(args.warmup // 2, 1))
    fam = None if args.no_families else bench_families(torch, args.steps, args.warmup,
                                                         args.seam_w)
    kda = None if args.no_families else bench_kda(torch, args.steps, args.warmup)
    adj = None if args.no_families else bench_adjacent(torch, args.steps)
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
        "ms_per_step_graph": seg["ms_per_step_graph"],
        "build_ms": seg["build_ms"],
        "build_ms_in_step": seg["build_ms_in_step"],
        "cpu_baseline": cpu,
        "compose_burst": burst,
        "families": fam,
        "kda": kda,
        "adjacent": adj,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
