"""Host-side checks of bench.py: the algorithmic work and bytes its roofline
figures divide by, and its one-GPU contract.  No GPU is touched."""

import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2607_01299_amd import workloads as W  # noqa: E402


def _products_per_chunk(C, d_k, d_v):
    """(m, n, k) of every matrix product of one chunk of the chunked delta
    rule (Sec. 3, Tab. 3 dense operator), state and operator columns."""
    return [
        (C, C, d_k),    # K K^T
        (C, C, d_k),    # Q K^T
        (C, d_k, C),    # W from the inverted unit-lower system
        (C, d_v, C),    # U from the same system
        (C, d_v, C),    # masked (Q K^T) times the corrected values
        (C, d_v, d_k),  # W S0
        (C, d_v, d_k),  # Q S0
        (d_k, d_v, C),  # K^T times the corrected values
        (C, d_k, d_k),  # W P0 (operator columns)
        (d_k, d_k, C),  # K^T X (operator columns)
    ]


def test_build_flops_are_the_chunk_products():
    for C, d_k, d_v in [(64, 128, 128), (64, 64, 128), (32, 128, 64), (16, 64, 64)]:
        per_chunk = sum(2 * m * n * k for m, n, k in _products_per_chunk(C, d_k, d_v))
        assert bench.flop_per_token_head(d_k, d_v, C) * C == per_chunk
    assert bench.flop_per_token_head(128, 128, 64) == 245_760


def test_build_flop_counts_the_gram_once_per_qk_head():
    """The algorithmic count: every v-head's chunk products, the K K^T and Q K^T Gram once
    per q/k head of a grouped-head group.  Equal heads give the per-head count;
    the long-context workload (16 q/k, 32 v heads, 131072 tokens) is 962 GFLOP."""
    assert bench.build_flop(16384, 16, 16, 128, 128, 64) == 16384 * 16 * 245_760
    C, d_k, d_v = 64, 128, 128
    gram = 2 * (2 * C * C * d_k) // C          # K K^T and Q K^T per token of one q/k head
    assert bench.gram_flop_per_token(d_k, C) == gram
    full = bench.flop_per_token_head(d_k, d_v, C)
    assert bench.build_flop(1, 16, 32, d_k, d_v, C) == 32 * (full - gram) + 16 * gram
    assert abs(bench.build_flop(131072, 16, 32, 128, 128, 64) - 962.1e9) < 0.1e9


def test_hbm_roofline_never_exceeds_the_counted_bytes():
    """The reported HBM fraction divides the bytes the counters saw (when a record
    exists) and never the larger algorithmic count of L2-served re-reads."""
    r = bench.hbm_roofline(8e9, 1.0, None, "nothing")        # 8 GB in 1 ms, no record
    assert abs(r["frac"] - 1.0) < 1e-12 and r["traffic"] is None
    assert abs(r["frac_algorithmic"] - 1.0) < 1e-12
    # above the peak with no counter record: no HBM fraction is claimed
    r = bench.hbm_roofline(9e9, 1.0, None, "nothing")
    assert r["frac"] is None and r["achieved"] is None and r["frac_algorithmic"] > 1.0


def test_kda_flop_split_sums_to_the_build_count():
    for C, d_k, d_v in [(64, 128, 128), (64, 64, 128), (64, 128, 64)]:
        state, operator = bench.kda_flops(d_k, d_v, C)
        assert state + operator == bench.flop_per_token_head(d_k, d_v, C)
        # the operator columns: (K . e^B) P0 and K^T N_P (two d_k x d_k
        # products per token) and N_P from the unit-lower solve (C x d_k)
        assert operator == 2 * C * d_k + 4 * d_k * d_k
    assert bench.kda_flops(128, 128, 64) == (163_840, 81_920)


def test_compose_bytes_per_head_step():
    # P_hat_i and S_i read, S_incoming written (float32), log_decay_i read
    d_k, d_v = 128, 128
    assert bench.compose_bytes_per_head_step(d_k, d_v) == 4 * (d_k * d_k + 2 * d_k * d_v) + 4
    assert bench.compose_bytes_per_head_step(d_k, d_v) == 196_612
    assert bench.compose_bytes_per_head_step(d_k, d_v, write_incoming=False) == \
        4 * (d_k * d_k + d_k * d_v) + 4


def test_family_build_bytes_are_the_tensors_one_launch_touches():
    """Sum of the sizes of the arrays a family build reads and writes, on the
    shapes of the layer workload (16 heads, d = 128, 8 x 2048 tokens)."""
    w = W.segment_workload(2)
    T, h_qk, d_k = w["q"].shape
    h_v, d_v = w["v"].shape[1:]
    n_seg = len(w["lengths"])
    bf16 = np.dtype(np.uint16).itemsize
    for family, g in (("scalar", 1), ("diagonal", d_k)):
        reads = (w["q"].size + w["k"].size + w["v"].size) * bf16 + T * h_v * g * 4
        writes = w["v"].size * bf16 + n_seg * h_v * (d_k * d_v + g) * 4
        assert bench.family_build_bytes(family, T, h_qk, h_v, d_k, d_v, n_seg) == reads + writes
    assert bench.family_build_bytes("scalar", T, h_qk, h_v, d_k, d_v, n_seg) == 277_873_152


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def test_traffic_records_hash_every_header_their_kernels_include():
    """A counter record is dropped when its kernel's code changes; the code is
    the kernel file and every local header it reaches through #include."""
    import re
    csrc = os.path.join(ROOT, "paper_2607_01299_amd", "csrc")

    def reach(name, seen):
        if name in seen:
            return seen
        seen.add(name)
        with open(os.path.join(csrc, name)) as f:
            for inc in re.findall(r'#include "([^"]+)"', f.read()):
                reach(inc, seen)
        return seen

    for kernel, files in bench.KERNEL_SOURCES.items():
        assert set(files) == reach(files[0], set()), kernel
