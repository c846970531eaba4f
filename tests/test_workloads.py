"""Seeded input generators: determinism, bf16 rounding, shapes.  CPU only."""

import hashlib

import numpy as np
import torch

from paper_2607_01299_amd import workloads as W


def _digest(d):
    h = hashlib.sha256()
    for key in sorted(d):
        val = d[key]
        if isinstance(val, np.ndarray):
            h.update(key.encode())
            h.update(np.ascontiguousarray(val).tobytes())
    return h.hexdigest()


def test_seeded_generation_is_deterministic():
    a = W.segment_workload(2, n_seg=2, seg_len=100, heads=(2, 2))
    b = W.segment_workload(2, n_seg=2, seg_len=100, heads=(2, 2))
    c = W.segment_workload(2, n_seg=2, seg_len=100, heads=(2, 2), seed=W.SEED_BASE + 99)
    assert _digest(a) == _digest(b)
    assert _digest(a) != _digest(c)


def test_bf16_rounding_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(100000, dtype=np.float32) * np.float32(3.7)
    # include exact ties: low 16 bits == 0x8000
    ties = (rng.integers(0, 2 ** 31, size=1000, dtype=np.uint32) & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    x = np.concatenate([x, ties.view(np.float32)[np.isfinite(ties.view(np.float32))]])
    ours = W.round_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours, ref)
    assert np.array_equal(W.round_bf16(ours), ours)


def test_config_shapes_and_distributions():
    w1 = W.segment_workload(1)
    assert w1["q"].shape == (1024, 1, 64) and w1["v"].shape == (1024, 1, 64)
    assert list(w1["cu_seqlens"]) == [0, 256, 512, 768, 1024]
    assert w1["dtype"] == W.F32
    n = np.linalg.norm(w1["k"].astype(np.float64), axis=-1)
    assert np.allclose(n, 1.0, atol=1e-6)
    assert np.all((w1["beta"] > 0) & (w1["beta"] < 1))
    assert np.all(w1["log_alpha"] < 0)
    w3 = W.segment_workload(3, n_seg=2, seg_len=64)
    assert w3["q"].shape[1] == 16 and w3["v"].shape[1] == 32
    assert w3["prefix"]["q"].shape == (1024, 16, 128)
    alpha = np.exp(w3["log_alpha"].astype(np.float64))
    assert alpha.min() >= 0.9 - 1e-6 and alpha.max() <= 1.0
    assert np.array_equal(W.round_bf16(w3["q"]), w3["q"])
    w4 = W.segment_workload(4, heads=(1, 1), d=16)
    lens = w4["lengths"]
    assert len(lens) == 64 and lens.min() >= 128 and lens.max() <= 16384
    assert w4["cu_seqlens"][-1] == lens.sum()


def test_pool_workload_structure():
    p = W.pool_workload(n_pool=40, n_req=10, n_min=8, n_max=20, heads=2, d=16,
                        seam_tokens=8, w=8)
    offs = p["req_offsets"]
    assert offs[0] == 0 and len(offs) == 11
    n_r = np.diff(offs)
    assert n_r.min() >= 8 and n_r.max() <= 20
    for r in range(10):
        ids = p["seg_ids"][offs[r]:offs[r + 1]]
        assert len(set(ids.tolist())) == len(ids)          # without replacement
        assert ids.min() >= 0 and ids.max() < 40
    assert np.array_equal(p["tok_start"], p["seg_ids"] * 8)
