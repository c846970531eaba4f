"""Seeded synthetic inputs for the segment build, composition and seam rescan.

This module only draws random numbers and lays them out.  It performs none of
the method's arithmetic (no recurrence, no operator, no composition) and is
shared by the tests, the bench and the smoke check so that the HIP path and the
float64 oracle see bit-identical inputs.

The paper's datasets (HotpotQA, TriviaQA, MultiNews, GovReport, a production
RAG trace) are not available; these inputs stand in for them with the shapes
the paper describes for its RAG / agentic prompts: segments longer than 512
tokens (Sec. 4.3), 1k-token cached segments (Sec. 6.3), d_k = d_v = 128 dense
GDN heads (Tab. 3).

Distributions (per token and head, drawn in this order: q, k, v, beta-logits,
gate-logits):

* q, k ~ N(0, 1), then L2-normalised per (token, head);
* v ~ N(0, 1);
* beta = sigmoid(N(0, 1));
* a = log(alpha) = -0.05 * softplus(N(0, 1)); the long-context configuration
  instead draws alpha ~ U(0.9, 1) and takes a = log(alpha).

Values are generated in float32; where the configuration is bf16, q, k and v are
rounded once to bf16 with round-to-nearest-even and kept in float32 arrays
(every value is exactly representable in bf16).  beta and a stay float32.
"""

import numpy as np

SEED_BASE = 260701299

F32 = "f32"
BF16 = "bf16"


def round_bf16(x):
    """Round float32 values to the nearest bf16 (ties to even), returned as
    float32 arrays holding exactly representable bf16 values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    r = ((u + bias) & np.uint32(0xFFFF0000)).astype(np.uint32)
    return r.view(np.float32)


def _l2_normalise(x):
    n = np.sqrt(np.sum(x.astype(np.float64) ** 2, axis=-1, keepdims=True))
    return (x / np.maximum(n, 1e-30)).astype(np.float32)


def _softplus(x):
    x = x.astype(np.float64)
    return np.log1p(np.exp(-np.abs(x))) + np.maximum(x, 0.0)


def draw_tokens(rng, T, h_qk, h_v, d_k, d_v, dtype, gate="softplus"):
    """Draw one packed token batch.  Returns dict of float32 arrays
    q, k [T, h_qk, d_k]; v [T, h_v, d_v]; beta, log_alpha [T, h_v]."""
    q = _l2_normalise(rng.standard_normal((T, h_qk, d_k), dtype=np.float32))
    k = _l2_normalise(rng.standard_normal((T, h_qk, d_k), dtype=np.float32))
    v = rng.standard_normal((T, h_v, d_v), dtype=np.float32)
    bl = rng.standard_normal((T, h_v), dtype=np.float32).astype(np.float64)
    beta = (1.0 / (1.0 + np.exp(-bl))).astype(np.float32)
    if gate == "softplus":
        gl = rng.standard_normal((T, h_v), dtype=np.float32)
        log_alpha = (-0.05 * _softplus(gl)).astype(np.float32)
    elif gate == "uniform_0.9_1":
        alpha = rng.uniform(0.9, 1.0, size=(T, h_v)).astype(np.float32)
        log_alpha = np.log(alpha.astype(np.float64)).astype(np.float32)
    elif gate == "slow":
        # slowest RetNet head of Tab. 2: alpha = 1 - 2^-10 for every token
        log_alpha = np.full((T, h_v), np.log1p(-2.0 ** -10), dtype=np.float32)
    else:
        raise ValueError(gate)
    if dtype == BF16:
        q, k, v = round_bf16(q), round_bf16(k), round_bf16(v)
    return {"q": q, "k": k, "v": v, "beta": beta, "log_alpha": log_alpha}


def cu_from_lengths(lengths):
    cu = np.zeros(len(lengths) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(np.asarray(lengths, dtype=np.int64))
    return cu


def log_uniform_lengths(rng, n, lo=128, hi=16384):
    """Segment lengths round(exp(U(ln lo, ln hi))) (agentic mixed lengths)."""
    return np.rint(np.exp(rng.uniform(np.log(lo), np.log(hi), size=n))).astype(np.int64)


# --------------------------------------------------------------------------
# The five workloads.  ``scale`` shrinks a workload for tests that must finish
# quickly on the CPU oracle while keeping its structure.
# --------------------------------------------------------------------------

CONFIG_NAMES = {
    1: "tiny-fp32: 1 head, d=64, 4x256 tokens, chunk 64",
    2: "layer-bf16: 16 heads, d=128, 8x2048 tokens, chunk 64",
    3: "rag-long: 32x4096 tokens, 16 qk / 32 v heads, d=128, bf16, alpha~U(0.9,1)",
    4: "agentic-ragged: 64 segments log-uniform[128,16384], 16 heads, d=128, bf16, seam w=32",
    5: "serve-burst: 256 requests x U{8..64} of a 512-entry fp32 pool, 16 heads, d=128, seam w=64",
}


def segment_workload(cfg, seed=None, n_seg=None, seg_len=None, heads=None,
                     d=None, lengths=None, gate=None, dtype=None):
    """Build-side workload of configurations 1-4 (overrides shrink it).

    Returns dict with the token arrays, cu_seqlens (int32), dims and, for
    configuration 3, the 1024 prefix tokens (key ``prefix``) and for
    configuration 4 the seam width.
    """
    if seed is None:
        seed = SEED_BASE + cfg
    rng = np.random.default_rng(seed)
    if cfg == 1:
        h_qk, h_v, dd, dt, g, lens = 1, 1, 64, F32, "softplus", [256] * 4
    elif cfg == 2:
        h_qk, h_v, dd, dt, g, lens = 16, 16, 128, BF16, "softplus", [2048] * 8
    elif cfg == 3:
        h_qk, h_v, dd, dt, g, lens = 16, 32, 128, BF16, "uniform_0.9_1", [4096] * 32
    elif cfg == 4:
        h_qk, h_v, dd, dt, g = 16, 16, 128, BF16, "softplus"
        lens = None  # drawn below, before any token
    else:
        raise ValueError("segment workloads are configurations 1-4")
    if heads is not None:
        h_qk, h_v = heads
    if d is not None:
        dd = d
    if gate is not None:
        g = gate
    if dtype is not None:
        dt = dtype
    if cfg == 4 and lengths is None:
        lens = list(log_uniform_lengths(rng, 64 if n_seg is None else n_seg))
        n_seg = None
    if lengths is not None:
        lens = list(lengths)
    else:
        if n_seg is not None:
            lens = [lens[0]] * n_seg
        if seg_len is not None:
            lens = [seg_len] * len(lens)
    cu = cu_from_lengths(lens)
    T = int(cu[-1])
    out = draw_tokens(rng, T, h_qk, h_v, dd, dd, dt, gate=g)
    out.update({"cu_seqlens": cu, "lengths": np.asarray(lens, dtype=np.int64),
                "h_qk": h_qk, "h_v": h_v, "d_k": dd, "d_v": dd, "dtype": dt,
                "chunk": 64, "cfg": cfg, "seed": seed})
    if cfg == 3:
        out["prefix"] = draw_tokens(rng, 1024, h_qk, h_v, dd, dd, dt, gate=g)
    if cfg == 4:
        out["w"] = 32
    return out


def pool_workload(seed=None, n_pool=512, n_req=256, n_min=8, n_max=64,
                  heads=16, d=128, seam_tokens=64, w=64):
    """Configuration 5: a pool of cached tuples and a burst of requests.

    The pool tuples are synthetic (the composition is exact algebra for any
    tuple): P_hat has i.i.d. N(0, (0.5)^2 / d) entries (spectral norm about 1),
    log_decay ~ U(-3, 0) (slow enough that earlier segments stay visible in the
    composed state), S ~ N(0, 0.25^2).  Each pool entry also owns
    ``seam_tokens`` bf16 tokens (configuration-2 distributions) for its seam.
    Requests: n_r ~ U{n_min..n_max} pool ids drawn without replacement, in
    random order; zero prefix.
    """
    if seed is None:
        seed = SEED_BASE + 5
    rng = np.random.default_rng(seed)
    P_hat = (rng.standard_normal((n_pool, heads, d, d), dtype=np.float32)
             * np.float32(0.5 / np.sqrt(d)))
    log_decay = rng.uniform(-3.0, 0.0, size=(n_pool, heads)).astype(np.float32)
    S_seg = rng.standard_normal((n_pool, heads, d, d), dtype=np.float32) * np.float32(0.25)
    n_r = rng.integers(n_min, n_max + 1, size=n_req)
    ids = [rng.choice(n_pool, size=int(n), replace=False) for n in n_r]
    seg_ids = np.concatenate(ids).astype(np.int32)
    req_offsets = cu_from_lengths(n_r)
    toks = draw_tokens(rng, n_pool * seam_tokens, heads, heads, d, d, BF16)
    # seam entry j (the j-th listed segment overall) reads the tokens owned by
    # pool entry seg_ids[j]
    tok_start = (seg_ids.astype(np.int64) * seam_tokens).astype(np.int32)
    tok_len = np.full(len(seg_ids), seam_tokens, dtype=np.int32)
    return {"P_hat": P_hat, "log_decay": log_decay, "S_seg": S_seg,
            "seg_ids": seg_ids, "req_offsets": req_offsets, "tokens": toks,
            "tok_start": tok_start, "tok_len": tok_len, "w": w,
            "tok_start_pool": (np.arange(n_pool) * seam_tokens).astype(np.int32),
            "seam_len_pool": np.full(n_pool, seam_tokens, dtype=np.int32),
            "h_qk": heads, "h_v": heads, "d_k": d, "d_v": d, "dtype": BF16,
            "chunk": 64, "cfg": 5, "seed": seed, "n_pool": n_pool}


# --------------------------------------------------------------------------
# gates of the scalar and diagonal transition families (Tab. 1)
# --------------------------------------------------------------------------

def family_gate(family, T, h_v, d_k, seed, kind="softplus"):
    """Log-gates of the scalar ([T, h_v]) or diagonal ([T, h_v, d_k]) family,
    float32, natural-log units, drawn from their own seeded stream.

    kind: "softplus"   a = -0.05 softplus(N(0, 1)) (the GDN gate distribution,
                       per channel for the diagonal family);
          "logsigmoid" a = log sigmoid(N(0, 1)) (un-normalised GLA-style gates,
                       strong decay: mean about -0.8 per token);
          "retnet"     scalar only: RetNet's fixed per-head decays
                       gamma_h = 1 - 2^(-5 - h), for every token.
    """
    rng = np.random.default_rng(seed)
    shape = (T, h_v) if family == "scalar" else (T, h_v, d_k)
    if kind == "retnet":
        if family != "scalar":
            raise ValueError("retnet gates are scalar")
        gam = 1.0 - 2.0 ** (-5.0 - np.arange(h_v, dtype=np.float64))
        return np.broadcast_to(np.log(gam).astype(np.float32), shape).copy()
    x = rng.standard_normal(shape, dtype=np.float32)
    if kind == "softplus":
        return (-0.05 * _softplus(x)).astype(np.float32)
    if kind == "logsigmoid":
        return (-_softplus(-x)).astype(np.float32)
    raise ValueError(kind)
