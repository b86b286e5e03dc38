"""Seeded synthetic inputs shaped like the paper's inference collectives.

This module only draws inputs.  It holds none of the datapath's arithmetic
(no reduction, no packing, no combine): the oracle and the HIP path both
receive what it returns.  bf16 inputs are produced by drawing binary32
values with numpy and converting them with torch's CPU ``bfloat16`` cast,
a library routine used here only to make input data.

Every array comes from ``numpy.random.Generator(PCG64)`` seeded by a
``SeedSequence``; per-rank buffers use ``SeedSequence(seed).spawn(P)[p]``
so that each rank's data is independent of how the work is chunked.

The paper measures with real models and serving traces that are not
available here (Section 5, "Application Performance"); these shapes stand in
for them:

=======================  ===================================================
name                     workload
=======================  ===================================================
AR_P4_FP32_256K          AllReduce, P=4, fp32, 262144 elements per rank,
                         U(-1, 1), chunk 16 KiB
AR_P8_BF16_DECODE        decode AllReduce, P=8, bf16 activations
                         [128 x 8192] per rank, N(0,1), chunk 64 KiB
RS_AG_P8_BF16_256MIB     ReduceScatter then AllGather (and AllReduce as the
                         check), P=8, bf16, 134217728 elements (256 MiB) per
                         rank, N(0, 0.02), chunk 1 MiB
MOE_CONFIG (dispatch)    x bf16 [4096 x 7168] N(0,1); E=256 experts over P=8
                         ranks; top-8 ids per token from Zipf(s=1.1) without
                         repeats
MOE_CONFIG (combine)     expert outputs bf16 [32768 x 7168] N(0,1) in the
                         dispatch's packed layout; softmax top-8 gate weights
                         in fp32
=======================  ===================================================
"""

from dataclasses import dataclass

import numpy as np

__all__ = [
    "CollectiveConfig",
    "MoEConfig",
    "AR_P4_FP32_256K",
    "AR_P8_BF16_DECODE",
    "RS_AG_P8_BF16_256MIB",
    "COLLECTIVE_CONFIGS",
    "MOE_CONFIG",
    "rank_rngs",
    "uniform_f32",
    "normal_bf16",
    "collective_inputs",
    "zipf_topk_ids",
    "softmax_gates",
    "moe_tokens",
    "moe_expert_outputs",
]


@dataclass(frozen=True)
class CollectiveConfig:
    name: str
    op: str  # "allreduce" | "reduce_scatter" | "allgather" | "alltoall"
    P: int
    count: int  # per-rank elements on the scattered side
    dtype: str  # "fp32" | "bf16"
    chunk: int  # bytes
    dist: str  # "uniform" | "normal"
    scale: float
    seed: int


@dataclass(frozen=True)
class MoEConfig:
    T: int
    H: int
    E: int
    P: int
    K: int
    zipf_s: float
    seed_ids: int
    seed_x: int
    seed_y: int
    seed_gates: int


# AllReduce, P = 4, fp32, 262144 elements per rank, uniform in [-1, 1]
AR_P4_FP32_256K = CollectiveConfig("ar_p4_fp32_256k", "allreduce", 4, 262144, "fp32", 16 * 1024, "uniform", 1.0, 1)
# decode-step AllReduce, P = 8, bf16 activations [128 tokens x 8192 hidden] per rank, N(0, 1)
AR_P8_BF16_DECODE = CollectiveConfig("ar_p8_bf16_128x8192", "allreduce", 8, 128 * 8192, "bf16", 64 * 1024, "normal",
                                     1.0, 2)
# prefill-size ReduceScatter then AllGather, P = 8, bf16, 256 MiB per rank, N(0, 0.02)
RS_AG_P8_BF16_256MIB = CollectiveConfig("rs_ag_p8_bf16_256MiB", "reduce_scatter", 8, 134217728, "bf16", 1 << 20,
                                        "normal", 0.02, 3)
COLLECTIVE_CONFIGS = {c.name: c for c in (AR_P4_FP32_256K, AR_P8_BF16_DECODE, RS_AG_P8_BF16_256MIB)}

MOE_CONFIG = MoEConfig(T=4096, H=7168, E=256, P=8, K=8, zipf_s=1.1, seed_ids=4, seed_x=40, seed_y=50, seed_gates=5)


def rank_rngs(seed, P):
    """One independent PCG64 generator per rank: SeedSequence(seed).spawn(P)[p]."""
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(P)]


def uniform_f32(rng, n, lo=-1.0, hi=1.0):
    """U(lo, hi) drawn in float64 and cast to float32."""
    return rng.uniform(lo, hi, n).astype(np.float32)


def _f32_to_bf16_bits(a):
    import torch  # input preparation only

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def normal_bf16(rng, n, scale=1.0, block=1 << 24):
    """N(0, scale) drawn as float32, converted to bf16 encodings (uint16)."""
    out = np.empty(n, dtype=np.uint16)
    for i in range(0, n, block):
        m = min(block, n - i)
        z = rng.standard_normal(m, dtype=np.float32)
        if scale != 1.0:
            z *= np.float32(scale)
        out[i:i + m] = _f32_to_bf16_bits(z)
    return out


def collective_inputs(cfg, count=None, seed=None):
    """Per-rank scattered-side inputs (list of P arrays of ``count`` elements).

    fp32 configs return float32 arrays; bf16 configs return uint16 encodings.
    ``count``/``seed`` override the config's (used by reduced-size tests).
    """
    n = cfg.count if count is None else count
    rngs = rank_rngs(cfg.seed if seed is None else seed, cfg.P)
    if cfg.dist == "uniform":
        data = [uniform_f32(r, n) for r in rngs]
        if cfg.dtype == "bf16":
            data = [_f32_to_bf16_bits(d) for d in data]
        return data
    if cfg.dtype == "fp32":
        return [(r.standard_normal(n, dtype=np.float32) * np.float32(cfg.scale)).astype(np.float32) for r in rngs]
    return [normal_bf16(r, n, cfg.scale) for r in rngs]


def zipf_topk_ids(T, E, K, s, seed):
    """Top-K expert ids per token, Zipf(s) over experts, no repeats in a token.

    Expert ``e`` has weight ``(e+1)**-s`` (popularity rank = expert id).
    Sampling K distinct experts proportionally to these weights, without
    replacement, is done with Gumbel-top-K: key = s*(-ln(e+1)) + Gumbel
    noise ``-ln(-ln U)``, U ~ U[0, 1); the K largest keys win, slot order is
    descending key, ties go to the lower id.  Returns int32 [T, K].
    """
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    U = rng.random((T, E))
    with np.errstate(divide="ignore"):
        gumbel = -np.log(-np.log(U))
    key = -s * np.log(np.arange(1, E + 1, dtype=np.float64))[None, :] + gumbel
    order = np.argsort(-key, axis=1, kind="stable")  # stable: equal keys keep the lower id first
    return order[:, :K].astype(np.int32)


def softmax_gates(T, K, seed):
    """Gate weights [T, K]: N(0,1) float32 logits, softmax in float64, cast to float32."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    logits = rng.standard_normal((T, K), dtype=np.float32).astype(np.float64)
    z = np.exp(logits - logits.max(axis=1, keepdims=True))
    return (z / z.sum(axis=1, keepdims=True)).astype(np.float32)


def moe_tokens(cfg=MOE_CONFIG, T=None, H=None):
    """Token activations x: bf16 encodings [T, H], N(0,1)."""
    T = cfg.T if T is None else T
    H = cfg.H if H is None else H
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg.seed_x)))
    return normal_bf16(rng, T * H).reshape(T, H)


def moe_expert_outputs(cfg=MOE_CONFIG, rows=None, H=None):
    """Expert outputs y in the packed layout: bf16 encodings [T*K, H], N(0,1)."""
    rows = cfg.T * cfg.K if rows is None else rows
    H = cfg.H if H is None else H
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(cfg.seed_y)))
    return normal_bf16(rng, rows * H).reshape(rows, H)


def zipf_split(total_bytes, W=8, s=0.125, min_unit=128):
    """Partition sizes in bytes for the variable-size collectives (Eq. 4,
    Appendix C.4 of the paper): units of u = max(min_unit, T / (8 W)) bytes,
    rank r gets floor(x_r) units with x_r = (T/u) (r+1)^-s / sum_k (k+1)^-s,
    and the leftover units go, one each, to the largest fractional parts of
    x_r, ties to the lower rank.  Exact for the power-of-two totals the paper
    uses (T a multiple of u)."""
    u = max(min_unit, total_bytes // (8 * W))
    units = total_bytes // u
    w = [(r + 1) ** (-s) for r in range(W)]
    tot = sum(w)
    x = [units * wr / tot for wr in w]
    base = [int(xr // 1) for xr in x]
    left = units - sum(base)
    order = sorted(range(W), key=lambda r: (-(x[r] - base[r]), r))
    for r in order[:left]:
        base[r] += 1
    return [u * b for b in base]


def rotate_right(v, k):
    """v rotated right by k positions: out[i] = v[(i - k) mod len(v)]."""
    n = len(v)
    return [v[(i - k) % n] for i in range(n)]


def alltoallv_counts(split):
    """AllToAllV sizes of Appendix C.4: rank p sends its split rotated right by
    (p + 1) mod W positions, so every rank sends and receives the total.
    Returns counts[p][r] = what rank p sends to rank r."""
    W = len(split)
    return [rotate_right(split, (p + 1) % W) for p in range(W)]
