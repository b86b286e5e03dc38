"""Seeded random shapes through the MoE kernels and the variable-size
collectives, every result bit-identical to the oracle's.

MoE: token count (including none), row length (rows that are and are not a
multiple of 16 bytes), slots per token, experts per rank, rank count and
routing skew are drawn per seed; pack, combine and their de-duplicated
variants are checked whole.  Variable-size: op, dtype, rank count, unit,
capacities (AllToAllV with a larger output than input side, so that its
items cover the sources), chunk, work-item size, bounded grid, transposed
counts and how full the sizes are, drawn per seed; outputs are guarded
buffers and nothing past the received sizes may change.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import Guarded, assert_bits_equal, np_dtype, to_device, to_host, torch_dtype
from paper_2609_36954_amd import purlin as PL

pytestmark = pytest.mark.gpu


def _normal_bf16(rng, shape):
    return oracle.narrow(rng.standard_normal(shape).astype(np.float32))


def _routing(rng, T, E, K, skew):
    """K distinct experts per token; skewed draws favour low expert ids."""
    w = (np.arange(E) + 1.0) ** -1.1 if skew else np.ones(E)
    w /= w.sum()
    ids = np.empty((T, K), dtype=np.int32)
    for t in range(T):
        ids[t] = rng.choice(E, K, replace=False, p=w)
    return ids


def _moe_case(seed):
    rng = np.random.default_rng(1000 + seed)
    P = int(rng.choice([1, 2, 3, 4, 8, 16]))
    L = int(rng.integers(1, 33))
    E = P * L
    K = int(rng.integers(1, min(8, E) + 1))
    if seed % 2 == 0:
        H = 8 * int(rng.integers(1, 513))  # 16-byte rows: one wave per 1 KiB slice
    else:
        H = int(rng.integers(1, 1500))     # any length: one wave per token
    T = 0 if seed % 11 == 5 else int(rng.integers(1, 600))
    return rng, T, H, K, E, P, bool(seed % 3)


@pytest.mark.parametrize("seed", range(24))
def test_random_moe_matches_oracle(seed):
    rng, T, H, K, E, P, skew = _moe_case(seed)
    what = f"seed {seed}: T={T} H={H} K={K} E={E} P={P} skew={skew}"
    x = _normal_bf16(rng, (T, H))
    ids = _routing(rng, T, E, K, skew)
    y = _normal_bf16(rng, (T * K, H))
    logits = rng.standard_normal((T, K))
    g = (np.exp(logits) / np.exp(logits).sum(axis=1, keepdims=True)).astype(np.float32)

    want = oracle.pack(x, ids, E, P)
    got = PL.purlin_pack(to_device(x).view(T, H), to_device(ids), E, P)
    torch.cuda.synchronize()
    for key in ("pos", "dest_counts", "dest_offsets", "expert_counts", "expert_offsets"):
        assert np.array_equal(to_host(got[key], np.int32).reshape(want[key].shape), want[key]), (what, key)
    assert np.array_equal(to_host(got["packed"], np.uint16).reshape(T * K, H), want["packed"]), what

    out = PL.purlin_unpack(to_device(y).view(T * K, H), got["pos"], to_device(g))
    torch.cuda.synchronize()
    assert_bits_equal(to_host(out, np.uint16).reshape(T, H), oracle.unpack(y, want["pos"], g), "bf16", what)

    wd = oracle.pack_dedup(x, ids, E, P)
    gd = PL.purlin_pack_dedup(to_device(x).view(T, H), to_device(ids), E, P)
    torch.cuda.synchronize()
    for key in ("dest_counts", "dest_offsets", "row_of"):
        assert np.array_equal(to_host(gd[key], np.int32).reshape(wd[key].shape), wd[key]), (what, key)
    n = int(wd["dest_counts"].sum())
    assert np.array_equal(to_host(gd["packed"], np.uint16).reshape(-1, H)[:n], wd["packed"][:n]), what
    yd = _normal_bf16(rng, (max(n, 1), H))
    od = PL.purlin_unpack_dedup(to_device(yd).view(-1, H), gd["row_of"])
    torch.cuda.synchronize()
    assert_bits_equal(to_host(od, np.uint16).reshape(T, H), oracle.unpack_dedup(yd, wd["row_of"]), "bf16", what)


def _inputs(rng, P, n, dtype):
    if dtype == "fp32":
        return [(rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32) for _ in range(P)]
    return [_normal_bf16(rng, n) for _ in range(P)]


def _fits(op, m, P, in_units, out_units):
    if op == "allgatherv":
        return all(c <= in_units for c in m[0]) and sum(m[0]) <= out_units
    if op == "reduce_scatterv":
        return all(c <= out_units for c in m[0]) and sum(m[0]) <= in_units
    return (all(sum(m[p]) <= in_units for p in range(P))
            and all(sum(m[p][r] for p in range(P)) <= out_units for r in range(P)))


@pytest.mark.parametrize("seed", range(24))
def test_random_variable_size_matches_oracle(seed):
    rng = np.random.default_rng(2000 + seed)
    op = ("allgatherv", "reduce_scatterv", "alltoallv")[seed % 3]
    dtype = ("fp32", "bf16")[(seed // 3) % 2]
    s = 4 if dtype == "fp32" else 2
    P = int(rng.integers(1, 17))
    unit = int(rng.choice([1, 2, 3, 5, 8]))
    in_cap = unit * int(rng.integers(0, 1200))
    out_cap = in_cap if op != "alltoallv" or seed % 2 else in_cap + unit * int(rng.integers(0, 800))
    if op == "allgatherv":
        out_cap = max(out_cap, in_cap * P)
    if op == "reduce_scatterv":
        in_cap, out_cap = max(in_cap, out_cap * P), out_cap
    in_units, out_units = in_cap // unit, out_cap // unit
    rows = P if op == "alltoallv" else 1
    fill = float(rng.uniform(0.0, 1.0))
    bound = max(in_units, out_units) // max(P, 1)
    m = [[int(x) for x in rng.integers(0, int(fill * bound) + 1, P)] for _ in range(rows)]
    while not _fits(op, m, P, in_units, out_units):
        m = [[c // 2 for c in row] for row in m]
    transposed = op == "alltoallv" and seed % 4 == 1
    flat = [m[r][p] for p in range(P) for r in range(P)] if transposed else [c for row in m for c in row]
    chunk = s * int(rng.integers(1, 3000))
    pol = dict(item_bytes=16 * int(rng.choice([0, 1, 3, 64, 256])),
               max_workgroups=int(rng.choice([0, 0, 1, 3, 64])))
    what = f"seed {seed}: {op} {dtype} P={P} unit={unit} caps={in_cap}/{out_cap} counts={m} policy={pol}"

    ins = _inputs(rng, P, in_cap, dtype)
    want = (oracle.all_gather_v(ins, [c * unit for c in m[0]], dtype) if op == "allgatherv" else
            oracle.reduce_scatter_v(ins, [c * unit for c in m[0]], dtype) if op == "reduce_scatterv" else
            oracle.all_to_all_v(ins, [[c * unit for c in row] for row in m], dtype))
    plan = PL.Plan(op, P, in_cap, dtype, chunk, policy=pol, unit=unit, out_capacity=out_cap,
                   counts_transposed=transposed)
    outs = [Guarded(plan.out_bytes, torch_dtype(dtype)) for _ in range(P)]
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    plan.exec_v([to_device(a) for a in ins], [o.t for o in outs], to_device(np.asarray(flat, np.int32)), dev_status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0, what
    for r in range(P):
        assert outs[r].intact(), what
        got = to_host(outs[r].t, np_dtype(dtype))
        n = len(want[r])
        assert_bits_equal(got[:n], want[r], dtype, f"{what} rank {r}")
        assert np.all(outs[r].t.view(torch.uint8)[n * s:].cpu().numpy() == 0xA5), f"{what}: wrote past rank {r}'s size"
