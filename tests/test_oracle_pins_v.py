"""Pins of the variable-size collectives and of the Eq. 4 split.

* the split against what the paper states (tests/golden/zipf_split.txt) and
  against vectors worked out by hand from Eq. 4;
* AllGatherV / ReduceScatterV / AllToAllV against pure-Python brute force;
* uniform sizes reduce them to AllGather / ReduceScatter / AllToAll;
* ReduceScatterV then AllGatherV with the same sizes is AllReduce.
"""

import os

import numpy as np
import pytest

import brute
import oracle
from paper_2609_36954_amd import workloads as W
from test_oracle_pins import _as_bits, _rand_inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "zipf_split.txt")


def _golden():
    g = {}
    for line in open(GOLDEN):
        line = line.strip()
        if line and not line.startswith("#"):
            k, *v = line.split()
            g[k] = v
    return g


def test_split_matches_the_papers_statements():
    g = _golden()
    Wr, s, mu = int(g["W"][0]), float(g["s"][0]), int(g["min_unit"][0])
    for k in range(10, 31):  # 1 KiB .. 1 GiB
        T = 1 << k
        n = W.zipf_split(T, Wr, s, mu)
        assert sum(n) == T, "total preserved"
        assert all(x % 128 == 0 for x in n), "128-byte alignment"
        if T >= 8 * 1024:
            assert max(n) / (T / Wr) == pytest.approx(float(g["max_over_mean_for_T_ge_8KiB"][0]), abs=0)
        if str(T) in g["uniform_totals_bytes"]:
            assert len(set(n)) == 1, f"{T} bytes should split uniformly"
        rows = W.alltoallv_counts(n)
        assert all(sum(row) == T for row in rows), "every rank sends T"
        assert all(sum(rows[p][r] for p in range(Wr)) == T for r in range(Wr)), "every rank receives T"


def test_split_hand_worked_vectors():
    """Eq. 4 by hand (weights (r+1)^-0.125, sum 6.8016):
    T >= 8 KiB: 64 units of T/64, x = [9.41 8.63 8.20 7.91 7.70 7.52 7.38 7.25],
      floors sum to 60, leftover 4 to ranks 3, 4, 1, 5 -> [9 9 8 8 8 8 7 7];
    T = 4 KiB: 32 units of 128 B, x = [4.70 4.31 4.10 3.96 3.85 3.76 3.69 3.63],
      floors sum to 27, leftover 5 to ranks 3, 4, 5, 0, 6 -> [5 4 4 4 4 4 4 3]."""
    for T in (8 << 10, 1 << 20, 256 << 20, 1 << 30):
        assert W.zipf_split(T) == [T // 64 * u for u in (9, 9, 8, 8, 8, 8, 7, 7)]
    assert W.zipf_split(4096) == [128 * u for u in (5, 4, 4, 4, 4, 4, 4, 3)]
    assert W.rotate_right([0, 1, 2, 3], 1) == [3, 0, 1, 2]


def _rand_counts(rng, P, total_max):
    c = rng.integers(0, total_max // P + 3, P).tolist()
    return c


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P", [1, 2, 3, 4])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_v_brute_force(dtype, P, seed):
    rng = np.random.default_rng(seed)
    n = 12
    ins = _rand_inputs(P, n, dtype, 300 + seed)
    as_list = [a.tolist() for a in ins]
    counts = [int(c) for c in rng.integers(0, n // P + 1, P)]

    def same(o, b):
        if dtype == "fp32":
            assert o.view(np.uint32).tolist() == [brute.f32_bits(v) for v in b]
        else:
            assert o.tolist() == b

    for o, b in zip(oracle.all_gather_v(ins, counts, dtype), brute.all_gather_v(as_list, counts)):
        same(o, b)
    for o, b in zip(oracle.reduce_scatter_v(ins, counts, dtype), brute.reduce_scatter_v(as_list, counts, dtype)):
        same(o, b)
    m = [[int(x) for x in rng.integers(0, n // P + 1, P)] for _ in range(P)]
    for o, b in zip(oracle.all_to_all_v(ins, m, dtype), brute.all_to_all_v(as_list, m)):
        same(o, b)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P", [1, 3, 8])
def test_uniform_sizes_reduce_to_fixed_size(dtype, P):
    M = 37
    ins = _rand_inputs(P, P * M, dtype, 400 + P)
    if dtype == "bf16":
        ins = [a & np.uint16(0xBFFF) for a in ins]
    eq = lambda a, b: np.array_equal(_as_bits(a, dtype), _as_bits(b, dtype))  # noqa: E731
    for a, b in zip(oracle.all_gather_v(ins, [M] * P, dtype), oracle.all_gather([x[:M] for x in ins], dtype)):
        assert eq(a, b)
    for a, b in zip(oracle.reduce_scatter_v(ins, [M] * P, dtype), oracle.reduce_scatter(ins, dtype)):
        assert eq(a, b)
    for a, b in zip(oracle.all_to_all_v(ins, [[M] * P] * P, dtype), oracle.all_to_all(ins, dtype)):
        assert eq(a, b)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_rsv_then_agv_is_allreduce(dtype):
    P = 8
    split = [s // 128 for s in W.zipf_split(8 << 10)]  # element counts 9 9 8 8 8 8 7 7
    total = sum(split)
    assert total % P == 0
    ins = _rand_inputs(P, total, dtype, 500)
    if dtype == "bf16":
        ins = [a & np.uint16(0xBFFF) for a in ins]
    ag = oracle.all_gather_v(oracle.reduce_scatter_v(ins, split, dtype), split, dtype)
    ar = oracle.all_reduce(ins, dtype)
    for r in range(P):
        assert np.array_equal(_as_bits(ag[r], dtype), _as_bits(ar[r], dtype))


def test_alltoallv_moves_each_element_once():
    P = 5
    rng = np.random.default_rng(9)
    m = [[int(x) for x in rng.integers(0, 6, P)] for _ in range(P)]
    ins = [np.arange(p * 1000, p * 1000 + sum(m[p]), dtype=np.uint16) for p in range(P)]
    outs = oracle.all_to_all_v(ins, m, "bf16")
    seen = sorted(int(v) for o in outs for v in o)
    assert seen == sorted(int(v) for a in ins for v in a)
    for r in range(P):
        assert len(outs[r]) == sum(m[p][r] for p in range(P))


def test_v_rejects_bad_sizes():
    a = [np.zeros(8, np.float32)] * 2
    with pytest.raises(ValueError):
        oracle.all_gather_v(a, [9, 1], "fp32")
    with pytest.raises(ValueError):
        oracle.reduce_scatter_v(a, [5, 4], "fp32")
    with pytest.raises(ValueError):
        oracle.all_to_all_v(a, [[5, 4], [1, 1]], "fp32")
