"""Variable-size collectives on the CPU: the plan's virtual index space and
the device-side size mapping (modelled by tests/interp.run_v) against the
oracle, and ABI validation."""

import ctypes

import numpy as np
import pytest

import interp
import oracle
from case_seed import case_seed
from paper_2609_36954_amd import purlin as PL
from paper_2609_36954_amd import workloads as W

S = {"fp32": 4, "bf16": 2}
INVALID = PL.PURLIN_ERR_INVALID


def _inputs(P, n, dtype, seed):
    rng = np.random.default_rng(seed)
    if dtype == "fp32":
        return [(rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32) for _ in range(P)]
    return [oracle.narrow(rng.standard_normal(n).astype(np.float32)) for _ in range(P)]


def _case_counts(kind, op, P, cap, rng):
    if kind == "zipf":
        split = [b // 128 for b in W.zipf_split(128 * 64)]  # element units
        split = (split * ((P + 7) // 8))[:P]
        if op == "alltoallv":
            return [x for row in W.alltoallv_counts(split) for x in row][: P * P] if P == 8 else \
                [int(x) for x in rng.integers(0, cap // P + 1, P * P)]
        return split
    if kind == "zero":
        return [0] * (P * P if op == "alltoallv" else P)
    if op == "alltoallv":
        return [int(x) for x in rng.integers(0, cap // P + 1, P * P)]
    return [int(x) for x in rng.integers(0, cap // P + 1, P)]


def _oracle_v(op, ins, counts, P, dtype, unit):
    c = [x * unit for x in counts]
    if op == "allgatherv":
        return oracle.all_gather_v(ins, c, dtype)
    if op == "reduce_scatterv":
        return oracle.reduce_scatter_v(ins, c, dtype)
    return oracle.all_to_all_v(ins, [c[p * P:(p + 1) * P] for p in range(P)], dtype)


CASES = [(op, dt, P, kind, unit) for op in ("allgatherv", "reduce_scatterv", "alltoallv") for dt in ("fp32", "bf16")
         for P in (1, 3, 8) for kind in ("random", "zipf", "zero") for unit in (1, 3)]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_v_mapping_matches_oracle(case):
    op, dtype, P, kind, unit = case
    rng = np.random.default_rng(case_seed(case) % 1000)
    cap = 600
    s = S[dtype]
    counts = _case_counts(kind, op, P, cap // unit, rng)
    ins = _inputs(P, cap, dtype, seed=len(counts))
    want = _oracle_v(op, ins, counts, P, dtype, unit)
    for chunk_elems, item in ((64, 0), (7, 16), (1000, 48)):
        plan = PL.Plan(op, P, cap, dtype, chunk_elems * s, policy=dict(item_bytes=item) if item else None,
                       host_only=True, unit=unit)
        items, pb = plan.items()
        assert pb[1] == pb[2]  # one launch
        bufs = [np.frombuffer(a.tobytes(), np.uint8).copy() for a in ins] + \
               [np.full(cap * s, 0xA5, np.uint8) for _ in range(P)]
        assert interp.run_v(items, bufs, counts, op, P, unit, dtype, cap)
        for r in range(P):
            n = len(want[r])
            got = bufs[P + r][: n * s].view(np.uint16 if dtype == "bf16" else np.uint32)
            assert np.array_equal(got, want[r].view(got.dtype)), (op, r)
            assert np.all(bufs[P + r][n * s:] == 0xA5), "written past the received size"


@pytest.mark.parametrize("op", ["allgatherv", "reduce_scatterv", "alltoallv"])
def test_v_rejects_oversized_and_negative_counts(op):
    P, cap = 4, 100
    bad = [[-1, 0, 0, 0], [60, 50, 0, 0]] if op != "alltoallv" else [[-1] + [0] * 15, [60, 50] + [0] * 14,
                                                                      [30, 0, 0, 0] * 4]
    plan = PL.Plan(op, P, cap, "fp32", 64, host_only=True, unit=1)
    items, _ = plan.items()
    for counts in bad:
        bufs = [np.zeros(cap * 4, np.uint8) for _ in range(2 * P)]
        assert not interp.run_v(items, bufs, counts, op, P, 1, "fp32", cap)


def test_v_plan_tables():
    P, cap = 8, 1 << 20
    for op, spaces in (("allgatherv", 1), ("reduce_scatterv", 1), ("alltoallv", P)):
        plan = PL.Plan(op, P, cap, "bf16", 1 << 16, host_only=True, unit=1)
        d = plan.descriptors()
        assert len(d) == spaces * (cap * 2 // (1 << 16))
        assert plan.in_bytes == plan.out_bytes == cap * 2
        if op == "alltoallv":
            assert sorted(set(d["part"].tolist())) == list(range(P))


def _plan_v_status(op, P, cap, dtype=1, chunk=256, unit=1, flags=PL.PLAN_HOST_ONLY):
    h = ctypes.c_void_p()
    st = PL.lib().purlin_plan_v(op, P, cap, cap, dtype, chunk, unit, None, flags, ctypes.byref(h))
    if h.value:
        PL.lib().purlin_plan_destroy(h)
    return st


@pytest.mark.parametrize("args,want", [
    ((8, 4, 1000), 0), ((9, 4, 1000), 0), ((10, 4, 1000), 0),
    ((0, 4, 1000), INVALID), ((4, 4, 1000), INVALID), ((11, 4, 1000), INVALID),  # non-V ops
    ((8, 0, 1000), INVALID), ((8, 17, 1000), INVALID),
    ((8, 4, 1000, 1, 3), INVALID),  # chunk not a multiple of the element size
    ((8, 4, 1000, 1, 256, 0), INVALID), ((8, 4, 1000, 1, 256, (1 << 31) + 1), INVALID),  # unit
    ((8, 4, 999), 0),  # capacity need not be a multiple of P
])
def test_plan_v_validation(args, want):
    assert _plan_v_status(*args) == want


def test_exec_v_and_exec_reject_the_other_kind():
    L = PL.lib()
    v = PL.Plan("allgatherv", 2, 64, "bf16", 32, host_only=True, unit=1)
    f = PL.Plan("allgather", 2, 64, "bf16", 32, host_only=True)
    bufs = (ctypes.c_void_p * 4)(0x1000, 0x2000, 0x3000, 0x4000)
    assert L.purlin_exec(v.handle, bufs, None) == INVALID
    assert L.purlin_exec_v(f.handle, bufs, 0x5000, None, None) == INVALID
    assert L.purlin_exec_v(v.handle, bufs, None, None, None) == INVALID  # no counts
    assert L.purlin_exec_v(v.handle, bufs, 0x5002, None, None) == INVALID  # misaligned counts


ASYM = [("allgatherv", 150, 1000), ("reduce_scatterv", 1000, 150), ("alltoallv", 400, 900), ("alltoallv", 900, 400)]


@pytest.mark.parametrize("op,in_cap,out_cap", ASYM)
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_v_mapping_with_separate_capacities(op, in_cap, out_cap, dtype):
    """Inputs and outputs of different sizes (e.g. expert-parallel dispatch:
    T*K rows sent, up to P*T*K received)."""
    P, s = 6, S[dtype]
    rng = np.random.default_rng(len(op) + in_cap)
    if op == "allgatherv":
        counts = [int(x) for x in rng.integers(0, in_cap + 1, P)]
        counts[-1] = in_cap  # a full input
    elif op == "reduce_scatterv":
        counts = [int(x) for x in rng.integers(0, out_cap + 1, P)]
        counts[0] = out_cap
    else:
        m = np.zeros((P, P), np.int64)
        for p in range(P):  # row sums <= in_cap, column sums <= out_cap
            for r in range(P):
                room = min(in_cap - m[p].sum(), out_cap - m[:, r].sum())
                m[p, r] = rng.integers(0, room + 1) if r < P - 1 else room
        counts = [int(x) for x in m.reshape(-1)]
    ins = _inputs(P, in_cap, dtype, seed=7)
    want = _oracle_v(op, ins, counts, P, dtype, 1)
    plan = PL.purlin_plan_v(op, P, in_cap, dtype, 64 * s, unit=1, out_capacity=out_cap, host_only=True)
    assert plan.in_bytes == in_cap * s and plan.out_bytes == out_cap * s
    items, _ = plan.items()
    bufs = [np.frombuffer(a.tobytes(), np.uint8).copy() for a in ins] + \
           [np.full(out_cap * s, 0xA5, np.uint8) for _ in range(P)]
    assert interp.run_v(items, bufs, counts, op, P, 1, dtype, in_cap, out_cap)
    for r in range(P):
        n = len(want[r])
        got = bufs[P + r][: n * s].view(np.uint16 if dtype == "bf16" else np.uint32)
        assert np.array_equal(got, want[r].view(got.dtype)), (op, r)
        assert np.all(bufs[P + r][n * s:] == 0xA5)


@pytest.mark.parametrize("op,in_cap,out_cap,counts", [
    ("allgatherv", 10, 100, [11, 0]),  # one input overflows its buffer
    ("allgatherv", 100, 10, [6, 5]),  # the gathered total overflows
    ("reduce_scatterv", 10, 100, [6, 5]),  # the partitioned total overflows the input
    ("reduce_scatterv", 100, 10, [11, 0]),  # one output overflows
    ("alltoallv", 10, 100, [6, 5, 0, 0]),  # a send row overflows the input
    ("alltoallv", 100, 10, [6, 0, 5, 0]),  # a receive column overflows the output
])
def test_v_rejects_sizes_beyond_either_capacity(op, in_cap, out_cap, counts):
    plan = PL.purlin_plan_v(op, 2, in_cap, "fp32", 64, unit=1, out_capacity=out_cap, host_only=True)
    items, _ = plan.items()
    bufs = [np.zeros(in_cap * 4, np.uint8) for _ in range(2)] + [np.zeros(out_cap * 4, np.uint8) for _ in range(2)]
    assert not interp.run_v(items, bufs, counts, op, 2, 1, "fp32", in_cap, out_cap)


@pytest.mark.parametrize("op,flags,want", [
    (10, 3, 0), (8, 3, INVALID), (9, 3, INVALID), (10, 5, INVALID)])
def test_plan_v_counts_transposed_flag(op, flags, want):
    assert _plan_v_status(op, 4, 1000, flags=flags) == want


@pytest.mark.parametrize("P", [1, 3, 8])
def test_alltoallv_transposed_counts(P):
    """Column-major sizes give the same exchange as the row-major matrix."""
    rng = np.random.default_rng(P)
    cap = 500
    m = rng.integers(0, cap // P + 1, (P, P))
    ins = _inputs(P, cap, "bf16", seed=P)
    want = oracle.all_to_all_v(ins, m.tolist(), "bf16")
    plan = PL.purlin_plan_v("alltoallv", P, cap, "bf16", 128, unit=1, host_only=True, counts_transposed=True)
    items, _ = plan.items()
    bufs = [np.frombuffer(a.tobytes(), np.uint8).copy() for a in ins] + \
           [np.full(cap * 2, 0xA5, np.uint8) for _ in range(P)]
    assert interp.run_v(items, bufs, m.T.reshape(-1).tolist(), "alltoallv", P, 1, "bf16", cap, transposed=True)
    for r in range(P):
        n = len(want[r])
        assert np.array_equal(bufs[P + r][: n * 2].view(np.uint16), want[r])
        assert np.all(bufs[P + r][n * 2:] == 0xA5)


def test_expert_parallel_round_trip_mapping():
    """Dispatch (pack, then AllToAllV of rows with the packs' dest_counts)
    and combine (the reverse AllToAllV with the same counts read
    column-major, then unpack) on the CPU: the reverse exchange restores
    every rank's packed order, so with identity experts the combine equals
    unpack(pack) of each rank (Table 2: EP dispatch / combine)."""
    P, T, H, K, E = 4, 40, 6, 3, 8
    rng = np.random.default_rng(11)
    xs = [oracle.narrow(rng.standard_normal((T, H)).astype(np.float32)) for _ in range(P)]
    ids = [np.stack([rng.permutation(E)[:K] for _ in range(T)]).astype(np.int32) for _ in range(P)]
    gates = [rng.random((T, K)).astype(np.float32) for _ in range(P)]
    packs = [oracle.pack(xs[p], ids[p], E, P) for p in range(P)]
    counts = [int(x) for p in range(P) for x in packs[p]["dest_counts"]]  # row p = rank p's dest_counts
    in_cap, out_cap = T * K * H, P * T * K * H
    fwd = PL.purlin_plan_v("alltoallv", P, in_cap, "bf16", 64, unit=H, out_capacity=out_cap, host_only=True)
    bwd = PL.purlin_plan_v("alltoallv", P, out_cap, "bf16", 64, unit=H, out_capacity=in_cap, host_only=True,
                           counts_transposed=True)
    bufs = [np.frombuffer(packs[p]["packed"].tobytes(), np.uint8).copy() for p in range(P)] + \
           [np.zeros(out_cap * 2, np.uint8) for _ in range(P)]
    assert interp.run_v(fwd.items()[0], bufs, counts, "alltoallv", P, H, "bf16", in_cap, out_cap)
    recv = bufs[P:]
    want_recv = oracle.all_to_all_v([pk["packed"].reshape(-1) for pk in packs],
                                    [[c * H for c in counts[p * P:(p + 1) * P]] for p in range(P)], "bf16")
    for r in range(P):
        assert np.array_equal(recv[r][: want_recv[r].size * 2].view(np.uint16), want_recv[r])
    bufs2 = recv + [np.zeros(in_cap * 2, np.uint8) for _ in range(P)]
    assert interp.run_v(bwd.items()[0], bufs2, counts, "alltoallv", P, H, "bf16", out_cap, in_cap, transposed=True)
    for p in range(P):
        back = bufs2[P + p].view(np.uint16).reshape(T * K, H)
        assert np.array_equal(back, packs[p]["packed"])
        want = oracle.unpack(packs[p]["packed"], packs[p]["pos"], gates[p])
        got = oracle.unpack(back, packs[p]["pos"], gates[p])
        assert np.array_equal(got, want)


@pytest.mark.parametrize("in_cap,out_cap,src_major", [(100, 800, True), (800, 100, False), (300, 300, False)])
def test_alltoallv_covers_the_smaller_side(in_cap, out_cap, src_major):
    P, chunk = 4, 64
    plan = PL.purlin_plan_v("alltoallv", P, in_cap, "fp32", chunk, unit=1, out_capacity=out_cap, host_only=True)
    d = plan.descriptors()
    space = min(in_cap, out_cap) * 4
    assert len(d) == P * -(-space // chunk)
    assert sorted(set(d["part"].tolist())) == list(range(P))
    if src_major:
        assert np.array_equal(d["src_buf"], d["part"]) and np.all(d["dst_step"] == 1) and np.all(d["dst_buf"] == P)
    else:
        assert np.array_equal(d["dst_buf"], d["part"] + P) and np.all(d["dst_step"] == 0)


def _item_layout_ok(d, spaces, chunk, item_bytes):
    """Item j of every space starts at (j // per_chunk) * chunk + (j % per_chunk) * item."""
    n = len(d)
    assert n % spaces == 0
    per_space = n // spaces
    per_chunk = -(-chunk // item_bytes)
    for k in range(spaces):
        seg = d[k * per_space:(k + 1) * per_space]
        assert np.all(seg["part"] == (k if spaces > 1 else 0))
        j = np.arange(per_space)
        assert np.array_equal(seg["src_off"], (j // per_chunk) * chunk + (j % per_chunk) * item_bytes)
    return per_space, per_chunk


def _active(extent, chunk, item_bytes, per_chunk, per_space):
    """The kernels' closed form: items of a space that start below `extent` bytes."""
    if extent == 0:
        return 0
    o = extent - 1
    return min(per_space, (o // chunk) * per_chunk + (o % chunk) // item_bytes + 1)


@pytest.mark.parametrize("op", ["allgatherv", "reduce_scatterv", "alltoallv"])
@pytest.mark.parametrize("cap,chunk_e,item", [(1000, 64, 0), (999, 7, 16), (4096, 1000, 48), (5, 1000, 0),
                                              (12345, 256, 128)])
def test_v_items_follow_the_closed_form_the_kernels_use(op, cap, chunk_e, item):
    """The V kernels enumerate only the items below the run-time extent by
    arithmetic on (chunk, item); this pins the table layout that relies on."""
    P, s = 4, 2
    plan = PL.Plan(op, P, cap, "bf16", chunk_e * s, policy=dict(item_bytes=item) if item else None, host_only=True,
                   unit=1)
    items, _ = plan.items()
    spaces = P if op == "alltoallv" else 1
    item_bytes = int(items["bytes"].max())
    per_space, per_chunk = _item_layout_ok(items, spaces, chunk_e * s, item_bytes)
    for extent in sorted({0, 1, s, chunk_e * s - s, chunk_e * s, chunk_e * s + s, cap * s // 2, cap * s - s, cap * s}):
        if extent < 0 or extent > cap * s:
            continue
        want = int(np.sum(items["src_off"][:per_space] < extent))
        assert _active(extent, chunk_e * s, item_bytes, per_chunk, per_space) == want, extent
