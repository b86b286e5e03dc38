"""GPU parity of the variable-size collectives (sizes read from device memory)."""

import numpy as np
import pytest
import torch

import oracle
from case_seed import case_seed
from gpu_util import CANARY, Guarded, assert_bits_equal, np_dtype, to_device, to_host, torch_dtype
from paper_2609_36954_amd import purlin as PL
from paper_2609_36954_amd import workloads as W
from test_planner_v import _case_counts, _inputs, _oracle_v

pytestmark = pytest.mark.gpu

S = {"fp32": 4, "bf16": 2}


def run_v(plan, ins_np, counts, dtype):
    P = plan.P
    ins = [to_device(a) for a in ins_np]
    outs = [Guarded(plan.out_bytes, torch_dtype(dtype)) for _ in range(P)]
    st = torch.full((4,), 7, dtype=torch.int32, device="cuda")
    plan.exec_v(ins, [o.t for o in outs], to_device(np.asarray(counts, np.int32)), dev_status=st)
    torch.cuda.synchronize()
    for o in outs:
        assert o.intact()
    return [to_host(o.t, np_dtype(dtype)) for o in outs], int(st[0].item())


CASES = [(op, dt, P, kind, unit) for op in ("allgatherv", "reduce_scatterv", "alltoallv") for dt in ("fp32", "bf16")
         for P in (1, 3, 8, 16) for kind in ("random", "zipf", "zero") for unit in (1, 5)]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_v_matches_oracle(case):
    op, dtype, P, kind, unit = case
    rng = np.random.default_rng(case_seed(case))
    cap = 6000
    s = S[dtype]
    counts = _case_counts(kind, op, P, cap // unit, rng)
    ins = _inputs(P, cap, dtype, seed=len(counts) + P)
    want = _oracle_v(op, ins, counts, P, dtype, unit)
    for chunk in (64 * s, 1 << 20):
        plan = PL.Plan(op, P, cap, dtype, chunk, unit=unit)
        got, status = run_v(plan, ins, counts, dtype)
        assert status == 0
        for r in range(P):
            n = len(want[r])
            assert_bits_equal(got[r][:n], want[r], dtype, f"{op} P={P} {kind} unit={unit} chunk={chunk} rank {r}")
            tail = got[r][n:].view(np.uint8)
            assert np.all(tail == CANARY), "wrote past the received size"


@pytest.mark.parametrize("op", ["allgatherv", "reduce_scatterv", "alltoallv"])
def test_v_invalid_sizes_write_nothing(op):
    P, cap = 4, 1000
    plan = PL.Plan(op, P, cap, "bf16", 256, unit=1)
    ins = _inputs(P, cap, "bf16", 3)
    n = P * P if op == "alltoallv" else P
    for counts in ([-1] + [0] * (n - 1), [cap] + [1] + [0] * (n - 2)):
        got, status = run_v(plan, ins, counts, "bf16")
        assert status == 1
        for g in got:
            assert np.all(g.view(np.uint8) == CANARY)


def test_v_sizes_change_between_graph_replays():
    """Sizes live in device memory: one captured graph, different sizes per replay."""
    P, cap = 8, 1 << 16
    ins_np = _inputs(P, cap, "bf16", 5)
    plan = PL.Plan("alltoallv", P, cap, "bf16", 1 << 14, unit=1)
    ins = [to_device(a) for a in ins_np]
    outs = [torch.zeros(cap, dtype=torch.int16, device="cuda") for _ in range(P)]
    counts = torch.zeros(P * P, dtype=torch.int32, device="cuda")
    plan.exec_v(ins, outs, counts)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            plan.exec_v(ins, outs, counts, stream=side)
    rng = np.random.default_rng(6)
    for rep in range(4):
        if rep % 2:
            split = [b // 2 for b in W.zipf_split(cap * 2)]
            host = [x for row in W.alltoallv_counts(split) for x in row]
        else:
            host = [int(x) for x in rng.integers(0, cap // P + 1, P * P)]
        counts.copy_(torch.tensor(host, dtype=torch.int32))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        want = oracle.all_to_all_v(ins_np, [host[p * P:(p + 1) * P] for p in range(P)], "bf16")
        for r in range(P):
            assert_bits_equal(to_host(outs[r], np.uint16)[: len(want[r])], want[r], "bf16", f"replay {rep} rank {r}")


def test_v_zipf_split_at_256MiB_per_rank():
    """The Appendix C.4 setup at T = 256 MiB per rank, P = 8, bf16."""
    P, N = 8, 134217728
    T = N * 2
    split = [b // 2 for b in W.zipf_split(T)]
    ins_np = [W.normal_bf16(r, N, 0.02) for r in W.rank_rngs(404, P)]
    ins = [to_device(a) for a in ins_np]
    counts = to_device(np.asarray(split, np.int32))
    rng = np.random.default_rng(7)
    # ReduceScatterV: sampled against the oracle (elementwise across ranks)
    rsv = PL.Plan("reduce_scatterv", P, N, "bf16", 1 << 20, unit=1)
    outs = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    rsv.exec_v(ins, outs, counts)
    torch.cuda.synchronize()
    idx = np.sort(rng.integers(0, N, 8 * 65536))
    want = oracle.all_reduce([a[idx] for a in ins_np], "bf16")[0]
    offs = np.concatenate([[0], np.cumsum(split)])
    owner = np.searchsorted(offs, idx, side="right") - 1
    got = np.empty(len(idx), np.uint16)
    host = [to_host(o, np.uint16) for o in outs]
    for r in range(P):
        sel = owner == r
        got[sel] = host[r][idx[sel] - offs[r]]
    assert_bits_equal(got, want, "bf16", "ReduceScatterV sample")
    del host
    # AllGatherV of those results: every rank gets the concatenation == AllReduce
    agv = PL.Plan("allgatherv", P, N, "bf16", 1 << 20, unit=1)
    ag = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    agv.exec_v(outs, ag, counts)
    ar = PL.Plan("allreduce", P, N, "bf16", 1 << 20)
    ar_out = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    ar.exec(ins, ar_out)
    torch.cuda.synchronize()
    for r in range(P):
        assert torch.equal(ag[r], ar_out[0]), f"RSV then AGV differs from AllReduce at rank {r}"
    del ag, ar_out, outs
    # AllToAllV with the rotated splits: compare with slices assembled by torch
    m = W.alltoallv_counts(split)
    a2av = PL.Plan("alltoallv", P, N, "bf16", 1 << 20, unit=1)
    out2 = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    a2av.exec_v(ins, out2, to_device(np.asarray([x for row in m for x in row], np.int32)))
    torch.cuda.synchronize()
    for r in range(P):
        pieces = []
        for p in range(P):
            start = sum(m[p][:r])
            pieces.append(ins[p][start:start + m[p][r]])
        assert torch.equal(out2[r], torch.cat(pieces)), f"AllToAllV rank {r}"


@pytest.mark.parametrize("op", ["allgatherv", "reduce_scatterv", "alltoallv"])
def test_v_zero_capacity_still_checks_sizes(op):
    P = 4
    plan = PL.Plan(op, P, 0, "bf16", 256, unit=1)
    n = P * P if op == "alltoallv" else P
    empty = [torch.empty(0, dtype=torch.int16, device="cuda") for _ in range(P)]
    for counts, want in (([0] * n, 0), ([0] * (n - 1) + [1], 1)):
        st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
        plan.exec_v(empty, empty, to_device(np.asarray(counts, np.int32)), dev_status=st)
        torch.cuda.synchronize()
        assert int(st.item()) == want


@pytest.mark.parametrize("op", ["allgatherv", "reduce_scatterv", "alltoallv"])
def test_v_small_sizes_in_a_large_capacity(op):
    """Most items lie beyond the run-time sizes (the waves skip them)."""
    P, cap = 8, 1 << 20
    rng = np.random.default_rng(len(op))
    n = P * P if op == "alltoallv" else P
    counts = [int(x) for x in rng.integers(0, 3000, n)]
    ins = _inputs(P, cap, "bf16", seed=11)
    want = _oracle_v(op, ins, counts, P, "bf16", 1)
    plan = PL.Plan(op, P, cap, "bf16", 4096, unit=1)
    got, status = run_v(plan, ins, counts, "bf16")
    assert status == 0
    for r in range(P):
        assert_bits_equal(got[r][: len(want[r])], want[r], "bf16", f"{op} rank {r}")
        assert np.all(got[r][len(want[r]):].view(np.uint8) == CANARY)


@pytest.mark.parametrize("op", ["allgatherv", "reduce_scatterv", "alltoallv"])
def test_v_zero_capacity_accepts_null_buffers(op):
    """A zero-capacity plan ignores bufs, so a C caller may pass NULL."""
    import ctypes
    P = 4
    plan = PL.Plan(op, P, 0, "bf16", 256, unit=1)
    n = P * P if op == "alltoallv" else P
    for counts, want in (([0] * n, 0), ([1] + [0] * (n - 1), 1)):
        dev_counts = to_device(np.asarray(counts, np.int32))
        st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
        rc = PL.lib().purlin_exec_v(plan.handle, None, ctypes.c_void_p(dev_counts.data_ptr()),
                                    ctypes.c_void_p(st.data_ptr()), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        assert rc == 0
        torch.cuda.synchronize()
        assert int(st.item()) == want
    # without a status word nothing is launched at all
    rc = PL.lib().purlin_exec_v(plan.handle, None, ctypes.c_void_p(dev_counts.data_ptr()), None, None)
    assert rc == 0
