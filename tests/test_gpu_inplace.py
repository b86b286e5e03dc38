"""In-place collectives on the GPU.

A rank's input and output may be one buffer where every element is read
before it is rewritten (AllReduce, Broadcast, Reduce: in_r == out_r;
ReduceScatter, Scatter: out_r = in_r + r * out_bytes; AllGather, Gather:
in_r = out_r + r * in_bytes).  The results must equal the oracle's on the
same inputs, bit for bit, for every AllReduce mode; every other overlap is
rejected on the host before anything runs.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_bits_equal, np_dtype, to_device, to_host
from paper_2609_36954_amd import purlin as PL
from test_gpu_exec import _inputs

pytestmark = pytest.mark.gpu

S = {"fp32": 4, "bf16": 2}
SHAPES = ((1, 1000), (3, 4099), (8, 20003))
# in place at an offset of r partitions: the partition must keep the 16-byte alignment
PART_SHAPES = ((1, 1000), (3, 4104), (8, 20008))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P,M", SHAPES)
@pytest.mark.parametrize("pol", [{"ar_mode": 1}, {"ar_mode": 1, "fanout": 2}, {"ar_mode": 2}, {"ar_mode": 3}])
def test_allreduce_in_place(dtype, P, M, pol):
    s = S[dtype]
    ins_np = _inputs(P, P * M, dtype, seed=P + M)
    want = oracle.all_reduce(ins_np, dtype)
    plan = PL.Plan("allreduce", P, P * M, dtype, 512 * s, policy=dict(item_bytes=1024, **pol))
    bufs = [to_device(a) for a in ins_np]
    for rep in range(2):  # twice: the second run reduces the first run's results
        plan.exec(bufs, bufs)
        torch.cuda.synchronize()
        for r in range(P):
            assert_bits_equal(to_host(bufs[r], np_dtype(dtype)), want[r], dtype, f"{pol} rank {r} run {rep}")
        ins_np = [w.copy() for w in want]
        want = oracle.all_reduce(ins_np, dtype)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P,M", PART_SHAPES)
def test_reduce_scatter_and_allgather_in_place(dtype, P, M):
    s = S[dtype]
    ins_np = _inputs(P, P * M, dtype, seed=3 * P + M)
    rs_want = oracle.reduce_scatter(ins_np, dtype)
    ag_want = oracle.all_gather(rs_want, dtype)
    bufs = [to_device(a) for a in ins_np]
    parts = [b[r * M:(r + 1) * M] for r, b in enumerate(bufs)]  # rank r's result lands in its own partition
    PL.Plan("reduce_scatter", P, P * M, dtype, 256 * s).exec(bufs, parts)
    torch.cuda.synchronize()
    for r in range(P):
        assert_bits_equal(to_host(parts[r], np_dtype(dtype)), rs_want[r], dtype, f"ReduceScatter rank {r}")
    # AllGather back in place: rank r's contribution already sits at out_r + r * M
    PL.Plan("allgather", P, P * M, dtype, 256 * s).exec(parts, bufs)
    torch.cuda.synchronize()
    for r in range(P):
        assert_bits_equal(to_host(bufs[r], np_dtype(dtype)), ag_want[r], dtype, f"AllGather rank {r}")


@pytest.mark.parametrize("op", ["broadcast", "reduce", "scatter", "gather"])
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_rooted_in_place_at_the_root(op, dtype):
    P, M = 5, 3000
    s = S[dtype]
    ins_np = _inputs(P, P * M, dtype, seed=17)
    root = 3
    if op == "gather":
        want = oracle.gather([a[:M] for a in ins_np], root, dtype)
    else:
        want = getattr(oracle, op)(ins_np, root, dtype)
    plan = PL.Plan(op, P, P * M, dtype, 256 * s, root=root)
    full = [to_device(a) for a in ins_np]
    if op == "broadcast":  # the root's input is its output
        ins = [full[root] if r == root else None for r in range(P)]
        outs = [full[root] if r == root else torch.empty_like(full[r]) for r in range(P)]
    elif op == "reduce":  # the root's output is its input
        ins = full
        outs = [full[root] if r == root else None for r in range(P)]
    elif op == "scatter":  # the root keeps its partition where it is
        ins = [full[root] if r == root else None for r in range(P)]
        outs = [full[root][root * M:(root + 1) * M] if r == root else torch.empty(M, dtype=full[0].dtype,
                                                                                  device="cuda") for r in range(P)]
    else:  # gather: the root's contribution already sits at out_root + root * M
        ins = [to_device(a[:M]) for a in ins_np]
        full[root][root * M:(root + 1) * M].copy_(ins[root])
        ins[root] = full[root][root * M:(root + 1) * M]
        outs = [full[root] if r == root else None for r in range(P)]
    plan.exec(ins, outs)
    torch.cuda.synchronize()
    for r in range(P):
        if want[r] is not None:
            assert_bits_equal(to_host(outs[r], np_dtype(dtype)), want[r], dtype, f"{op} rank {r}")


def test_other_overlaps_are_rejected():
    P, M = 4, 1024
    bufs = [torch.zeros(P * M, dtype=torch.float32, device="cuda") for _ in range(P)]
    ar = PL.Plan("allreduce", P, P * M, "fp32", 1024)
    with pytest.raises(PL.PurlinError):  # in_0 is out_1
        ar.exec(bufs, [bufs[1], bufs[0], bufs[2], bufs[3]])
    with pytest.raises(PL.PurlinError):  # aliased inputs written in place
        ar.exec([bufs[0], bufs[0], bufs[2], bufs[3]], [bufs[0], bufs[0], bufs[2], bufs[3]])
    rs = PL.Plan("reduce_scatter", P, P * M, "fp32", 1024)
    with pytest.raises(PL.PurlinError):  # out_1 at the start of in_1 instead of its partition
        rs.exec(bufs, [b[:M] for b in bufs])
    a2a = PL.Plan("alltoall", P, P * M, "fp32", 1024)
    with pytest.raises(PL.PurlinError):
        a2a.exec(bufs, bufs)
    # nothing ran: the buffers are untouched
    torch.cuda.synchronize()
    assert all(bool((b == 0).all()) for b in bufs)
