"""One rank's share of a collective (purlin_plan_share) on the GPU.

* every op: the P shares, executed rank after rank in reverse order into
  guarded outputs, give the oracle's result bit for bit; a share executed
  alone writes its own output and leaves every other output untouched;
* AllReduce: a share's phase 1 pulls partition k from out_k, which rank k's
  share wrote in its phase 0.  So the outputs first hold the full result,
  then each share is executed alone with its own output reset: it must
  rebuild that output exactly and change nothing else;
* rank 0's share of ReduceScatter and AllGather at 256 MiB per rank (P = 8,
  bf16), compared with the oracle in full.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import Guarded, assert_bits_equal, np_dtype, to_device, to_host, torch_dtype
from paper_2609_36954_amd import purlin as PL
from paper_2609_36954_amd import workloads as W
from test_gpu_exec import _inputs

pytestmark = pytest.mark.gpu

S = {"fp32": 4, "bf16": 2}
SENTINEL = 0x5A


def _want(op, ins, dtype, P, M, root):
    if op == "allgather":
        return oracle.all_gather([a[:M] for a in ins], dtype)
    if op == "gather":
        return oracle.gather([a[:M] for a in ins], root, dtype)
    if op in PL.ROOTED:
        return getattr(oracle, op)(ins, root, dtype)
    return {"allreduce": oracle.all_reduce, "reduce_scatter": oracle.reduce_scatter,
            "alltoall": oracle.all_to_all}[op](ins, dtype)


CASES = []
for _op in ("reduce_scatter", "allgather", "alltoall", "broadcast", "reduce", "scatter", "gather"):
    for _dt in ("fp32", "bf16"):
        for _P, _M, _ce in ((1, 1000, 64), (2, 4099, 1024), (3, 1001, 100), (8, 65553, 16384)):
            CASES.append((_op, _dt, _P, _M, _ce))


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_shares_match_oracle(case):
    op, dtype, P, M, ce = case
    s = S[dtype]
    ins_np = _inputs(P, P * M, dtype, seed=P * 31 + M)
    for root in ([0, P - 1] if op in PL.ROOTED else [None]):
        want = _want(op, ins_np, dtype, P, M, root)
        shares = [PL.Plan(op, P, P * M, dtype, ce * s, root=root, share=r) for r in range(P)]
        nbytes_in, nbytes_out = shares[0].in_bytes, shares[0].out_bytes
        ins = [to_device(a[: nbytes_in // s]) for a in ins_np]
        outs = [Guarded(nbytes_out, torch_dtype(dtype)) for _ in range(P)]
        for o in outs:
            o.t.view(torch.uint8).fill_(SENTINEL)
        # one share alone: its own output only
        r0 = P // 2
        shares[r0].exec(ins, [o.t for o in outs])
        torch.cuda.synchronize()
        for r in range(P):
            if r != r0:
                assert bool((outs[r].t.view(torch.uint8) == SENTINEL).all()), f"share {r0} wrote output {r}"
        for r in reversed(range(P)):
            shares[r].exec(ins, [o.t for o in outs])
        torch.cuda.synchronize()
        for r in range(P):
            assert outs[r].intact(), "write outside an output buffer"
            if want[r] is None:
                assert bool((outs[r].t.view(torch.uint8) == SENTINEL).all())
            else:
                assert_bits_equal(to_host(outs[r].t, np_dtype(dtype)), want[r], dtype, f"{op} root={root} rank {r}")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P,M,ce,pol", [(2, 4099, 1024, None), (3, 1001, 100, {"fanout": 2}),
                                        (8, 65553, 16384, None), (8, 3000, 512, {"ar_mode": 2})])
def test_allreduce_share_rebuilds_its_output(dtype, P, M, ce, pol):
    s = S[dtype]
    ins_np = _inputs(P, P * M, dtype, seed=P * 13 + M)
    want = oracle.all_reduce(ins_np, dtype)
    ins = [to_device(a) for a in ins_np]
    outs = [Guarded(P * M * s, torch_dtype(dtype)) for _ in range(P)]
    PL.Plan("allreduce", P, P * M, dtype, ce * s).exec(ins, [o.t for o in outs])
    torch.cuda.synchronize()
    for r in range(P):
        sh = PL.Plan("allreduce", P, P * M, dtype, ce * s, policy=pol, share=r)
        before = [to_host(o.t, np_dtype(dtype)).copy() for o in outs]
        outs[r].t.view(torch.uint8).fill_(SENTINEL)
        sh.exec(ins, [o.t for o in outs])
        torch.cuda.synchronize()
        for q in range(P):
            assert outs[q].intact()
            got = to_host(outs[q].t, np_dtype(dtype))
            if q == r:
                assert_bits_equal(got, want[r], dtype, f"share {r}")
            else:
                assert_bits_equal(got, before[q], dtype, f"share {r} changed output {q}")


def test_rank0_share_at_256MiB_per_rank():
    """Rank 0's ReduceScatter share (8 x 32 MiB in, 32 MiB out) and AllGather
    share (8 x 32 MiB in, 256 MiB out), bf16, chunk 1 MiB."""
    P, N = 8, 134217728
    M = N // P
    ins_np = [W.normal_bf16(r, N, 0.02) for r in W.rank_rngs(404, P)]
    ins = [to_device(a) for a in ins_np]
    rs = PL.Plan("reduce_scatter", P, N, "bf16", 1 << 20, share=0)
    rs_out = [torch.empty(M, dtype=torch.int16, device="cuda")] + [None] * (P - 1)
    rs.exec(ins, rs_out)
    # partition 0 of every rank reduced in rank order = an AllReduce of those partitions
    want = oracle.all_reduce([a[:M] for a in ins_np], "bf16")[0]
    assert_bits_equal(to_host(rs_out[0], np.uint16), want, "bf16", "ReduceScatter share of rank 0")
    # AllGather share: rank p contributes the first M elements of its input
    ag = PL.Plan("allgather", P, N, "bf16", 1 << 20, share=0)
    ag_in = [t[:M] for t in ins]
    ag_out = [torch.empty(N, dtype=torch.int16, device="cuda")] + [None] * (P - 1)
    ag.exec(ag_in, ag_out)
    got = to_host(ag_out[0], np.uint16)
    assert np.array_equal(got, np.concatenate([a[:M] for a in ins_np]))


PUSH_CASES = [c for c in CASES if c[0] in ("allgather", "alltoall", "broadcast", "scatter", "gather")]


@pytest.mark.parametrize("case", PUSH_CASES, ids=lambda c: "-".join(map(str, c)))
def test_push_shares_match_oracle(case):
    """Every rank pushes its input into the others' outputs (the descriptors
    that read in_rank); together the P push shares give the collective."""
    op, dtype, P, M, ce = case
    s = S[dtype]
    ins_np = _inputs(P, P * M, dtype, seed=P * 37 + M)
    for root in ([0, P - 1] if op in PL.ROOTED else [None]):
        want = _want(op, ins_np, dtype, P, M, root)
        shares = [PL.Plan(op, P, P * M, dtype, ce * s, root=root, share=r, push=True) for r in range(P)]
        ins = [to_device(a[: shares[0].in_bytes // s]) for a in ins_np]
        outs = [Guarded(shares[0].out_bytes, torch_dtype(dtype)) for _ in range(P)]
        for o in outs:
            o.t.view(torch.uint8).fill_(SENTINEL)
        for r in range(P):
            shares[r].exec(ins, [o.t for o in outs])
        torch.cuda.synchronize()
        for r in range(P):
            assert outs[r].intact()
            if want[r] is None:
                assert bool((outs[r].t.view(torch.uint8) == SENTINEL).all())
            else:
                assert_bits_equal(to_host(outs[r].t, np_dtype(dtype)), want[r], dtype, f"{op} push root={root} r={r}")
