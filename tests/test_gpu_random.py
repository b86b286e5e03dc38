"""Seeded random configurations through the GPU kernels: any op, rank
count, ragged size, chunk and policy (item size, fan-out, AllReduce mode,
cache hints, bounded grid, copy depth), rank shares and in-place runs among
them; every result bit-identical to the oracle's."""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import Guarded, assert_bits_equal, np_dtype, to_device, to_host, torch_dtype
from paper_2609_36954_amd import purlin as PL

pytestmark = pytest.mark.gpu

S = {"fp32": 4, "bf16": 2}
OPS = ("allreduce", "reduce_scatter", "allgather", "alltoall", "broadcast", "reduce", "scatter", "gather")


def _inputs(P, n, dtype, rng):
    if dtype == "fp32":
        return [(rng.standard_normal(n) * np.exp2(rng.integers(-30, 30, n))).astype(np.float32) for _ in range(P)]
    return [oracle.narrow(rng.standard_normal(n).astype(np.float32)) for _ in range(P)]


def _want(op, ins, dtype, P, M, root):
    if op == "allgather":
        return oracle.all_gather([a[:M] for a in ins], dtype)
    if op == "gather":
        return oracle.gather([a[:M] for a in ins], root, dtype)
    if op in PL.ROOTED:
        return getattr(oracle, op)(ins, root, dtype)
    return {"allreduce": oracle.all_reduce, "reduce_scatter": oracle.reduce_scatter,
            "alltoall": oracle.all_to_all}[op](ins, dtype)


def _case(seed):
    rng = np.random.default_rng(seed)
    op = OPS[rng.integers(len(OPS))]
    dtype = ("fp32", "bf16")[rng.integers(2)]
    P = int(rng.integers(1, 17))
    M = int(rng.integers(0, 6000))
    pol = {"item_bytes": int(rng.choice([0, 16, 48, 256, 4096])), "fanout": int(rng.integers(0, 3)),
           "ar_mode": int(rng.integers(0, 4)), "load_hint": int(rng.integers(0, 3)),
           "store_hint": int(rng.integers(0, 3)), "max_workgroups": int(rng.choice([0, 0, 1, 5, 64])),
           "copy_depth": int(rng.choice([0, 1, 2, 4, 8]))}
    if pol["ar_mode"] == 3 and pol["max_workgroups"]:
        pol["max_workgroups"] = 0
    root = int(rng.integers(P)) if op in PL.ROOTED else None
    chunk = int(rng.integers(1, 2000)) * S[dtype]
    share = bool(rng.integers(4) == 0) and pol["ar_mode"] != 3
    return rng, op, dtype, P, M, pol, root, chunk, share


@pytest.mark.parametrize("seed", range(48))
def test_random_configuration_matches_oracle(seed):
    rng, op, dtype, P, M, pol, root, chunk, share = _case(seed)
    s = S[dtype]
    ins_np = _inputs(P, P * M, dtype, rng)
    want = _want(op, ins_np, dtype, P, M, root)
    plans = ([PL.Plan(op, P, P * M, dtype, chunk, policy=pol, root=root, share=r) for r in range(P)] if share
             else [PL.Plan(op, P, P * M, dtype, chunk, policy=pol, root=root)])
    in_b, out_b = plans[0].in_bytes, plans[0].out_bytes
    ins = [to_device(a[: in_b // s]) for a in ins_np]
    outs = [Guarded(out_b, torch_dtype(dtype)) for _ in range(P)]
    if share and op == "allreduce":
        # a share's second phase pulls the other ranks' reduced partitions:
        # every share's first phase is run by the full plan first
        PL.Plan(op, P, P * M, dtype, chunk).exec(ins, [o.t for o in outs])
    for pl in plans:
        pl.exec(ins, [o.t for o in outs])
    torch.cuda.synchronize()
    for r in range(P):
        assert outs[r].intact(), (seed, op, r)
        if want[r] is None:
            continue
        assert_bits_equal(to_host(outs[r].t, np_dtype(dtype)), want[r], dtype,
                          f"seed {seed}: {op} {dtype} P={P} M={M} {pol} root={root} chunk={chunk} share={share} r={r}")
