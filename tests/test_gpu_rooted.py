"""GPU parity of the rooted collectives (Appendix A) with the oracle.

Buffers a rooted plan does not use are passed as NULL (the host planner
tests show no descriptor names them); the outputs it does write carry guard
bands.
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


def run_rooted(plan, ins_np, dtype):
    s = S[dtype]
    use_in, use_out = PL.used_buffers(plan)
    ins = [to_device(a[: plan.in_bytes // s]) if u else None for a, u in zip(ins_np, use_in)]
    outs = [Guarded(plan.out_bytes, torch_dtype(dtype)) if u else None for u in use_out]
    plan.exec(ins, [o.t if o is not None else None for o in outs])
    torch.cuda.synchronize()
    got = []
    for o in outs:
        if o is None:
            got.append(None)
            continue
        assert o.intact(), "write outside an output buffer"
        got.append(to_host(o.t, np_dtype(dtype)))
    return got


CASES = []
for _op in ("broadcast", "reduce", "scatter", "gather"):
    for _dt in ("fp32", "bf16"):
        for _P, _M in ((1, 1000), (2, 16), (3, 1001), (8, 8200), (16, 520)):
            CASES.append((_op, _dt, _P, _M))


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_rooted_matches_oracle(case):
    op, dtype, P, M = case
    s = S[dtype]
    count = P * M
    ins = _inputs(P, count, dtype, seed=P * 77 + M)
    for root in sorted({0, P - 1, P // 2}):
        if op == "gather":
            want = oracle.gather([a[:M] for a in ins], root, dtype)
        else:
            want = getattr(oracle, op)(ins, root, dtype)
        for chunk in (s * 64, 1 << 20):
            plan = PL.Plan(op, P, count, dtype, chunk, root=root)
            got = run_rooted(plan, ins, dtype)
            for r in range(P):
                if want[r] is None:
                    assert got[r] is None
                else:
                    assert_bits_equal(got[r], want[r], dtype, f"{op} root={root} P={P} M={M} chunk={chunk} rank {r}")


def test_rooted_at_256MiB_per_rank():
    """Broadcast and Reduce of 256 MiB per rank, P = 8, bf16 (the streaming regime)."""
    P, N = 8, 134217728
    ins_np = [W.normal_bf16(r, N, 0.02) for r in W.rank_rngs(303, P)]
    rng = np.random.default_rng(3)
    root = 5
    ins = [to_device(a) for a in ins_np]
    red = PL.Plan("reduce", P, N, "bf16", 1 << 20, root=root)
    out = torch.empty(N, dtype=torch.int16, device="cuda")
    red.exec(ins, [out if r == root else None for r in range(P)])
    ar = PL.Plan("allreduce", P, N, "bf16", 1 << 20)
    ar_out = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    ar.exec(ins, ar_out)
    torch.cuda.synchronize()
    assert torch.equal(out, ar_out[root]), "Reduce at the root differs from the AllReduce result"
    del ar_out
    bc = PL.Plan("broadcast", P, N, "bf16", 1 << 20, root=root)
    outs = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    bc.exec([ins[r] if r == root else None for r in range(P)], outs)
    torch.cuda.synchronize()
    for r in range(P):
        assert torch.equal(outs[r], ins[root])
    idx = np.sort(rng.integers(0, N, 65536 * P))
    want = oracle.reduce([a[idx] for a in ins_np], root, "bf16")[root]
    assert_bits_equal(to_host(out, np.uint16)[idx], want, "bf16", "reduce sample")
