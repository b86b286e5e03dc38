"""One rank's share of a collective (purlin_plan_share), on the CPU.

On P GPUs every rank pulls what it consumes (Section 3.2), so rank r runs
the descriptors that write out_r.  Checked here on host-only plans:

* a share's descriptors write out_r and nothing else, each to one
  destination;
* the P shares together write every byte of every output exactly as often
  as the full plan does (per phase);
* the shares run on the CPU interpreter, rank after rank (AllReduce: every
  share's phase 0 before any share's phase 1, as the ranks would run them),
  reproduce the oracle bit for bit;
* the buffers a share names are the ones the binding asks for;
* invalid requests are rejected.
"""

import numpy as np
import pytest

import interp
import oracle
from paper_2609_36954_amd import purlin as PL

S = {"fp32": 4, "bf16": 2}
FIXED = ("allreduce", "reduce_scatter", "allgather", "alltoall")
ROOTED = ("broadcast", "reduce", "scatter", "gather")


def _plan(op, P, count, dtype, chunk, share=None, root=None, **pol):
    return PL.Plan(op, P, count, dtype, chunk, policy=pol or None, host_only=True, root=root, share=share)


def _dsts(d, P):
    return [int(d["dst_buf"]) + j * int(d["dst_step"]) - P for j in range(int(d["ndst"]))]


def _writes(plan, P):
    """(phase, output rank, byte offset, length) of every write, sorted."""
    w = []
    for d in plan.descriptors():
        for r in _dsts(d, P):
            w.append((int(d["phase"]), r, int(d["dst_off"]), int(d["bytes"])))
    return sorted(w)


def _byte_counts(writes, P, out_bytes, phase):
    cnt = np.zeros((P, out_bytes), dtype=np.int32)
    for ph, r, off, n in writes:
        if ph == phase:
            cnt[r, off:off + n] += 1
    return cnt


SHAPE_CASES = []
for _op in FIXED + ROOTED:
    for _P, _M, _chunk in ((1, 40, 16), (2, 64, 32), (3, 100, 64), (8, 257, 96)):
        for _pol in ({}, dict(fanout=1), dict(fanout=2)):
            SHAPE_CASES.append((_op, _P, _M, _chunk, _pol))
for _P in (2, 3, 8):
    SHAPE_CASES.append(("allreduce", _P, 64, 32, dict(ar_mode=1, fanout=2)))
    SHAPE_CASES.append(("allreduce", _P, 64, 32, dict(ar_mode=2)))


@pytest.mark.parametrize("case", SHAPE_CASES, ids=lambda c: f"{c[0]}-P{c[1]}-M{c[2]}-{c[4]}")
def test_shares_partition_the_writes(case):
    op, P, M, chunk, pol = case
    roots = range(P) if op in ROOTED else [None]
    for root in roots:
        full_pol = dict(pol)
        if op == "allreduce" and "ar_mode" not in pol:
            full_pol["ar_mode"] = 1  # what a share's automatic choice is
        full = _plan(op, P, P * M, "fp32", chunk, root=root, **full_pol)
        shares = [_plan(op, P, P * M, "fp32", chunk, share=r, root=root, **pol) for r in range(P)]
        fw = _writes(full, P)
        ar_one_phase = op == "allreduce" and pol.get("ar_mode") == 2
        for r, sh in enumerate(shares):
            for d in sh.descriptors():
                assert _dsts(d, P) == [r], "a share writes only its own output, one destination per descriptor"
        if ar_one_phase:
            # every rank reduces the whole buffer into its own output
            assert all(sh.n_desc == full.n_desc for sh in shares)
        sw = sorted(w for sh in shares for w in _writes(sh, P))
        phases = sorted({w[0] for w in fw} | {w[0] for w in sw})
        for ph in phases:
            a = _byte_counts(fw, P, full.out_bytes, ph)
            b = _byte_counts(sw, P, full.out_bytes, ph)
            assert np.array_equal(a, b), (root, ph)


def test_allreduce_share_defaults_to_compose():
    P, M = 8, 1 << 14
    full = _plan("allreduce", P, P * M, "bf16", 4096)  # small: the full plan takes the one-phase form
    assert int((full.descriptors()["phase"] == 1).sum()) == 0
    sh = _plan("allreduce", P, P * M, "bf16", 4096, share=3)
    d = sh.descriptors()
    red, cp = d[d["kind"] == PL.KIND_REDUCE], d[d["kind"] == PL.KIND_COPY]
    assert set(red["part"].tolist()) == {3} and set(red["phase"].tolist()) == {0}
    assert set(cp["part"].tolist()) == set(range(P)) - {3} and set(cp["phase"].tolist()) == {1}
    # its bytes: P partitions read and one written (phase 0), P-1 read and written (phase 1)
    assert sh.sched_bytes == (P + 1 + 2 * (P - 1)) * M * 2


def _inputs(P, n, dtype, seed):
    rng = np.random.default_rng(seed)
    if dtype == "fp32":
        return [(rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32) for _ in range(P)]
    return [oracle.narrow(rng.standard_normal(n).astype(np.float32)) for _ in range(P)]


def _want(op, ins, dtype, P, M, root):
    if op == "allgather":
        return oracle.all_gather([a[:M] for a in ins], dtype)
    if op == "gather":
        return oracle.gather([a[:M] for a in ins], root, dtype)
    if op in ROOTED:
        return getattr(oracle, op)(ins, root, dtype)
    return {"allreduce": oracle.all_reduce, "reduce_scatter": oracle.reduce_scatter,
            "alltoall": oracle.all_to_all}[op](ins, dtype)


INTERP_CASES = []
for _op in FIXED + ROOTED:
    for _dt in ("fp32", "bf16"):
        for _P, _M, _ce in ((1, 37, 7), (2, 16, 1), (3, 100, 64), (8, 257, 1000)):
            INTERP_CASES.append((_op, _dt, _P, _M, _ce))


@pytest.mark.parametrize("case", INTERP_CASES, ids=lambda c: "-".join(map(str, c)))
def test_shares_rank_after_rank_match_oracle(case):
    op, dtype, P, M, ce = case
    s = S[dtype]
    ins = _inputs(P, P * M, dtype, seed=sum(map(ord, str(case))) % 997)
    for root in ([0, P - 1] if op in ROOTED else [None]):
        want = _want(op, ins, dtype, P, M, root)
        shares = [_plan(op, P, P * M, dtype, ce * s, share=r, root=root) for r in range(P)]
        in_b = shares[0].in_bytes
        bufs = [np.frombuffer(a.tobytes()[:in_b], dtype=np.uint8).copy() for a in ins]
        bufs += [np.full(shares[0].out_bytes, 0xA5, dtype=np.uint8) for _ in range(P)]
        tables = [sh.items() for sh in shares]
        for phase in (0, 1):  # what every rank does in phase 0 precedes any phase 1
            for r in reversed(range(P)):
                items, pb = tables[r]
                for i in range(pb[phase], pb[phase + 1]):
                    interp.apply_item(items[i], bufs, dtype)
        for r in range(P):
            if want[r] is None:
                assert np.all(bufs[P + r] == 0xA5)
                continue
            got = bufs[P + r].view(np.uint16 if dtype == "bf16" else np.uint32)
            exp = want[r].view(np.uint16 if dtype == "bf16" else np.uint32)
            assert np.array_equal(got, exp), (root, r)


@pytest.mark.parametrize("op", FIXED + ROOTED)
def test_share_names_only_the_buffers_it_uses(op):
    P, M = 5, 300
    for root in ([0, 3] if op in ROOTED else [None]):
        for r in range(P):
            sh = _plan(op, P, P * M, "bf16", 128, share=r, root=root)
            use_in, use_out = PL.used_buffers(sh)
            touched_in, touched_out = set(), set()
            for d in sh.descriptors():
                for j in range(int(d["nsrc"])):
                    b = int(d["src_buf"]) + j * int(d["src_step"])
                    (touched_in if b < P else touched_out).add(b % P)
                touched_out.update(_dsts(d, P))
            assert {i for i in range(P) if use_in[i]} == touched_in
            assert {i for i in range(P) if use_out[i]} == touched_out
            if sh.n_desc:
                assert use_out[r]
            if op == "allreduce":
                assert touched_out == set(range(P))  # phase 1 pulls partition k from out_k
            elif sh.n_desc:
                assert touched_out == {r}


def test_share_rejections():
    L = PL.lib()
    h = PL.ctypes.c_void_p(1)
    args = (PL.OPS["reduce_scatter"], 4, -1)
    for rank in (-1, 4):
        assert L.purlin_plan_share(*args, rank, 64, 0, 64, None, PL.PLAN_HOST_ONLY, PL.ctypes.byref(h)) == 1
        assert h.value is None
    assert L.purlin_plan_share(PL.OPS["alltoallv"], 4, -1, 0, 64, 0, 64, None, PL.PLAN_HOST_ONLY,
                               PL.ctypes.byref(h)) == 1
    assert L.purlin_plan_share(PL.OPS["broadcast"], 4, -1, 0, 64, 0, 64, None, PL.PLAN_HOST_ONLY,
                               PL.ctypes.byref(h)) == 1  # rooted op without a root
    assert L.purlin_plan_share(PL.OPS["reduce_scatter"], 4, 0, 0, 64, 0, 64, None, PL.PLAN_HOST_ONLY,
                               PL.ctypes.byref(h)) == 1  # root on a non-rooted op
    pol = PL.Policy(ar_mode=3)
    assert L.purlin_plan_share(PL.OPS["allreduce"], 4, -1, 0, 64, 0, 64, PL.ctypes.byref(pol), PL.PLAN_HOST_ONLY,
                               PL.ctypes.byref(h)) == PL.PURLIN_ERR_UNSUPPORTED
    with pytest.raises(PL.PurlinError):
        PL.Plan("alltoallv", 4, 64, "fp32", 64, unit=1, share=0, host_only=True)


PUSH_OPS = ("allgather", "alltoall", "broadcast", "scatter", "gather")


def _key(d):
    return tuple(int(d[f]) for f in ("kind", "phase", "nsrc", "src_buf", "src_step", "ndst", "dst_buf", "dst_step",
                                      "src_off", "dst_off", "bytes"))


@pytest.mark.parametrize("op", PUSH_OPS)
@pytest.mark.parametrize("P,M,pol", [(1, 40, {}), (3, 100, {"fanout": 1}), (8, 257, {"fanout": 2}), (5, 64, {})])
def test_push_shares_are_the_plan_split_by_source(op, P, M, pol):
    for root in ([0, P - 1] if op in ROOTED else [None]):
        full = _plan(op, P, P * M, "bf16", 96, root=root, **pol)
        shares = [PL.Plan(op, P, P * M, "bf16", 96, policy=pol or None, host_only=True, root=root, share=r, push=True)
                  for r in range(P)]
        for r, sh in enumerate(shares):
            use_in, _ = PL.used_buffers(sh)
            assert [i for i in range(P) if use_in[i]] == ([r] if sh.n_desc else [])
            for d in sh.descriptors():
                assert int(d["kind"]) == PL.KIND_COPY and int(d["nsrc"]) == 1 and int(d["src_buf"]) == r
        got = sorted(_key(d) for sh in shares for d in sh.descriptors())
        assert got == sorted(_key(d) for d in full.descriptors())


@pytest.mark.parametrize("case", [c for c in INTERP_CASES if c[0] in PUSH_OPS], ids=lambda c: "-".join(map(str, c)))
def test_push_shares_match_oracle(case):
    op, dtype, P, M, ce = case
    s = S[dtype]
    ins = _inputs(P, P * M, dtype, seed=sum(map(ord, str(case))) % 991)
    for root in ([0, P - 1] if op in ROOTED else [None]):
        want = _want(op, ins, dtype, P, M, root)
        shares = [PL.Plan(op, P, P * M, dtype, ce * s, host_only=True, root=root, share=r, push=True)
                  for r in range(P)]
        bufs = [np.frombuffer(a.tobytes()[:shares[0].in_bytes], dtype=np.uint8).copy() for a in ins]
        bufs += [np.full(shares[0].out_bytes, 0xA5, dtype=np.uint8) for _ in range(P)]
        for sh in reversed(shares):
            items, _ = sh.items()
            for it in items:
                interp.apply_item(it, bufs, dtype)
        for r in range(P):
            if want[r] is None:
                assert np.all(bufs[P + r] == 0xA5)
                continue
            bits = np.uint16 if dtype == "bf16" else np.uint32
            assert np.array_equal(bufs[P + r].view(bits), want[r].view(bits)), (root, r)


def test_push_share_rejections():
    L = PL.lib()
    h = PL.ctypes.c_void_p(1)
    push = PL.PLAN_HOST_ONLY | PL.PLAN_SHARE_PUSH
    for op in ("allreduce", "reduce_scatter"):
        assert L.purlin_plan_share(PL.OPS[op], 4, -1, 0, 64, 0, 64, None, push,
                                   PL.ctypes.byref(h)) == PL.PURLIN_ERR_UNSUPPORTED
    assert L.purlin_plan_share(PL.OPS["reduce"], 4, 1, 0, 64, 0, 64, None, push,
                               PL.ctypes.byref(h)) == PL.PURLIN_ERR_UNSUPPORTED
    # the push flag belongs to shares only
    assert L.purlin_plan_ex(PL.OPS["allgather"], 4, 64, 0, 64, None, push, PL.ctypes.byref(h)) == 1
    with pytest.raises(PL.PurlinError):
        PL.Plan("allgather", 4, 64, "fp32", 64, host_only=True, push=True)
