"""Host planner checks (CPU only: host-only plans, no device upload).

* descriptor counts of the paper-shaped configurations;
* the address rule of Listing 2 (Section 3.2): packed output at
  dst + offset, scattered / transposed output at dst + peer*partBytes + offset;
* every output byte written exactly once per phase, sources in bounds,
  AllReduce's second phase reading only what its first phase wrote;
* work items tile their descriptors exactly;
* the CPU interpreter running the table in shuffled order reproduces the
  oracle bit for bit, for every op, dtype, policy and ragged shape.
"""

import numpy as np
import pytest

import interp
import oracle
from case_seed import case_seed
from paper_2609_36954_amd import purlin as PL

S = {"fp32": 4, "bf16": 2}


def host_plan(op, P, count, dtype, chunk, **policy):
    return PL.Plan(op, P, count, dtype, chunk, policy=policy or None, host_only=True)


# ---------------------------------------------------------------------------
# descriptor counts of the configurations
# ---------------------------------------------------------------------------

COUNT_CASES = [
    # (op, P, count, dtype, chunk, policy, reduce descs, copy descs)
    ("allreduce", 4, 262144, "fp32", 16 * 1024, dict(ar_mode=1, fanout=1), 64, 192),
    ("allreduce", 8, 128 * 8192, "bf16", 64 * 1024, dict(ar_mode=1, fanout=1), 32, 224),
    ("reduce_scatter", 8, 134217728, "bf16", 1 << 20, {}, 256, 0),
    ("allgather", 8, 134217728, "bf16", 1 << 20, dict(fanout=1), 0, 2048),
    ("allgather", 8, 134217728, "bf16", 1 << 20, dict(fanout=2), 0, 256),
    ("allreduce", 8, 134217728, "bf16", 1 << 20, dict(ar_mode=1, fanout=1), 256, 1792),
    ("allreduce", 8, 134217728, "bf16", 1 << 20, dict(ar_mode=2), 256, 0),
    ("alltoall", 8, 134217728, "bf16", 1 << 20, {}, 0, 2048),
]


@pytest.mark.parametrize("case", COUNT_CASES, ids=lambda c: f"{c[0]}-P{c[1]}-{c[3]}-{c[5]}")
def test_descriptor_counts(case):
    op, P, count, dtype, chunk, pol, n_red, n_copy = case
    d = host_plan(op, P, count, dtype, chunk, **pol).descriptors()
    assert int((d["kind"] == PL.KIND_REDUCE).sum()) == n_red
    assert int((d["kind"] == PL.KIND_COPY).sum()) == n_copy


@pytest.mark.parametrize(
    "op,P,count,dtype,pol,want",
    [
        # AllReduce in two phases moves (3P-1)*N*s bytes; in one phase 2P*N*s
        ("allreduce", 4, 262144, "fp32", dict(ar_mode=1, fanout=1), (3 * 4 - 1) * 262144 * 4),
        ("allreduce", 8, 1 << 20, "bf16", dict(ar_mode=1, fanout=1), (3 * 8 - 1) * (1 << 20) * 2),
        # two phases with multi-destination copies: phase 1 reads each reduced
        # chunk once per destination run (two runs, r < k and r > k, except
        # at the ends): (P+1)*N*s + (P-1)*N*s + (2P-2)/P*N*s
        ("allreduce", 8, 1 << 20, "bf16", dict(ar_mode=1, fanout=2), (9 + 7) * (1 << 21) + 14 * (1 << 21) // 8),
        ("allreduce", 8, 1 << 20, "bf16", dict(ar_mode=2), 2 * 8 * (1 << 20) * 2),
        # ReduceScatter (P+1)*N*s; AllGather with one read per source chunk (P+1)*N*s
        ("reduce_scatter", 8, 1 << 20, "bf16", {}, 9 * (1 << 20) * 2),
        ("allgather", 8, 1 << 20, "bf16", dict(fanout=2), 9 * (1 << 20) * 2),
        ("allgather", 8, 1 << 20, "bf16", dict(fanout=1), 16 * (1 << 20) * 2),
        ("alltoall", 8, 1 << 20, "bf16", {}, 2 * 8 * (1 << 20) * 2),
    ],
)
def test_scheduled_bytes(op, P, count, dtype, pol, want):
    assert host_plan(op, P, count, dtype, 65536, **pol).sched_bytes == want


# ---------------------------------------------------------------------------
# structure of the table
# ---------------------------------------------------------------------------

STRUCT_CASES = [
    ("reduce_scatter", 3, 3 * 1000, "bf16", 256, {}),
    ("reduce_scatter", 8, 8 * 4096, "fp32", 4096, {}),
    ("allgather", 5, 5 * 999, "bf16", 100, dict(fanout=1)),
    ("allgather", 5, 5 * 999, "bf16", 100, dict(fanout=2)),
    ("alltoall", 4, 4 * 777, "fp32", 64, {}),
    ("allreduce", 4, 4 * 1000, "fp32", 160, dict(ar_mode=1, fanout=1)),
    ("allreduce", 6, 6 * 1000, "bf16", 160, dict(ar_mode=1, fanout=2)),
    ("allreduce", 7, 7 * 500, "bf16", 96, dict(ar_mode=2)),
    ("allreduce", 1, 100, "bf16", 32, dict(ar_mode=1)),
    ("allreduce", 16, 16 * 64, "bf16", 2, dict(ar_mode=1, fanout=2)),
]


def _intervals_cover_once(ivals, total):
    ivals = sorted(ivals)
    pos = 0
    for lo, hi in ivals:
        if lo != pos:
            return False
        pos = hi
    return pos == total


@pytest.mark.parametrize("case", STRUCT_CASES, ids=lambda c: f"{c[0]}-P{c[1]}-{c[3]}-{c[5]}")
def test_table_structure(case):
    op, P, count, dtype, chunk, pol = case
    plan = host_plan(op, P, count, dtype, chunk, **pol)
    s = S[dtype]
    M = count // P
    part = M * s
    d = plan.descriptors()
    assert plan.n_desc == len(d)
    assert plan.sched_bytes == int(sum((int(x["nsrc"]) + int(x["ndst"])) * int(x["bytes"]) for x in d))

    writes = {}  # (phase, buffer) -> list of intervals
    for x in d:
        ph, n = int(x["phase"]), int(x["bytes"])
        assert n > 0 and n % s == 0
        assert n <= chunk
        c, k = int(x["chunk"]), int(x["part"])
        off = c * chunk  # offset of the chunk inside its partition
        # Listing 2 address rule
        for j in range(int(x["ndst"])):
            b = int(x["dst_buf"]) + j * int(x["dst_step"])
            assert P <= b < 2 * P
            r = b - P
            if op == "reduce_scatter":  # packed output
                assert int(x["dst_off"]) == off and k == r
            elif op == "allgather":  # scattered output, peer = k
                assert int(x["dst_off"]) == k * part + off
            elif op == "alltoall":  # transposed output, peer = source rank
                p = int(x["src_buf"])
                assert int(x["dst_off"]) == p * part + off and k == r
            else:  # allreduce: scattered output, partition k
                assert int(x["dst_off"]) == k * part + off
            writes.setdefault((ph, b), []).append((int(x["dst_off"]), int(x["dst_off"]) + n))
        # sources
        for p in range(int(x["nsrc"])):
            b = int(x["src_buf"]) + p * int(x["src_step"])
            lim = plan.in_bytes if b < P else plan.out_bytes
            assert int(x["src_off"]) + n <= lim
            if ph == 0:
                assert b < P, "phase 0 reads inputs only"
        if int(x["kind"]) == PL.KIND_REDUCE:
            assert int(x["nsrc"]) == P and int(x["src_buf"]) == 0 and int(x["src_step"]) == 1
        else:
            assert int(x["nsrc"]) == 1

    # exactly-once coverage
    if op == "allreduce" and plan.descriptors()["phase"].max() == 1:
        for r in range(P):
            w0 = writes.get((0, P + r), [])
            assert _intervals_cover_once(w0 and [(a - r * part, b - r * part) for a, b in w0], part)
            w1 = writes.get((1, P + r), [])
            full = sorted(w0 + w1)
            assert _intervals_cover_once(full, plan.out_bytes)
        # phase 1 reads out_k's partition k only (written in phase 0)
        for x in d[d["phase"] == 1]:
            k = int(x["src_buf"]) - P
            assert k * part <= int(x["src_off"]) and int(x["src_off"]) + int(x["bytes"]) <= (k + 1) * part
    else:
        for r in range(P):
            assert _intervals_cover_once(writes.get((0, P + r), []), plan.out_bytes)


@pytest.mark.parametrize("case", STRUCT_CASES, ids=lambda c: f"{c[0]}-P{c[1]}-{c[3]}-{c[5]}")
@pytest.mark.parametrize("item_bytes", [0, 16, 48, 1024])
def test_items_tile_descriptors(case, item_bytes):
    op, P, count, dtype, chunk, pol = case
    plan = host_plan(op, P, count, dtype, chunk, item_bytes=item_bytes, **pol)
    d = plan.descriptors()
    items, pb = plan.items()
    assert pb[0] == 0 and pb[2] == len(items) and pb[0] <= pb[1] <= pb[2]
    assert np.all(items["phase"][: pb[1]] == 0) and np.all(items["phase"][pb[1]:] == 1)
    if item_bytes:
        assert int(items["bytes"].max()) <= item_bytes
    # walk items in order; they must cut each descriptor into consecutive pieces
    i = 0
    for x in d:
        covered = 0
        while covered < int(x["bytes"]):
            it = items[i]
            for f in ("kind", "phase", "nsrc", "src_buf", "src_step", "ndst", "dst_buf", "dst_step", "part", "chunk"):
                assert it[f] == x[f]
            assert int(it["src_off"]) == int(x["src_off"]) + covered
            assert int(it["dst_off"]) == int(x["dst_off"]) + covered
            covered += int(it["bytes"])
            i += 1
        assert covered == int(x["bytes"])
    assert i == len(items)
    # a phase holds one consume op (one kernel per phase)
    for lo, hi in ((pb[0], pb[1]), (pb[1], pb[2])):
        assert len(set(items["kind"][lo:hi].tolist())) <= 1


# ---------------------------------------------------------------------------
# the table, run on the CPU in shuffled order, equals the oracle
# ---------------------------------------------------------------------------


def _inputs(P, n, dtype, seed):
    rng = np.random.default_rng(seed)
    if dtype == "fp32":
        return [(rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32) for _ in range(P)]
    return [oracle.narrow(rng.standard_normal(n).astype(np.float32)) for _ in range(P)]


def _oracle(op, ins, dtype):
    if op == "allgather":
        M = len(ins[0]) // len(ins)
        return oracle.all_gather([a[:M] for a in ins], dtype)
    return {"allreduce": oracle.all_reduce, "reduce_scatter": oracle.reduce_scatter, "alltoall": oracle.all_to_all}[op](
        ins, dtype
    )


INTERP_CASES = []
for _op in ("allreduce", "reduce_scatter", "allgather", "alltoall"):
    for _dt in ("fp32", "bf16"):
        for _P, _M in ((1, 37), (2, 16), (3, 100), (4, 256), (8, 257), (16, 9)):
            for _chunk_elems in (1, 7, 64, 1000):
                INTERP_CASES.append((_op, _dt, _P, _M, _chunk_elems))


@pytest.mark.parametrize("case", INTERP_CASES, ids=lambda c: "-".join(map(str, c)))
def test_interpreter_matches_oracle(case):
    op, dtype, P, M, chunk_elems = case
    s = S[dtype]
    count = P * M
    ins = _inputs(P, count, dtype, seed=case_seed(case) % 1000)
    want = _oracle(op, ins, dtype)
    policies = [{}]
    if op == "allreduce":
        policies = [dict(ar_mode=1, fanout=1), dict(ar_mode=1, fanout=2), dict(ar_mode=2, item_bytes=32)]
    elif op == "allgather":
        policies = [dict(fanout=1, item_bytes=48), dict(fanout=2)]
    for pol in policies:
        plan = host_plan(op, P, count, dtype, chunk_elems * s, **pol)
        items, pb = plan.items()
        in_bytes = [np.frombuffer(a.tobytes()[: plan.in_bytes], dtype=np.uint8).copy() for a in ins]
        outs = [np.full(plan.out_bytes, 0xA5, dtype=np.uint8) for _ in range(P)]
        interp.run(items, pb, in_bytes + outs, dtype, seed=len(items))
        for r in range(P):
            got = outs[r].view(np.uint16 if dtype == "bf16" else np.uint32)
            exp = want[r].view(np.uint16 if dtype == "bf16" else np.uint32)
            assert np.array_equal(got, exp), (pol, r)


# ---------------------------------------------------------------------------
# rooted collectives (Appendix A)
# ---------------------------------------------------------------------------

ROOTED_CASES = []
for _op in ("broadcast", "reduce", "scatter", "gather"):
    for _dt in ("fp32", "bf16"):
        for _P, _M in ((1, 9), (2, 16), (3, 100), (8, 257)):
            for _chunk_elems in (1, 64, 1000):
                ROOTED_CASES.append((_op, _dt, _P, _M, _chunk_elems))


@pytest.mark.parametrize("case", ROOTED_CASES, ids=lambda c: "-".join(map(str, c)))
def test_rooted_interpreter_matches_oracle(case):
    op, dtype, P, M, chunk_elems = case
    s = S[dtype]
    count = P * M
    ins = _inputs(P, count, dtype, seed=case_seed(case) % 1000)
    for root in sorted({0, P - 1, P // 2}):
        if op == "gather":
            want = oracle.gather([a[:M] for a in ins], root, dtype)
        else:
            want = getattr(oracle, op)(ins, root, dtype)
        plan = PL.Plan(op, P, count, dtype, chunk_elems * s, host_only=True, root=root)
        use_in, use_out = PL.used_buffers(plan)
        items, pb = plan.items()
        # buffers a rooted plan does not use are poisoned: reading them would show
        in_bytes = [np.frombuffer(a.tobytes()[: plan.in_bytes], dtype=np.uint8).copy() if u
                    else np.full(plan.in_bytes, 0xEE, np.uint8) for a, u in zip(ins, use_in)]
        outs = [np.full(plan.out_bytes, 0xA5, dtype=np.uint8) for _ in range(P)]
        interp.run(items, pb, in_bytes + outs, dtype, seed=len(items))
        for r in range(P):
            if not use_out[r]:
                assert want[r] is None
                assert np.all(outs[r] == 0xA5), "a buffer the plan does not use was written"
                continue
            got = outs[r].view(np.uint16 if dtype == "bf16" else np.uint32)
            exp = want[r].view(np.uint16 if dtype == "bf16" else np.uint32)
            assert np.array_equal(got, exp), (op, root, r)


@pytest.mark.parametrize("op", ["broadcast", "reduce", "scatter", "gather"])
def test_rooted_tables_touch_only_used_buffers(op):
    P, M = 6, 1000
    for root in range(P):
        plan = host_plan_rooted(op, P, P * M, "bf16", 256, root)
        use_in, use_out = PL.used_buffers(plan)
        d = plan.descriptors()
        for x in d:
            for p in range(int(x["nsrc"])):
                b = int(x["src_buf"]) + p * int(x["src_step"])
                assert b < P and use_in[b]
            for j in range(int(x["ndst"])):
                b = int(x["dst_buf"]) + j * int(x["dst_step"]) - P
                assert 0 <= b < P and use_out[b]
        expected = {"broadcast": P * 8, "reduce": P * 8, "scatter": P * 8, "gather": P * 8}[op]
        assert len(d) == expected  # one descriptor per (partition, chunk): 2000 B / 256 B = 8 chunks


def host_plan_rooted(op, P, count, dtype, chunk, root, **policy):
    return PL.Plan(op, P, count, dtype, chunk, policy=policy or None, host_only=True, root=root)


# ---------------------------------------------------------------------------
# single-launch AllReduce (ar_mode 3): the claim order is a valid schedule
# ---------------------------------------------------------------------------

FUSED_CASES = [(P, M, dt, ce, it) for P in (2, 3, 8, 16) for M in (16, 1000, 4099)
               for dt in ("fp32", "bf16") for ce in (1, 100, 4096) for it in (0, 32)]


@pytest.mark.parametrize("case", FUSED_CASES, ids=lambda c: "-".join(map(str, c)))
def test_fused_allreduce_claim_order(case):
    """Waves claim items in table order.  Every copy item must find all
    reduce items of its chunk already claimed (they never wait), the number
    of reduce items per chunk must be what the kernel computes from
    (partBytes, chunk, item size), and running the items in claim order
    must reproduce the oracle."""
    P, M, dtype, chunk_elems, item = case
    s = S[dtype]
    chunk = chunk_elems * s
    plan = host_plan("allreduce", P, P * M, dtype, chunk, ar_mode=3, fanout=2, item_bytes=item)
    items, pb = plan.items()
    part = M * s
    reduce_item = int(items["bytes"][: pb[1]].max())  # the reduce items' cut size (the last of a chunk may be shorter)
    if item:
        assert reduce_item <= item
    claimed = {}
    for i, it in enumerate(items):
        key = (int(it["part"]), int(it["chunk"]))
        if it["kind"] == PL.KIND_REDUCE:
            assert i < pb[1]
            claimed[key] = claimed.get(key, 0) + 1
        else:
            assert i >= pb[1]
            off = int(it["chunk"]) * chunk
            length = min(chunk, part - off)
            cut = item if item else None
            if cut:
                assert claimed.get(key, 0) == -(-length // cut), "copy claimed before its chunk's reductions"
            else:
                assert claimed.get(key, 0) >= 1
    ins = _inputs(P, P * M, dtype, seed=P + M)
    want = oracle.all_reduce(ins, dtype)
    bufs = [np.frombuffer(a.tobytes(), np.uint8).copy() for a in ins] + [np.zeros(plan.out_bytes, np.uint8) for _ in range(P)]
    for it in items:  # claim order
        interp.apply_item(it, bufs, dtype)
    for r in range(P):
        got = bufs[P + r].view(np.uint16 if dtype == "bf16" else np.uint32)
        assert np.array_equal(got, want[r].view(got.dtype))


def _partition_of(i):
    """The kernel's partition of item (or wave) i: its workgroup of 4 waves, mod 8."""
    return (i // 4) % 8


@pytest.mark.parametrize("n", [1, 3, 4, 5, 31, 32, 33, 64, 100, 1000, 4099])
def test_fused_partition_sizes_and_ticket_to_item_map(n):
    """Partition k holds nk = 4 * (n // 32) + min(max(n % 32 - 4k, 0), 4)
    items, as many as it has waves, and the j-th ticket of partition k names
    its j-th item in table order: ((j // 4) * 8 + k) * 4 + j % 4."""
    for k in range(8):
        items = [i for i in range(n) if _partition_of(i) == k]
        nk = 4 * (n // 32) + min(max(n % 32 - 4 * k, 0), 4)
        assert len(items) == nk
        assert [((j // 4) * 8 + k) * 4 + j % 4 for j in range(nk)] == items


@pytest.mark.parametrize("case", FUSED_CASES[::3], ids=lambda c: "-".join(map(str, c)))
def test_fused_allreduce_partitioned_claims_never_deadlock(case):
    """The waves of each of the 8 partitions claim that partition's items in
    table order.  Run the partitions round-robin, a copy item blocking its
    partition until every reduce item of its chunk has run: some partition
    can always move (no deadlock), and the result is the oracle's."""
    P, M, dtype, chunk_elems, item = case
    s = S[dtype]
    plan = host_plan("allreduce", P, P * M, dtype, chunk_elems * s, ar_mode=3, fanout=2, item_bytes=item)
    items, pb = plan.items()
    n, n_reduce = len(items), int(pb[1])
    need = {}
    for it in items[:n_reduce]:
        key = (int(it["part"]), int(it["chunk"]))
        need[key] = need.get(key, 0) + 1
    queues = [[i for i in range(n) if _partition_of(i) == k] for k in range(8)]
    for q in queues:  # within a partition every reduce item precedes every copy item
        kinds = [int(items[i]["kind"]) for i in q]
        assert kinds == sorted(kinds, key=lambda kd: kd != PL.KIND_REDUCE)
    ins = _inputs(P, P * M, dtype, seed=P + M + 1)
    want = oracle.all_reduce(ins, dtype)
    bufs = [np.frombuffer(a.tobytes(), np.uint8).copy() for a in ins] + [np.zeros(plan.out_bytes, np.uint8) for _ in range(P)]
    done = {}
    heads = [0] * 8
    while any(heads[k] < len(queues[k]) for k in range(8)):
        moved = False
        for k in range(8):
            if heads[k] == len(queues[k]):
                continue
            it = items[queues[k][heads[k]]]
            key = (int(it["part"]), int(it["chunk"]))
            if it["kind"] != PL.KIND_REDUCE and done.get(key, 0) < need[key]:
                continue  # waits for its chunk
            interp.apply_item(it, bufs, dtype)
            if it["kind"] == PL.KIND_REDUCE:
                done[key] = done.get(key, 0) + 1
            heads[k] += 1
            moved = True
        assert moved, "every partition waits"
    for r in range(P):
        got = bufs[P + r].view(np.uint16 if dtype == "bf16" else np.uint32)
        assert np.array_equal(got, want[r].view(got.dtype))


# ---------------------------------------------------------------------------
# automatic work-item sizes by regime (P = 8, bf16, chunk 1 MiB)
# ---------------------------------------------------------------------------

MiB = 1 << 20


@pytest.mark.parametrize("op,mib_per_rank,want", [
    ("reduce_scatter", 256, 4096),     # 8-way reduce: 32 KiB read per item
    ("reduce_scatter", 1024, 4096),
    ("allgather", 256, 32 * 1024),     # one read, 8 writes per item; 2.25 GiB moved
    ("allgather", 512, 2048),          # 4.5 GiB moved: the large-copy size
    ("alltoall", 16, 4096),            # one-to-one below the streaming threshold: still 4 KiB
    ("allgather", 32, 8192),           # multi-destination below it: 32 MiB of items / 4096
    ("alltoall", 128, 4096),           # one-to-one, 2 GiB moved
    ("alltoall", 256, 2048),           # 4 GiB moved
])
def test_automatic_item_size(op, mib_per_rank, want):
    N = mib_per_rank * MiB // 2
    items, _ = PL.Plan(op, 8, N, "bf16", MiB, host_only=True).items()
    assert int(items["bytes"].max()) == want


@pytest.mark.parametrize("op", ["alltoallv", "allgatherv"])
def test_variable_size_plans_keep_the_streaming_item_size(op):
    # the same traffic as the fixed-size AllToAll at 256 MiB/rank, but the
    # waves of a variable-size launch also map items onto run-time sizes
    N = 256 * MiB // 2
    items, _ = PL.Plan(op, 8, N, "bf16", MiB, unit=1, host_only=True).items()
    assert int(items["bytes"].max()) > 2048


@pytest.mark.parametrize("P,mib_per_rank,dtype,two_phase", [
    (8, 48, "bf16", False),   # one-phase traffic 768 MiB: reduce once, write all 8 outputs
    (8, 64, "bf16", True),    # 1 GiB: compose<RS, AG> in two launches
    (8, 256, "bf16", True),   # the reduced 256 MiB still fits the last-level cache
    (8, 512, "bf16", False),  # it no longer does: phase 1 would read it from HBM
    (4, 1, "fp32", False),    # the small fp32 AllReduce
    (8, 2, "bf16", False),    # the decode AllReduce
])
def test_automatic_allreduce_mode(P, mib_per_rank, dtype, two_phase):
    """Two launches (compose<RS, AG>) from 1 GiB of one-phase traffic while
    the reduced buffer fits the 256 MB last-level cache; otherwise one."""
    s = S[dtype]
    N = mib_per_rank * MiB // s
    items, pb = PL.Plan("allreduce", P, N, dtype, MiB, host_only=True).items()
    assert (pb[1] < pb[2]) == two_phase
    phase0 = items[:pb[1]]
    assert np.all(phase0["kind"] == PL.KIND_REDUCE)
    assert np.all(phase0["ndst"] == (1 if two_phase else P))
