"""GPU parity of the collective executor (purlin_plan / purlin_exec) with the oracle.

Bit-exact for every op and dtype: copies are bit copies and every reduction
follows Eq. 2 (rank order, FP32, one rounding back to bf16) on both sides.
Outputs carry guard bands that must come back untouched.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import Guarded, assert_bits_equal, np_dtype, to_device, to_host, torch_dtype
from paper_2609_36954_amd import purlin as PL
from paper_2609_36954_amd import workloads as W

pytestmark = pytest.mark.gpu

S = {"fp32": 4, "bf16": 2}


def _inputs(P, n, dtype, seed):
    rng = np.random.default_rng(seed)
    if dtype == "fp32":
        return [(rng.standard_normal(n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32) for _ in range(P)]
    return [oracle.narrow(rng.standard_normal(n).astype(np.float32)) for _ in range(P)]


def _oracle(op, ins, dtype):
    if op == "allgather":
        M = len(ins[0]) // len(ins)
        return oracle.all_gather([a[:M] for a in ins], dtype)
    fn = {"allreduce": oracle.all_reduce, "reduce_scatter": oracle.reduce_scatter, "alltoall": oracle.all_to_all}[op]
    return fn(ins, dtype)


def run_plan(plan, ins_np, dtype):
    """Upload inputs (trimmed to the plan's input size), run, return outputs."""
    s = S[dtype]
    ins = [to_device(a[: plan.in_bytes // s]) for a in ins_np]
    outs = [Guarded(plan.out_bytes, torch_dtype(dtype)) for _ in range(plan.P)]
    plan.exec(ins, [o.t for o in outs])
    torch.cuda.synchronize()
    for o in outs:
        assert o.intact(), "write outside an output buffer"
    return [to_host(o.t, np_dtype(dtype)) for o in outs]


CASES = []
for _op in ("allreduce", "reduce_scatter", "allgather", "alltoall"):
    for _dt in ("fp32", "bf16"):
        for _P, _M in ((1, 1000), (2, 16), (3, 1001), (4, 4096), (5, 777), (8, 8200), (16, 520)):
            CASES.append((_op, _dt, _P, _M))


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(map(str, c)))
def test_exec_matches_oracle(case):
    op, dtype, P, M = case
    s = S[dtype]
    count = P * M
    ins = _inputs(P, count, dtype, seed=P * 1000 + M)
    want = _oracle(op, ins, dtype)
    policies = [None]
    if op == "allreduce":
        policies = [None, dict(ar_mode=1, fanout=1), dict(ar_mode=1, fanout=2)]
    elif op == "allgather":
        policies = [None, dict(fanout=1)]
    for chunk in (s * 64, 4096, 1 << 20):
        for pol in policies:
            plan = PL.Plan(op, P, count, dtype, chunk, policy=pol)
            got = run_plan(plan, ins, dtype)
            for r in range(P):
                assert_bits_equal(got[r], want[r], dtype, f"{op} P={P} M={M} chunk={chunk} {pol} rank {r}")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("item_bytes", [16, 48, 1024, 65536])
def test_result_does_not_depend_on_chunk_or_item(dtype, item_bytes):
    P, M = 8, 3000
    ins = _inputs(P, P * M, dtype, seed=7)
    want = oracle.all_reduce(ins, dtype)
    s = S[dtype]
    for chunk in (s, 6 * s, 1000 * s, M * s):
        for mode in (1, 2):
            plan = PL.Plan("allreduce", P, P * M, dtype, chunk, policy=dict(item_bytes=item_bytes, ar_mode=mode))
            got = run_plan(plan, ins, dtype)
            for r in range(P):
                assert_bits_equal(got[r], want[r], dtype, f"chunk={chunk} item={item_bytes} mode={mode}")


def test_repeated_runs_are_bit_identical():
    P, M = 8, 1 << 16
    ins = _inputs(P, P * M, "bf16", seed=3)
    plan = PL.Plan("allreduce", P, P * M, "bf16", 65536)
    first = run_plan(plan, ins, "bf16")
    for _ in range(4):
        again = run_plan(plan, ins, "bf16")
        for a, b in zip(first, again):
            assert np.array_equal(a, b)


def test_rank_order_on_device():
    """[2**24, 1, -2**24] in rank order is 0 on the GPU too (no tree, no reassociation)."""
    n = 3 * 64
    ins = [np.full(n, v, np.float32) for v in (2.0**24, 1.0, -(2.0**24))]
    for mode in (1, 2):
        plan = PL.Plan("allreduce", 3, n, "fp32", 64, policy=dict(ar_mode=mode))
        for out in run_plan(plan, ins, "fp32"):
            assert np.all(out == 0.0)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_special_values(dtype):
    """Signed zeros, denormals, infinities, NaN and overflow, against the oracle."""
    P, n = 4, 4 * 64
    if dtype == "fp32":
        vals = np.array([-0.0, 2.0**-140, -(2.0**-149), np.inf, -np.inf, 3.0e38, 1.0, -1.0], np.float32)
    else:
        vals = np.array([0x8000, 0x0001, 0x8001, 0x7F80, 0xFF80, 0x7F7F, 0x3F80, 0xBF80], np.uint16)
    rng = np.random.default_rng(5)
    ins = [vals[rng.integers(0, len(vals), n)] for _ in range(P)]
    ins[0][:8] = vals  # make sure each value shows up
    want = oracle.all_reduce(ins, dtype)
    plan = PL.Plan("allreduce", P, n, dtype, 128)
    got = run_plan(plan, ins, dtype)
    f = (lambda a: a) if dtype == "fp32" else oracle.widen
    for g, w in zip(got, want):
        nan_g, nan_w = np.isnan(f(g)), np.isnan(f(w))
        assert np.array_equal(nan_g, nan_w), "NaN positions differ"
        assert_bits_equal(g[~nan_w], w[~nan_w], dtype, "special values")
    # all -0 sums to +0
    zero = [np.full(n, vals[0]) for _ in range(P)]
    for out in run_plan(plan, zero, dtype):
        assert np.all((out.view(np.uint32) if dtype == "fp32" else out) == 0)


def test_rejects_bad_buffers_before_enqueueing():
    plan = PL.Plan("allreduce", 2, 1024, "bf16", 256)
    a = torch.zeros(4096, dtype=torch.int16, device="cuda")
    L = PL.lib()
    base = a.data_ptr()

    def call(ptrs):
        arr = (PL.ctypes.c_void_p * 4)(*ptrs)
        return L.purlin_exec(plan.handle, arr, None)

    nb = 1024 * 2
    assert call([base, base + nb, base + 2 * nb, base + 3 * nb]) == 0
    torch.cuda.synchronize()
    assert call([base + 2, base + nb, base + 2 * nb, base + 3 * nb]) == PL.PURLIN_ERR_INVALID  # misaligned
    assert call([base, base + nb, base + nb, base + 3 * nb]) == PL.PURLIN_ERR_INVALID  # input overlaps output
    assert call([base, base + nb, base + 2 * nb, base + 2 * nb + 16]) == PL.PURLIN_ERR_INVALID  # outputs overlap
    assert call([base, 0, base + 2 * nb, base + 3 * nb]) == PL.PURLIN_ERR_INVALID  # null
    assert call([base, base, base + 2 * nb, base + 3 * nb]) == 0  # inputs may alias
    torch.cuda.synchronize()


def test_graph_capture_replays_match_eager():
    P, M = 8, 1 << 14
    ins_np = _inputs(P, P * M, "bf16", seed=11)
    plan = PL.Plan("allreduce", P, P * M, "bf16", 65536)
    ins = [to_device(a) for a in ins_np]
    outs = [torch.empty(P * M, dtype=torch.int16, device="cuda") for _ in range(P)]
    plan.exec(ins, outs)
    torch.cuda.synchronize()
    eager = [o.clone() for o in outs]
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        for o in outs:
            o.zero_()
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            plan.exec(ins, outs, stream=side)
    for _ in range(3):
        for o in outs:
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs, eager):
            assert torch.equal(o, e)


# ---------------------------------------------------------------------------
# full-size configurations
# ---------------------------------------------------------------------------


def test_allreduce_p4_fp32_262144_per_rank():
    cfg = W.AR_P4_FP32_256K
    ins = W.collective_inputs(cfg)
    want = oracle.all_reduce(ins, cfg.dtype)
    plan = PL.Plan(cfg.op, cfg.P, cfg.count, cfg.dtype, cfg.chunk)
    got = run_plan(plan, ins, cfg.dtype)
    for r in range(cfg.P):
        assert_bits_equal(got[r], want[r], "fp32", f"AllReduce P=4 fp32 rank {r}")


def test_decode_allreduce_p8_bf16_128x8192():
    cfg = W.AR_P8_BF16_DECODE
    ins = W.collective_inputs(cfg)
    want = oracle.all_reduce(ins, cfg.dtype)
    for pol in (None, dict(ar_mode=1)):
        plan = PL.Plan(cfg.op, cfg.P, cfg.count, cfg.dtype, cfg.chunk, policy=pol)
        got = run_plan(plan, ins, cfg.dtype)
        for r in range(cfg.P):
            assert_bits_equal(got[r], want[r], "bf16", f"decode AllReduce rank {r} {pol}")


def test_reduce_scatter_then_all_gather_256MiB_per_rank():
    """256 MiB per rank, P=8, bf16, chunk 1 MiB, in the launch shapes the bench times.

    Every ReduceScatter output (8 x 32 MiB) and every AllGather output
    (8 x 256 MiB) is compared with the oracle bit for bit over the whole
    buffer, and so is the AllReduce output of every rank; RS then AG must
    also equal the AllReduce on the device.
    """
    cfg = W.RS_AG_P8_BF16_256MIB
    P, N = cfg.P, cfg.count
    M = N // P
    ins_np = W.collective_inputs(cfg)
    ins = [to_device(a) for a in ins_np]
    rs = PL.Plan("reduce_scatter", P, N, "bf16", cfg.chunk)
    ag = PL.Plan("allgather", P, N, "bf16", cfg.chunk)
    ar = PL.Plan("allreduce", P, N, "bf16", cfg.chunk)
    rs_out = [torch.empty(M, dtype=torch.int16, device="cuda") for _ in range(P)]
    ag_out = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    rs.exec(ins, rs_out)
    ag.exec(rs_out, ag_out)
    ar_out = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    ar.exec(ins, ar_out)
    torch.cuda.synchronize()
    for r in range(P):
        assert torch.equal(ag_out[r], ar_out[r]), f"RS then AG differs from AR at rank {r}"
    del ins
    want_rs = oracle.reduce_scatter(ins_np, "bf16")
    for r in range(P):
        assert_bits_equal(to_host(rs_out[r], np.uint16), want_rs[r], "bf16", f"ReduceScatter rank {r}, 256 MiB/rank")
    want_ag = oracle.all_gather(want_rs, "bf16")
    for r in range(P):
        assert_bits_equal(to_host(ag_out[r], np.uint16), want_ag[r], "bf16", f"AllGather rank {r}, 256 MiB/rank")
    del ag_out, want_ag
    want_ar = oracle.all_reduce(ins_np, "bf16")
    for r in range(P):
        assert_bits_equal(to_host(ar_out[r], np.uint16), want_ar[r], "bf16", f"AllReduce rank {r}, 256 MiB/rank")


# ---------------------------------------------------------------------------
# single-launch AllReduce (ar_mode 3): per-chunk counters with epochs
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P,M", [(2, 16), (3, 1001), (8, 8200), (16, 520)])
def test_fused_allreduce_matches_oracle(dtype, P, M):
    s = S[dtype]
    ins = _inputs(P, P * M, dtype, seed=900 + P)
    want = oracle.all_reduce(ins, dtype)
    for chunk in (s * 64, 4096, 1 << 20):
        for pol in (dict(ar_mode=3), dict(ar_mode=3, fanout=1, item_bytes=256)):
            plan = PL.Plan("allreduce", P, P * M, dtype, chunk, policy=pol)
            for rep in range(3):  # the epoch advances on every launch
                got = run_plan(plan, ins, dtype)
                for r in range(P):
                    assert_bits_equal(got[r], want[r], dtype, f"fused P={P} M={M} chunk={chunk} {pol} rep={rep}")
            assert plan.device_error() == 0


def test_fused_allreduce_graph_replays():
    P, M = 8, 1 << 14
    ins_np = _inputs(P, P * M, "bf16", seed=12)
    want = oracle.all_reduce(ins_np, "bf16")
    plan = PL.Plan("allreduce", P, P * M, "bf16", 65536, policy=dict(ar_mode=3))
    ins = [to_device(a) for a in ins_np]
    outs = [torch.empty(P * M, dtype=torch.int16, device="cuda") for _ in range(P)]
    plan.exec(ins, outs)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            for _ in range(4):
                plan.exec(ins, outs, stream=side)
    for _ in range(3):
        for o in outs:
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for r in range(P):
            assert_bits_equal(to_host(outs[r], np.uint16), want[r], "bf16", "fused AR graph replay")
    assert plan.device_error() == 0


def test_fused_allreduce_full_size_equals_two_launches():
    cfg = W.RS_AG_P8_BF16_256MIB
    P, N = cfg.P, cfg.count
    ins = [to_device(a) for a in W.collective_inputs(cfg)]
    fused = PL.Plan("allreduce", P, N, "bf16", cfg.chunk, policy=dict(ar_mode=3))
    two = PL.Plan("allreduce", P, N, "bf16", cfg.chunk, policy=dict(ar_mode=1))
    a = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    fused.exec(ins, a)
    fused.exec(ins, a)
    torch.cuda.synchronize()
    b = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    two.exec(ins, b)
    torch.cuda.synchronize()
    for r in range(P):
        assert torch.equal(a[r], b[r])
    assert fused.device_error() == 0


def test_offsets_beyond_4GiB_per_rank():
    """P = 2 AllReduce of 5 GiB per rank: byte offsets above 2^32 in every
    buffer.  Inputs are drawn on the device with a seeded torch generator;
    sampled elements are checked against the oracle, and RS then AG must equal
    the AllReduce bit for bit."""
    P, N = 2, (5 << 30) // 2
    g = torch.Generator(device="cuda").manual_seed(55)
    ins = [torch.randn(N, device="cuda", generator=g).to(torch.bfloat16).view(torch.int16) for _ in range(P)]
    ar = PL.Plan("allreduce", P, N, "bf16", 1 << 20)
    outs = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    ar.exec(ins, outs)
    torch.cuda.synchronize()
    rng = np.random.default_rng(56)
    idx = np.sort(np.concatenate([rng.integers(0, N, 65536), np.arange(N - 4096, N)]))
    idx_t = torch.from_numpy(idx).to("cuda")
    sample = [to_host(t[idx_t], np.uint16) for t in ins]
    want = oracle.all_reduce([s[: len(s) // P * P] for s in sample], "bf16")[0]
    assert_bits_equal(to_host(outs[0][idx_t], np.uint16)[: len(want)], want, "bf16", "AR beyond 4 GiB")
    assert torch.equal(outs[0], outs[1])
    rs = PL.Plan("reduce_scatter", P, N, "bf16", 1 << 20)
    rs_out = [torch.empty(N // P, dtype=torch.int16, device="cuda") for _ in range(P)]
    rs.exec(ins, rs_out)
    del ins
    ag = PL.Plan("allgather", P, N, "bf16", 1 << 20)
    ag.exec(rs_out, [outs[1], torch.empty(N, dtype=torch.int16, device="cuda")])
    torch.cuda.synchronize()
    assert torch.equal(outs[1], outs[0])


def test_collectives_at_1GiB_per_rank():
    """P = 8, bf16, 1 GiB per rank, chunk 1 MiB: the bandwidth sweep's
    largest calls, in the launch shapes it times (the reduces' outputs are
    larger than the last-level cache and written non-temporally).  Inputs are
    drawn on the device with a seeded torch generator; sampled elements of
    every ReduceScatter and AllReduce output are checked against the oracle,
    and RS then AG must equal the AllReduce bit for bit on every rank."""
    P, N = 8, (1 << 30) // 2
    M = N // P
    g = torch.Generator(device="cuda").manual_seed(57)
    ins = [(torch.randn(N, device="cuda", generator=g) * 0.02).to(torch.bfloat16).view(torch.int16) for _ in range(P)]
    rs_out = [torch.empty(M, dtype=torch.int16, device="cuda") for _ in range(P)]
    ar_out = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    PL.Plan("reduce_scatter", P, N, "bf16", 1 << 20).exec(ins, rs_out)
    PL.Plan("allreduce", P, N, "bf16", 1 << 20).exec(ins, ar_out)
    torch.cuda.synchronize()
    rng = np.random.default_rng(58)
    # random elements, both ends, and both sides of every partition boundary
    edges = ((np.arange(1, P) * M)[:, None] + np.arange(-64, 64)[None, :]).ravel()
    idx = np.unique(np.concatenate([rng.integers(0, N, 1 << 17), np.arange(4096), np.arange(N - 4096, N), edges]))
    idx_t = torch.from_numpy(idx).to("cuda")
    sample = [to_host(t[idx_t], np.uint16) for t in ins]
    want = oracle.all_reduce([np.concatenate([x, np.zeros((-len(x)) % P, np.uint16)]) for x in sample], "bf16")[0][: len(idx)]
    rs_cat = torch.cat(rs_out)
    assert_bits_equal(to_host(rs_cat[idx_t], np.uint16), want, "bf16", "ReduceScatter, 1 GiB/rank, sampled")
    for r in range(P):
        assert_bits_equal(to_host(ar_out[r][idx_t], np.uint16), want, "bf16", f"AllReduce rank {r}, 1 GiB/rank, sampled")
    del ins, rs_cat
    ag_out = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    PL.Plan("allgather", P, N, "bf16", 1 << 20).exec(rs_out, ag_out)
    torch.cuda.synchronize()
    for r in range(P):
        assert torch.equal(ag_out[r], ar_out[r]), f"RS then AG differs from AR at rank {r}, 1 GiB/rank"


def test_plans_run_concurrently_on_two_streams():
    """A plan is immutable: executions on different streams with distinct
    buffers may overlap (AllReduce on one stream, AllToAll and AllGather on
    another), each matching the oracle."""
    P, M = 8, 65536
    ins_a = _inputs(P, P * M, "bf16", seed=501)
    ins_b = _inputs(P, P * M, "bf16", seed=502)
    ar = PL.Plan("allreduce", P, P * M, "bf16", 1 << 16)
    a2a = PL.Plan("alltoall", P, P * M, "bf16", 1 << 16)
    ag = PL.Plan("allgather", P, P * M, "bf16", 1 << 16)
    d_a = [to_device(a) for a in ins_a]
    d_b = [to_device(a) for a in ins_b]
    d_g = [to_device(a[:M]) for a in ins_b]
    out_a = [torch.empty(P * M, dtype=torch.int16, device="cuda") for _ in range(P)]
    out_b = [torch.empty(P * M, dtype=torch.int16, device="cuda") for _ in range(P)]
    out_g = [torch.empty(P * M, dtype=torch.int16, device="cuda") for _ in range(P)]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(3):
        with torch.cuda.stream(s1):
            ar.exec(d_a, out_a, stream=s1)
        with torch.cuda.stream(s2):
            a2a.exec(d_b, out_b, stream=s2)
            ag.exec(d_g, out_g, stream=s2)
    torch.cuda.synchronize()
    want_a = oracle.all_reduce(ins_a, "bf16")
    want_b = oracle.all_to_all(ins_b, "bf16")
    want_g = oracle.all_gather([a[:M] for a in ins_b], "bf16")
    for r in range(P):
        assert_bits_equal(to_host(out_a[r], np.uint16), want_a[r], "bf16", f"AllReduce rank {r}")
        assert_bits_equal(to_host(out_b[r], np.uint16), want_b[r], "bf16", f"AllToAll rank {r}")
        assert_bits_equal(to_host(out_g[r], np.uint16), want_g[r], "bf16", f"AllGather rank {r}")


def test_bound_plan_matches_exec():
    """Plan.bind validates once and enqueues the same work as exec."""
    P, M = 8, 4096
    ins_np = _inputs(P, P * M, "bf16", seed=611)
    ins = [to_device(a) for a in ins_np]
    outs = [torch.empty(P * M, dtype=torch.int16, device="cuda") for _ in range(P)]
    plan = PL.Plan("allreduce", P, P * M, "bf16", 4096)
    run = plan.bind(ins, outs)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    want = oracle.all_reduce(ins_np, "bf16")
    for r in range(P):
        assert_bits_equal(to_host(outs[r], np.uint16), want[r], "bf16", f"bound AllReduce rank {r}")
    v = PL.purlin_plan_v("alltoallv", P, P * M, "bf16", 4096, unit=1)
    counts = to_device(np.full(P * P, M, np.int32))
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    runv = v.bind(ins, outs, counts=counts, dev_status=st)
    runv()
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    want = oracle.all_to_all(ins_np, "bf16")
    for r in range(P):
        assert_bits_equal(to_host(outs[r], np.uint16), want[r], "bf16", f"bound AllToAllV rank {r}")
    with pytest.raises(PL.PurlinError):
        v.bind(ins, outs)  # counts missing


@pytest.mark.parametrize("op", ["allreduce", "reduce_scatter"])
def test_repeated_runs_are_bit_identical(op):
    """Eq. 2's fixed order: five runs, and runs with another chunk size and
    item cut, give the same bits (no order depends on scheduling)."""
    P, M = 8, 1 << 18
    ins = [to_device(a) for a in _inputs(P, P * M, "bf16", seed=777)]
    plan = PL.Plan(op, P, P * M, "bf16", 1 << 16)
    outs = [torch.empty(plan.out_bytes // 2, dtype=torch.int16, device="cuda") for _ in range(P)]
    plan.exec(ins, outs)
    torch.cuda.synchronize()
    first = [o.clone() for o in outs]
    others = [plan] * 4 + [PL.Plan(op, P, P * M, "bf16", 4096, policy=dict(item_bytes=1024)),
                           PL.Plan(op, P, P * M, "bf16", 3 << 20, policy=dict(ar_mode=2))]
    for pl in others:
        for o in outs:
            o.fill_(0x5A5A)
        pl.exec(ins, outs)
        torch.cuda.synchronize()
        for r in range(P):
            assert torch.equal(outs[r], first[r]), f"{op} rank {r} differs between runs"


@pytest.mark.parametrize("nbytes", [16, 16 * 1023, 16 * 1024, 16 * 1024 * 37 + 48, 64 << 20])
def test_stream_copy_is_a_bit_copy(nbytes):
    """The plain reference copy: every byte lands, the guard band after the
    copied range stays untouched (ragged last workgroup included)."""
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device="cuda")
    dst = torch.full((nbytes + 4096,), 0xA5, dtype=torch.uint8, device="cuda")
    PL.purlin_stream_copy(dst, src)
    torch.cuda.synchronize()
    assert torch.equal(dst[:nbytes], src)
    assert bool((dst[nbytes:] == 0xA5).all())
