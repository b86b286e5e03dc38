#!/usr/bin/env python3
"""Benchmark of the datapath executor on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input:

  1. ReduceScatter, P=8 ranks, bf16, 134217728 elements (256 MiB) per rank,
     chunk 1 MiB                               (one executor launch)
  2. AllGather of its result (RS then AG = AllReduce), same shape (one launch)
  3. MoE dispatch: pack 4096 x 7168 bf16 tokens, top-8 Zipf(1.1) routing over
     256 experts on 8 ranks                     (three launches)
  4. MoE combine of 32768 x 7168 bf16 expert outputs with fp32 gates
                                                (one launch)

Plans are built once per shape (host orchestration, like the paper's
compile-time specialisation) and reused; every step re-executes them.

value = algorithmic bytes of a step (reads + writes each op must make at
least once) / wall time of a step, in GB/s (1e9 bytes/s); in the timed steps
only the dominant kernel is bracketed by HIP events (its launch duration
gives the roofline).  Per-op times come from as many steps before them, with
HIP events recorded between all the ops, on the stream the kernels run on.  The decode-size
AllReduce (P=8, bf16, 128 x 8192 per rank) and the small AllReduce (P=4,
fp32, 262144 per rank) are timed separately as latency: 128 calls captured
in a graph, one warm-up replay, eight timed replays, time / 1024 (the
paper's methodology, Section 5); so is the paper's latency sweep of
AllReduce, ReduceScatter, AllGather and AllToAll at 1 KiB..512 KiB per rank.

Prints ONE JSON line.
"""

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "datapath GB/s (read+write) and % of HBM peak; small-message latency µs"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
KERNEL_SOURCES = ["paper_2609_36954_amd/csrc/exec.hip", "paper_2609_36954_amd/csrc/moe.hip"]
# kernel (as rocprofv3 names it, a distinctive substring) of each single-launch op
KERNEL_OF_OP = {
    "reduce_scatter": "exec_reduce<8, true",
    "allgather": "exec_copy<",
    "moe_pack": "::pack_onepass<",  # the single-launch pack (the three-launch form: pack_tiles, pack_scan, pack_rows)
    "moe_combine": "unpack_rows<",
}
CALIBRATION_KERNEL = "copy"  # torch's device-to-device copy of --calibrate-copy
CALIBRATION_BYTES = 1 << 30


class TimingEvent:
    """A HIP event for timing only, created with hipEventDisableSystemFence:
    recording it skips the system-scope cache write-back and invalidation
    that a default event performs (several µs of stream time between two
    kernels), so bracketing a kernel barely perturbs the step.  Recorded on
    the stream the kernels run on; read after a device synchronisation.
    The HIP runtime is the one torch loaded (same soname)."""

    _hip = None

    def __init__(self, torch):
        import ctypes

        if TimingEvent._hip is None:
            h = ctypes.CDLL("libamdhip64.so.7")
            h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventDestroy.argtypes = [ctypes.c_void_p]
            TimingEvent._hip = h
        self._ctypes = ctypes
        self._torch = torch
        self.ev = ctypes.c_void_p()
        if TimingEvent._hip.hipEventCreateWithFlags(ctypes.byref(self.ev), 0x20000000) != 0:  # hipEventDisableSystemFence
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self):
        st = self._ctypes.c_void_p(self._torch.cuda.current_stream().cuda_stream)
        if TimingEvent._hip.hipEventRecord(self.ev, st) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end):
        """Milliseconds from this event to ``end`` (both recorded and complete)."""
        ms = self._ctypes.c_float()
        if TimingEvent._hip.hipEventElapsedTime(self._ctypes.byref(ms), self.ev, end.ev) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        if TimingEvent._hip is not None and self.ev:
            TimingEvent._hip.hipEventDestroy(self.ev)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash():
    """Hash of the kernel sources' code: comments, trailing blanks and empty
    lines are left out, so recorded counters stay tied to what compiles."""
    import re

    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        lines = (re.sub(r"//.*$", "", line).rstrip() for line in text.splitlines())
        h.update("\n".join(line for line in lines if line).encode())
    return h.hexdigest()[:16]


def collective_bytes(op, P, N, s):
    """Algorithmic bytes: every input byte read once, every output byte written once."""
    if op == "reduce_scatter":
        return P * N * s + N * s
    if op == "allgather":
        return N * s + P * N * s
    if op in ("allreduce", "alltoall"):
        return 2 * P * N * s
    raise ValueError(op)


def pack_bytes(T, H, K, E, P):
    return T * H * 2 + T * K * H * 2 + T * K * 4 + T * K * 4 + (2 * P + 2 * E) * 4


def unpack_bytes(T, H, K):
    return T * K * H * 2 + T * H * 2 + T * K * 4 + T * K * 4


def to_dev(torch, a):
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to("cuda")


def _counter_means(d, counter):
    """Mean and largest Counter_Value per kernel name over the dispatches in
    a rocprofv3 --pmc CSV directory (…_counter_collection.csv)."""
    import csv
    import glob

    sums = {}
    for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for row in csv.DictReader(f):
                if row.get("Counter_Name") != counter:
                    continue
                k = row["Kernel_Name"]
                v = sums.setdefault(k, [0.0, 0, 0.0])
                x = float(row["Counter_Value"])
                v[0] += x
                v[1] += 1
                v[2] = max(v[2], x)
    return {k: v[0] / v[1] for k, v in sums.items()}, {k: v[2] for k, v in sums.items()}


def ingest_counters(fetch_dir, write_dir, path=None):
    """FETCH_SIZE / WRITE_SIZE (KiB per dispatch) -> HBM bytes per launch,
    written to ``path`` (default profiles/traffic.json).

    Each counter is scaled by what it reads for a plain 1 GiB device copy
    (reads 1 GiB, writes 1 GiB), run in the same process."""
    fetch, fetch_max = _counter_means(fetch_dir, "FETCH_SIZE")
    write, write_max = _counter_means(write_dir, "WRITE_SIZE")

    def pick(table, sub, exclude=None):
        names = [k for k in table if sub in k and (exclude is None or exclude not in k)]
        if not names:
            raise SystemExit(f"no kernel matching {sub!r} in the counter CSVs")
        return max(names, key=lambda k: table[k])

    # the calibration copy is the largest dispatch of the copy kernel in the run
    cal_f = pick(fetch_max, CALIBRATION_KERNEL, exclude="purlin")
    cal_w = pick(write_max, CALIBRATION_KERNEL, exclude="purlin")
    f_scale = CALIBRATION_BYTES / (fetch_max[cal_f] * 1024.0)
    w_scale = CALIBRATION_BYTES / (write_max[cal_w] * 1024.0)
    out = {
        "kernel_source_hash": kernel_source_hash(),
        "calibration": {"kernel": cal_f, "bytes_read": CALIBRATION_BYTES, "bytes_written": CALIBRATION_BYTES,
                        "fetch_KiB": fetch_max[cal_f], "write_KiB": write_max[cal_w],
                        "fetch_scale": f_scale, "write_scale": w_scale},
        "ops": {},
    }
    for op, sub in KERNEL_OF_OP.items():
        kf, kw = pick(fetch, sub), pick(write, sub)
        fb, wb = fetch[kf] * 1024.0 * f_scale, write[kw] * 1024.0 * w_scale
        out["ops"][op] = {"kernel": kf, "fetch_KiB": fetch[kf], "write_KiB": write[kw],
                          "hbm_read_bytes": round(fb), "hbm_write_bytes": round(wb),
                          "hbm_bytes_per_launch": round(fb + wb)}
    if path is None:
        path = os.path.join(ROOT, "profiles", "traffic.json")
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))
    return 0


def load_traffic(src_hash):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they
    were taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_hash") != src_hash:
        return None
    return t


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-latency-sweep", action="store_true",
                    help="skip the sweep of AllReduce, ReduceScatter, AllGather, AllToAll at 1 KiB..512 KiB per rank")
    ap.add_argument("--no-latency", action="store_true", help="skip the graph-replayed latency measurement")
    ap.add_argument("--bandwidth-sweep", action="store_true",
                    help="also time AllReduce, ReduceScatter, AllGather and AllToAll at 1 MiB..1 GiB per rank "
                         "(the paper's bandwidth range; 16 GiB of buffers)")
    ap.add_argument("--sweep-only", action="store_true",
                    help="only the bandwidth sweep (its kernels alone, for counter runs)")
    ap.add_argument("--plateau", action="store_true",
                    help="also time ReduceScatter and AllGather with the grid capped at 4..512 workgroups "
                         "(off by default: the capped launches share the step's kernels and would skew their "
                         "per-kernel profiler averages)")
    ap.add_argument("--no-extra", action="store_true", help="skip timing the other collectives (outside the step)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run one 1 GiB device-to-device tensor copy first (reference for HBM counter scaling)")
    ap.add_argument("--ingest-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) into profiles/traffic.json")
    args = ap.parse_args()
    if args.ingest_counters:
        return ingest_counters(*args.ingest_counters)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "purlin-mi355x runs on one GPU: the P ranks are P buffers on that GPU; "
                          "--gpus above 1 is not supported"}))
        return 2

    import torch

    from paper_2609_36954_amd import purlin as PL
    from paper_2609_36954_amd import workloads as W

    PL.lib()  # fail loudly if the HIP library is missing
    torch.cuda.set_device(0)
    if args.sweep_only:
        print(json.dumps(measure_bandwidth_sweep(torch, PL)), flush=True)
        return 0
    dev_name = torch.cuda.get_device_name(0)
    src_hash = kernel_source_hash()

    # ---------------- inputs (seeded, synthetic) ----------------
    c3 = W.RS_AG_P8_BF16_256MIB
    P, N, s = c3.P, c3.count, 2
    M = N // P
    moe = W.MOE_CONFIG
    T, H, E, K = moe.T, moe.H, moe.E, moe.K
    t0 = time.time()
    log(f"bench: generating inputs (RS/AG P={P} N={N} bf16; MoE T={T} H={H} E={E} K={K})")
    ins_np = W.collective_inputs(c3)
    ids_np = W.zipf_topk_ids(T, E, K, moe.zipf_s, moe.seed_ids)
    x_np = W.moe_tokens(moe)
    y_np = W.moe_expert_outputs(moe)
    g_np = W.softmax_gates(T, K, moe.seed_gates)
    log(f"bench: inputs ready in {time.time() - t0:.1f}s; uploading")

    if args.calibrate_copy:
        a = torch.empty(1 << 29, dtype=torch.int16, device="cuda").fill_(1)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    ins = [to_dev(torch, a) for a in ins_np]
    rs_out = [torch.empty(M, dtype=torch.int16, device="cuda") for _ in range(P)]
    ag_out = [torch.empty(N, dtype=torch.int16, device="cuda") for _ in range(P)]
    x, ids, y, g = to_dev(torch, x_np), to_dev(torch, ids_np), to_dev(torch, y_np), to_dev(torch, g_np)
    pack_out = dict(
        packed=torch.empty((T * K, H), dtype=torch.int16, device="cuda"),
        dest_counts=torch.empty(P, dtype=torch.int32, device="cuda"),
        dest_offsets=torch.empty(P, dtype=torch.int32, device="cuda"),
        expert_counts=torch.empty(E, dtype=torch.int32, device="cuda"),
        expert_offsets=torch.empty(E, dtype=torch.int32, device="cuda"),
        pos=torch.empty((T, K), dtype=torch.int32, device="cuda"),
    )
    ws = torch.empty(PL.purlin_pack_workspace_size(T, K, E), dtype=torch.uint8, device="cuda")
    comb_out = torch.empty((T, H), dtype=torch.int16, device="cuda")

    # ---------------- plans (host orchestration, once per shape) ----------------
    tp = time.perf_counter()
    rs_plan = PL.Plan("reduce_scatter", P, N, "bf16", c3.chunk)
    ag_plan = PL.Plan("allgather", P, N, "bf16", c3.chunk)
    plan_ms = (time.perf_counter() - tp) * 1e3

    ops = [
        ("reduce_scatter", collective_bytes("reduce_scatter", P, N, s), rs_plan.sched_bytes),
        ("allgather", collective_bytes("allgather", P, N, s), ag_plan.sched_bytes),
        ("moe_pack", pack_bytes(T, H, K, E, P), pack_bytes(T, H, K, E, P)),
        ("moe_combine", unpack_bytes(T, H, K), unpack_bytes(T, H, K)),
    ]
    step_bytes = sum(b for _, b, _ in ops)

    op_names = [name for name, _, _ in ops]

    def step(evs=None, only=None):
        """One pass of the hot path.  ``evs``: events recorded between the ops
        (``only``: just around that op)."""
        def mark(k):
            if evs is not None and (only is None or k in (only, only + 1)):
                evs[k if only is None else k - only].record()
        mark(0)
        rs_plan.exec(ins, rs_out)
        mark(1)
        ag_plan.exec(rs_out, ag_out)
        mark(2)
        PL.purlin_pack(x, ids, E, P, out=pack_out, workspace=ws)
        mark(3)
        PL.purlin_unpack(y, pack_out["pos"], g, out=comb_out)
        mark(4)

    log("bench: warmup")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # Per-op breakdown first: as many steps as timed, HIP events between the
    # ops (on the stream the kernels run on).  Figures are the mean over the
    # steps, with the median beside it (a host stall that lets the stream
    # drain inflates one step's gap).
    log(f"bench: per-op breakdown ({args.steps} steps, events between the ops)")
    events = [[TimingEvent(torch) for _ in range(5)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    per_op = {}
    for j, (name, bmin, bsched) in enumerate(ops):
        ts = [events[i][j].elapsed_time(events[i][j + 1]) for i in range(args.steps)]
        avg_ms = float(np.mean(ts))
        per_op[name] = {
            "avg_us": round(avg_ms * 1e3, 2),
            "median_us": round(float(np.median(ts)) * 1e3, 2),
            "min_us": round(float(np.min(ts)) * 1e3, 2),
            "bytes_min": int(bmin),
            "bytes_sched": int(bsched),
            "GBps_min": round(bmin / (avg_ms * 1e-3) / 1e9, 1),
            "frac_of_hbm_peak": round(bmin / (avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        }
        if name in ("reduce_scatter", "allgather"):  # the paper's algorithm bandwidth: per-rank message / time
            per_op[name]["algbw_GBps"] = round(N * s / (avg_ms * 1e-3) / 1e9, 1)

    # dominant single-kernel op (RS, AG and combine are one launch each)
    single = ["reduce_scatter", "allgather", "moe_combine"]
    dom = max(single, key=lambda n: per_op[n]["median_us"])
    di = op_names.index(dom)

    # The timed region: exactly `steps` steps between two synchronisations,
    # wall-clocked for the value; events only around the dominant kernel (two
    # per step: its launch duration for the roofline, live on its stream).
    log(f"bench: timing {args.steps} steps")
    dom_ev = [[TimingEvent(torch) for _ in range(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for i in range(args.steps):
        step(dom_ev[i], only=di)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_per_step = wall * 1e3 / args.steps
    value = step_bytes / (ms_per_step * 1e-3) / 1e9

    dom_ts = [e[0].elapsed_time(e[1]) for e in dom_ev]
    dom_us = float(np.mean(dom_ts)) * 1e3
    achieved = per_op[dom]["bytes_min"] / (dom_us * 1e-6) / 1e9
    traffic = None
    tr = load_traffic(src_hash)
    if tr and dom in tr.get("ops", {}):
        traffic = tr["ops"][dom].get("hbm_bytes_per_launch")
    roofline = {
        "bound": "hbm",
        "kernel": KERNEL_OF_OP[dom],
        "op": dom,
        "achieved": round(achieved, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4),
        "traffic": traffic,
        "launch_us": round(dom_us, 2),
        "launch_us_median": round(float(np.median(dom_ts)) * 1e3, 2),
        "timing": "HIP events (no system fence) around the kernel in each timed step, on its stream",
    }

    # ---------------- latency: decode-size AllReduce ----------------
    def graph_latency_us(plan, lin, lout, calls=128, reps=8):
        return graph_call_us(torch, lambda st: plan.exec(lin, lout, stream=st), calls, reps)

    # ---------------- CPU baseline: the oracle on a bounded sample ----------------
    # (first: it compares the step's own outputs, which the later measurements overwrite)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(torch, ins_np, rs_out, ag_out, x_np, ids_np, y_np, g_np, pack_out, comb_out, P, N, M, E, K)

    # ---------------- the MoE ops' access mixes as plain streams, in the ops' place ----------------
    in_step = measure_in_step_streams(torch, PL, rs_plan, ag_plan, ins, rs_out, ag_out, x, y, pack_out["packed"],
                                      comb_out, T, H, K, per_op, args.steps)

    # ---------------- the pack's status word (repeated and out-of-range ids) ----------------
    in_step["pack_status_word"] = measure_pack_status_in_step(torch, PL, rs_plan, ag_plan, ins, rs_out, ag_out, x, ids,
                                                              y, g, pack_out, comb_out, ws, E, P, args.steps)

    # ---------------- how the chip's dies share the pack's time ----------------
    in_step["xcd_balance"] = measure_xcd_balance(torch, PL, rs_plan, ag_plan, ins, rs_out, ag_out, x, ids, y, g,
                                                 pack_out, comb_out, T, H, E, K, P)

    # ---------------- the other collectives at the same shape (not in the step) ----------------
    extra = None
    if not args.no_extra:
        extra = measure_extra_ops(torch, PL, ins, rs_out, ag_out, P, N, s)

        extra["expert_parallel_p8"] = measure_ep(torch, PL, W, P, T, H, E, K)
        extra["rank0_share"] = measure_share(torch, PL, ins, rs_out, ag_out, P, N, s)
        if args.plateau:
            extra["workgroup_plateau"] = measure_plateau(torch, PL, ins, rs_out, ag_out, P, N, s)
        if args.bandwidth_sweep:
            extra["bandwidth_sweep"] = measure_bandwidth_sweep(torch, PL)

    latency = None
    if not args.no_latency:
        latency = measure_latency(torch, PL, W, graph_latency_us, not args.no_latency_sweep)
    ceilings = None if args.no_extra else measure_ceilings(torch, PL)
    return emit(args, value, ms_per_step, step_bytes, P, N, T, H, E, K, roofline, cpu, per_op, latency, plan_ms,
                dev_name, src_hash, extra, ceilings, in_step)


def graph_call_us(torch, enqueue, calls=128, reps=8):
    """The paper's small-message timing (Section 5): `calls` calls captured
    in one graph on a side stream, one warm-up replay, then `reps` timed
    replays; returns µs per call (elapsed / (calls * reps)).  `enqueue(st)`
    issues one call on stream `st`."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        enqueue(side)
    torch.cuda.synchronize()
    gph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gph, stream=side):
        for _ in range(calls):
            enqueue(side)
    gph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        gph.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / (calls * reps)


def measure_extra_ops(torch, PL, ins, rs_out, ag_out, P, N, s, reps=5):
    """AllReduce, AllToAll, the rooted and the variable-size collectives at
    256 MiB/rank, P=8, bf16, chunk 1 MiB: event-timed on the current stream,
    outside the step."""
    root = 0
    cases = [
        ("allreduce", PL.Plan("allreduce", P, N, "bf16", 1 << 20), ins, ag_out, 2 * P * N * s),
        ("alltoall", PL.Plan("alltoall", P, N, "bf16", 1 << 20), ins, ag_out, 2 * P * N * s),
        ("broadcast", PL.Plan("broadcast", P, N, "bf16", 1 << 20, root=root),
         [ins[root]] + [None] * (P - 1), ag_out, N * s + P * N * s),
        ("reduce", PL.Plan("reduce", P, N, "bf16", 1 << 20, root=root), ins,
         [ag_out[root]] + [None] * (P - 1), P * N * s + N * s),
        ("scatter", PL.Plan("scatter", P, N, "bf16", 1 << 20, root=root),
         [ins[root]] + [None] * (P - 1), rs_out, 2 * N * s),
        ("gather", PL.Plan("gather", P, N, "bf16", 1 << 20, root=root), rs_out,
         [ag_out[root]] + [None] * (P - 1), 2 * N * s),
    ]
    # variable-size collectives with the Appendix C.4 split of T = 256 MiB per rank
    from paper_2609_36954_amd import workloads as W

    split = [b // s for b in W.zipf_split(N * s)]
    dev_split = torch.tensor(split, dtype=torch.int32, device="cuda")
    dev_a2av = torch.tensor([x for row in W.alltoallv_counts(split) for x in row], dtype=torch.int32, device="cuda")
    vcases = [
        ("allgatherv_zipf", PL.Plan("allgatherv", P, N, "bf16", 1 << 20, unit=1), ins, ag_out, dev_split,
         (P + 1) * N * s),
        ("reduce_scatterv_zipf", PL.Plan("reduce_scatterv", P, N, "bf16", 1 << 20, unit=1), ins, ag_out, dev_split,
         (P + 1) * N * s),
        ("alltoallv_zipf", PL.Plan("alltoallv", P, N, "bf16", 1 << 20, unit=1), ins, ag_out, dev_a2av,
         2 * P * N * s),
    ]
    out = {}
    for name, plan, i, o, counts, bmin in vcases:
        cases.append((name, plan, i, o, bmin))
        plan._bench_counts = counts
    for name, plan, i, o, bmin in cases:
        if plan.unit is not None:
            run = (lambda plan=plan, i=i, o=o: plan.exec_v(i, o, plan._bench_counts))
        else:
            run = (lambda plan=plan, i=i, o=o: plan.exec(i, o))
        run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            run()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        out[name] = {"avg_us": round(us, 2), "bytes_min": int(bmin), "bytes_sched": int(plan.sched_bytes),
                     "GBps_min": round(bmin / (us * 1e-6) / 1e9, 1),
                     "frac_of_hbm_peak": round(bmin / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                     "algbw_GBps": round(N * s / (us * 1e-6) / 1e9, 1)}
    return out


def _time_stages(torch, stages, bmin, reps):
    """Event-time each stage (a callable) of a sequence, averaged over reps."""
    for _, f in stages:
        f()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)]
    tot = [0.0] * len(stages)
    for _ in range(reps):
        ev[0].record()
        for i, (_, f) in enumerate(stages):
            f()
            ev[i + 1].record()
        torch.cuda.synchronize()
        for i in range(len(stages)):
            tot[i] += ev[i].elapsed_time(ev[i + 1])
    out = {}
    for (name, _), t in zip(stages, tot):
        us = t * 1e3 / reps
        out[name] = {"avg_us": round(us, 2), "bytes_min": int(bmin[name]),
                     "GBps_min": round(bmin[name] / (us * 1e-6) / 1e9, 1),
                     "frac_of_hbm_peak": round(bmin[name] / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    total_us = sum(v["avg_us"] for v in out.values())
    total_b = sum(bmin.values())
    out["round_trip"] = {"avg_us": round(total_us, 2), "bytes_min": int(total_b),
                         "GBps_min": round(total_b / (total_us * 1e-6) / 1e9, 1),
                         "frac_of_hbm_peak": round(total_b / (total_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    return out


def measure_ep(torch, PL, W, P, T, H, E, K, reps=5):
    """Expert-parallel dispatch and combine of P ranks with T tokens each
    (Table 2): dispatch = P packs, then the AllToAllV of the packed rows with
    the packs' dest_counts (read on the device, unit = H); combine = the
    reverse AllToAllV (same counts, column-major), then P unpacks.  Receive
    buffers hold the worst case.  Routing: Zipf(1.1) top-K per rank, seeded
    per rank.  Three variants: one row per (token, slot); de-duplicated
    (one row per token and destination rank; its combine sums the ranks'
    partial rows); and one pass each way (purlin_ep_dispatch writes the rows
    straight into the receive buffers, purlin_ep_combine reads them back from
    there: the per-slot result without the packed buffers), also
    de-duplicated.  Event-timed on the current stream."""
    i32 = dict(dtype=torch.int32, device="cuda")
    row = H * 2
    xs, ids, gates = [], [], []
    rngs = W.rank_rngs(4040, P)
    for p in range(P):
        xs.append(to_dev(torch, W.normal_bf16(rngs[p], T * H).reshape(T, H)))
        ids.append(torch.from_numpy(W.zipf_topk_ids(T, E, K, 1.1, 4000 + p)).to("cuda"))
        gates.append(torch.from_numpy(W.softmax_gates(T, K, 5000 + p)).to("cuda"))
    result = {}
    for variant in ("per_slot", "dedup"):
        dedup = variant == "dedup"
        rows_in = T * (min(K, P) if dedup else K)
        rows_out = P * rows_in
        counts = torch.zeros((P, P), **i32)
        if dedup:
            packs = [dict(packed=torch.empty((rows_in, H), dtype=torch.int16, device="cuda"), dest_counts=counts[p],
                          dest_offsets=torch.empty(P, **i32), row_of=torch.empty((T, P), **i32)) for p in range(P)]
            ws = torch.empty(max(PL.purlin_pack_dedup_workspace_size(T, P), 16), dtype=torch.uint8, device="cuda")
        else:
            packs = [dict(packed=torch.empty((rows_in, H), dtype=torch.int16, device="cuda"), dest_counts=counts[p],
                          dest_offsets=torch.empty(P, **i32), expert_counts=torch.empty(E, **i32),
                          expert_offsets=torch.empty(E, **i32), pos=torch.empty((T, K), **i32)) for p in range(P)]
            ws = torch.empty(max(PL.purlin_pack_workspace_size(T, K, E), 16), dtype=torch.uint8, device="cuda")
        recv = [torch.empty(rows_out * H, dtype=torch.int16, device="cuda") for _ in range(P)]
        back = [torch.empty(rows_in * H, dtype=torch.int16, device="cuda") for _ in range(P)]
        outs = [torch.empty((T, H), dtype=torch.int16, device="cuda") for _ in range(P)]
        fwd = PL.purlin_plan_v("alltoallv", P, rows_in * H, "bf16", 1 << 20, unit=H, out_capacity=rows_out * H)
        bwd = PL.purlin_plan_v("alltoallv", P, rows_out * H, "bf16", 1 << 20, unit=H, out_capacity=rows_in * H,
                               counts_transposed=True)
        flat = counts.view(-1)

        def pack_all(dedup=dedup, packs=packs, ws=ws):
            for p in range(P):
                if dedup:
                    PL.purlin_pack_dedup(xs[p], ids[p], E, P, out=packs[p], workspace=ws)
                else:
                    PL.purlin_pack(xs[p], ids[p], E, P, out=packs[p], workspace=ws)

        def unpack_all(dedup=dedup, packs=packs, back=back, outs=outs, rows_in=rows_in):
            for p in range(P):
                if dedup:
                    PL.purlin_unpack_dedup(back[p].view(rows_in, H), packs[p]["row_of"], out=outs[p])
                else:
                    PL.purlin_unpack(back[p].view(rows_in, H), packs[p]["pos"], gates[p], out=outs[p])

        stages = [("pack", pack_all),
                  ("dispatch_alltoallv", lambda fwd=fwd, packs=packs, recv=recv, flat=flat:
                   fwd.exec_v([pk["packed"].view(-1) for pk in packs], recv, flat)),
                  ("combine_alltoallv", lambda bwd=bwd, recv=recv, back=back, flat=flat: bwd.exec_v(recv, back, flat)),
                  ("unpack", unpack_all)]
        pack_all()
        torch.cuda.synchronize()
        m = counts.cpu().numpy()
        sent = m.sum(axis=1)  # rows each rank sends (= receives back)
        meta = P * T * K * 4 + (P * T * P * 4 if dedup else P * T * K * 4)  # ids + row_of / pos
        bmin = {
            "pack": P * T * row + int(sent.sum()) * row + meta,
            "dispatch_alltoallv": 2 * int(sent.sum()) * row,
            "combine_alltoallv": 2 * int(sent.sum()) * row,
            "unpack": int(sent.sum()) * row + P * T * row + (P * T * P * 4 if dedup else 2 * P * T * K * 4),
        }
        r = _time_stages(torch, stages, bmin, reps)
        r["rows_sent_per_rank"] = [int(v) for v in sent]
        r["rows_received_per_rank"] = [int(v) for v in m.sum(axis=0)]
        result[variant] = r
        del packs, recv, back, outs, ws
    # one pass each way: rows straight to the receive buffers and back
    cap = P * T * K
    recv = [torch.empty((cap, H), dtype=torch.int16, device="cuda") for _ in range(P)]
    outs = [torch.empty((T, H), dtype=torch.int16, device="cuda") for _ in range(P)]
    counts = torch.empty(P * P, dtype=torch.int32, device="cuda")
    recv_pos = torch.empty((P, T, K), dtype=torch.int32, device="cuda")
    ws = torch.empty(PL.purlin_ep_dispatch_workspace_size(T, K, E, P), dtype=torch.uint8, device="cuda")
    stages = [("dispatch", lambda: PL.purlin_ep_dispatch(xs, ids, E, recv, counts=counts, recv_pos=recv_pos,
                                                         workspace=ws)),
              ("combine", lambda: PL.purlin_ep_combine(recv, ids, recv_pos, gates, E, outs=outs))]
    stages[0][1]()
    torch.cuda.synchronize()
    sent = int(counts.sum().item())
    bmin = {"dispatch": P * T * row + sent * row + 2 * P * T * K * 4,
            "combine": sent * row + P * T * row + 3 * P * T * K * 4}
    r = _time_stages(torch, stages, bmin, reps)
    r["rows_sent_total"] = sent
    result["one_pass"] = r
    # de-duplicated, one pass each way
    ws2 = torch.empty(PL.purlin_ep_dispatch_dedup_workspace_size(T, P), dtype=torch.uint8, device="cuda")
    recv_row = torch.empty((P, T, P), dtype=torch.int32, device="cuda")
    stages = [("dispatch", lambda: PL.purlin_ep_dispatch_dedup(xs, ids, E, recv, counts=counts, recv_row=recv_row,
                                                               workspace=ws2)),
              ("combine", lambda: PL.purlin_ep_combine_dedup(recv, recv_row, outs=outs))]
    stages[0][1]()
    torch.cuda.synchronize()
    sent = int(counts.sum().item())
    bmin = {"dispatch": P * T * row + sent * row + P * T * K * 4 + P * T * P * 4,
            "combine": sent * row + P * T * row + P * T * P * 4}
    r = _time_stages(torch, stages, bmin, reps)
    r["rows_sent_total"] = sent
    result["one_pass_dedup"] = r
    del recv, outs, ws, ws2
    result["workload"] = {"P": P, "T_per_rank": T, "H": H, "E": E, "K": K, "routing": "Zipf(1.1) top-K"}
    result["dedup_speedup"] = round(result["per_slot"]["round_trip"]["avg_us"] /
                                    result["dedup"]["round_trip"]["avg_us"], 3)
    result["one_pass_speedup"] = round(result["per_slot"]["round_trip"]["avg_us"] /
                                       result["one_pass"]["round_trip"]["avg_us"], 3)
    result["one_pass_dedup_speedup"] = round(result["per_slot"]["round_trip"]["avg_us"] /
                                             result["one_pass_dedup"]["round_trip"]["avg_us"], 3)
    del xs, ids, gates
    return result


def measure_share(torch, PL, ins, rs_out, ag_out, P, N, s, reps=5):
    """Rank 0's share of ReduceScatter, AllGather and AllReduce at 256 MiB
    per rank (purlin_plan_share: the descriptors that write out_0, what one
    GPU would execute with the path sharded over P GPUs).  Bytes = what the
    share reads and writes, each byte once."""
    out = {}
    cases = [
        ("reduce_scatter", PL.Plan("reduce_scatter", P, N, "bf16", 1 << 20, share=0), ins,
         [rs_out[0]] + [None] * (P - 1)),
        ("allgather", PL.Plan("allgather", P, N, "bf16", 1 << 20, share=0), rs_out, [ag_out[0]] + [None] * (P - 1)),
        ("allreduce", PL.Plan("allreduce", P, N, "bf16", 1 << 20, share=0), ins, ag_out),
    ]
    # push shares (the descriptors that read in_0): the copy collectives only
    cases += [
        ("allgather_push", PL.Plan("allgather", P, N, "bf16", 1 << 20, share=0, push=True), rs_out, ag_out),
        ("alltoall_push", PL.Plan("alltoall", P, N, "bf16", 1 << 20, share=0, push=True), ins, ag_out),
        ("alltoall", PL.Plan("alltoall", P, N, "bf16", 1 << 20, share=0), ins, [ag_out[0]] + [None] * (P - 1)),
    ]
    for name, plan, i, o in cases:
        run = plan.bind(i, o)
        run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            run()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        out[name] = {"avg_us": round(us, 2), "bytes": int(plan.sched_bytes),
                     "GBps": round(plan.sched_bytes / (us * 1e-6) / 1e9, 1),
                     "frac_of_hbm_peak": round(plan.sched_bytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    out["what"] = ("rank 0's share at P=8, 256 MiB per rank, bf16, chunk 1 MiB: pull (the descriptors writing out_0) "
                   "and, for the copies, push (the descriptors reading in_0); the other ranks' buffers stand in for "
                   "peer memory")
    return out


def measure_bandwidth_sweep(torch, PL, P=8, reps=5):
    """The paper's bandwidth range (Section 5: 1 MiB..1 GiB per rank), P=8,
    bf16, chunk 1 MiB, for the four collectives: µs, algorithmic GB/s and
    the paper's algorithm bandwidth (per-rank message / time)."""
    s = 2
    big = (1 << 30) // s
    ins = [torch.empty(big, dtype=torch.int16, device="cuda").fill_(0x3F80) for _ in range(P)]
    outs = [torch.empty(big, dtype=torch.int16, device="cuda") for _ in range(P)]
    out = {}
    for op in ("allreduce", "reduce_scatter", "allgather", "alltoall"):
        row = {}
        for mib in (1, 4, 16, 64, 256, 1024):
            n = (mib << 20) // s
            i = [t[: n // P] for t in ins] if op == "allgather" else [t[:n] for t in ins]
            o = [t[: n // P] for t in outs] if op == "reduce_scatter" else [t[:n] for t in outs]
            run = PL.Plan(op, P, n, "bf16", 1 << 20).bind(i, o)
            run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                run()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            b = collective_bytes(op, P, n, s)
            row[f"{mib}MiB"] = {"us": round(us, 1), "GBps": round(b / (us * 1e-6) / 1e9, 1),
                                "algbw_GBps": round(n * s / (us * 1e-6) / 1e9, 1)}
        out[op] = row
        log(f"bandwidth sweep: {op} done")
    # The same calls on fresh buffers.  Above, every call reuses the buffers
    # of the call before, and at 256 MiB/rank the smaller side of a
    # ReduceScatter or AllGather (its output or its input, 256 MiB in all)
    # is then partly still in the 256 MB last-level cache.  Here the calls
    # rotate over four sets of that side and two of the full-size outputs.
    small = [[torch.empty(big // P, dtype=torch.int16, device="cuda").fill_(0x3F80) for _ in range(P)]
             for _ in range(4)]
    outs2 = [torch.empty(big, dtype=torch.int16, device="cuda") for _ in range(P)]
    cold = {}
    for op in ("allreduce", "reduce_scatter", "allgather", "alltoall"):
        row = {}
        for mib in (256, 1024):
            n = (mib << 20) // s
            runs = []
            for j in range(4):
                sm = [t[: n // P] for t in small[j]]
                full_out = [t[:n] for t in (outs if j % 2 == 0 else outs2)]
                i = sm if op == "allgather" else [t[:n] for t in ins]
                o = sm if op == "reduce_scatter" else full_out
                runs.append(PL.Plan(op, P, n, "bf16", 1 << 20).bind(i, o))
            runs[0]()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for r in range(2 * len(runs)):
                runs[r % len(runs)]()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / (2 * len(runs))
            b = collective_bytes(op, P, n, s)
            row[f"{mib}MiB"] = {"us": round(us, 1), "GBps": round(b / (us * 1e-6) / 1e9, 1)}
        cold[op] = row
        log(f"bandwidth sweep, fresh buffers: {op} done")
    out["fresh_buffers"] = cold
    # Reference streams of the same access mixes at 1 GiB per buffer (the
    # best of the four load/store hint pairs): what each mix reaches at that
    # size without descriptors.
    G = big * s
    mixes = {}
    for name, d, src in (("8_to_8", outs, ins), ("1_to_8", outs, ins[:1]), ("8_to_1", outs[:1], ins),
                         ("1_to_1", outs[:1], ins[:1])):
        best = None
        for ntl in (False, True):
            for nts in (False, True):
                fn = lambda: PL.purlin_stream(d, src, nbytes=G, nt_load=ntl, nt_store=nts)
                fn()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(3):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                us = e0.elapsed_time(e1) * 1e3 / 3
                if best is None or us < best[0]:
                    best = (us, ntl, nts)
        us, ntl, nts = best
        mixes[name] = {"us": round(us, 1), "GBps": round((len(d) + len(src)) * G / (us * 1e-6) / 1e9, 1),
                       "hints": f"{'nt' if ntl else 'cached'} loads {'nt' if nts else 'cached'} stores"}
    out["stream_ceilings_1GiB"] = mixes
    log("bandwidth sweep: 1 GiB reference streams done")
    del ins, outs, outs2, small
    torch.cuda.empty_cache()
    return out


def measure_plateau(torch, PL, ins, rs_out, ag_out, P, N, s, reps=3):
    """ReduceScatter and AllGather at 256 MiB/rank with the grid capped at
    W workgroups (policy max_workgroups; one workgroup occupies one CU): the
    bandwidth a collective reaches on a bounded share of the GPU, and the
    smallest cap within 90% of the uncapped launch (the resource plateau the
    paper measures for its copy, Section 5)."""
    out = {}
    for name, op, i, o in (("reduce_scatter", "reduce_scatter", ins, rs_out), ("allgather", "allgather", rs_out, ag_out)):
        row = {}
        for cap in (4, 8, 16, 32, 64, 128, 256, 512, 0):
            plan = PL.Plan(op, P, N, "bf16", 1 << 20, policy={"max_workgroups": cap} if cap else None)
            run = plan.bind(i, o)
            run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                run()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            row[str(cap) if cap else "uncapped"] = round(collective_bytes(op, P, N, s) / (us * 1e-6) / 1e9, 1)
        full = row["uncapped"]
        knee = next((int(k) for k, v in row.items() if k != "uncapped" and v >= 0.9 * full), None)
        out[name] = {"GBps_by_workgroups": row, "smallest_cap_within_90pct": knee}
    # the pipeline depth of the copies (Eq. 1: bandwidth ~ bytes in flight /
    # latency): 16-byte loads per lane in flight, on a bounded grid
    depth = {}
    for cap in (16, 64, 0):
        row = {}
        for d in (1, 2, 4, 8):
            pol = {"copy_depth": d}
            if cap:
                pol["max_workgroups"] = cap
            plan = PL.Plan("allgather", P, N, "bf16", 1 << 20, policy=pol)
            run = plan.bind(rs_out, ag_out)
            run()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                run()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            row[str(d)] = round(collective_bytes("allgather", P, N, s) / (us * 1e-6) / 1e9, 1)
        depth[str(cap) if cap else "uncapped"] = row
    out["allgather_GBps_by_copy_depth"] = depth
    out["what"] = "256 MiB/rank, P=8, bf16, chunk 1 MiB; GB/s = algorithmic bytes / time; 256 CUs on the chip"
    return out


def measure_ceilings(torch, PL, nbytes=1 << 30, reps=20):
    """Reference streams on the same GPU, for scale: hipMemcpyAsync (torch's
    same-device tensor copy), the library's plain copy kernel
    (purlin_stream_copy) and its descriptor-free streams (purlin_stream):
    read-only and write-only 1 GiB, a 1 GiB copy, 8 sources of 256 MiB
    XOR-ed into one (ReduceScatter's 8-to-1 mix) and one 256 MiB source
    written to 8 destinations (AllGather's 1-to-8 mix).  Each purlin_stream
    mix runs with the four load/store cache-hint combinations; the mix's
    figure is the best of them (all four are kept under "by_hints").
    GB/s = bytes read + written / time, HIP events without a system fence
    around `reps` back-to-back calls on the current stream, after 3 untimed
    calls."""
    part = nbytes // 4
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(7)
    dst = torch.empty_like(src)
    srcs8 = [torch.empty(part, dtype=torch.uint8, device="cuda").fill_(p) for p in range(8)]
    dsts8 = [torch.empty(part, dtype=torch.uint8, device="cuda") for _ in range(8)]
    sink = torch.empty(16, dtype=torch.uint8, device="cuda")

    def timed(fn, moved):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0, e1 = TimingEvent(torch), TimingEvent(torch)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        return {"avg_us": round(us, 1), "bytes": int(moved), "GBps": round(moved / (us * 1e-6) / 1e9, 1),
                "frac_of_hbm_peak": round(moved / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}

    out = {"hip_memcpy_dtod": timed(lambda: dst.copy_(src), 2 * nbytes),
           "plain_dwordx4_copy_kernel": timed(lambda: PL.purlin_stream_copy(dst, src), 2 * nbytes)}
    mixes = (
        ("read_only", [], [src], nbytes),
        ("write_only", [dst], [], nbytes),
        ("copy_1to1", [dst], [src], 2 * nbytes),
        ("reduce_shape_8to1", [dsts8[0]], srcs8, 9 * part),
        ("gather_shape_1to8", dsts8, [srcs8[0]], 9 * part),
    )
    for name, ds, ss, moved in mixes:
        by = {}
        for ntl in (False, True):
            for nts in (False, True):
                if (not ss and ntl) or (not ds and nts):
                    continue  # the hint has nothing to act on
                key = ("nt" if ntl else "cached") + "_loads_" + ("nt" if nts else "cached") + "_stores"
                by[key] = timed(lambda ds=ds, ss=ss, ntl=ntl, nts=nts: PL.purlin_stream(ds, ss, sink=sink, nt_load=ntl,
                                                                                      nt_store=nts), moved)
        best = max(by, key=lambda k: by[k]["GBps"])
        out[name] = dict(by[best], hints=best, by_hints=by)
    out["bytes_copied"] = nbytes
    del src, dst, srcs8, dsts8, sink
    return out


def measure_in_step_streams(torch, PL, rs_plan, ag_plan, ins, rs_out, ag_out, x, y, packed, comb_out, T, H, K,
                            per_op, steps):
    """The MoE ops against plain streams of their own access mix, timed in
    their place in the step: the same ReduceScatter and AllGather run first
    (their 2 GiB streams evict the token matrix from the last-level cache, as
    in the step), then the pack's mix (the token matrix, T x H, read once and
    written to K destinations of T x H each: the packed buffer's K
    consecutive slices, cached loads and non-temporal stores as the pack's
    rows kernel) and the combine's mix (K sources of T x H, the expert
    outputs' slices, into one T x H output, non-temporal loads and stores as
    the combine), with the step's events between all four ops.  The streams
    move the rows' bytes in sequential order, so an op's ratio to its stream
    is what its own access order costs."""
    nb = T * H * 2
    dsts = [packed[i * T:(i + 1) * T] for i in range(K)]
    srcs = [y[i * T:(i + 1) * T] for i in range(K)]
    evs = [[TimingEvent(torch) for _ in range(5)] for _ in range(steps)]
    for i in range(steps + 2):
        ev = evs[i - 2] if i >= 2 else None  # two untimed passes first
        if ev:
            ev[0].record()
        rs_plan.exec(ins, rs_out)
        if ev:
            ev[1].record()
        ag_plan.exec(rs_out, ag_out)
        if ev:
            ev[2].record()
        PL.purlin_stream(dsts, [x], nbytes=nb, nt_load=False, nt_store=True)
        if ev:
            ev[3].record()
        PL.purlin_stream([comb_out], srcs, nbytes=nb, nt_load=True, nt_store=True)
        if ev:
            ev[4].record()
    torch.cuda.synchronize()
    out = {}
    for name, j, desc in (("moe_pack", 2, f"1 source ({nb} B) -> {K} destinations, cached loads, nt stores"),
                          ("moe_combine", 3, f"{K} sources ({nb} B each) -> 1 destination, nt loads, nt stores")):
        ts = [e[j].elapsed_time(e[j + 1]) * 1e3 for e in evs]
        us = float(np.mean(ts))
        moved = (K + 1) * nb
        op = per_op[name]
        out[name] = {"stream": desc, "bytes": moved, "avg_us": round(us, 2), "median_us": round(float(np.median(ts)), 2),
                     "GBps": round(moved / (us * 1e-6) / 1e9, 1),
                     "frac_of_hbm_peak": round(moved / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                     "op_avg_us": op["avg_us"], "op_over_stream": round(op["avg_us"] / us, 4)}
    return out


def measure_pack_status_in_step(torch, PL, rs_plan, ag_plan, ins, rs_out, ag_out, x, ids, y, g, pack_out, comb_out,
                                ws, E, P, steps):
    """The pack in its step place with and without the status word
    (dev_status: every token checked for repeated ids, every id for range),
    alternating step by step, events around the pack only."""
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    ts = {False: [], True: []}
    for i in range(2 * steps + 2):
        with_status = bool(i % 2)
        ev = [TimingEvent(torch) for _ in range(2)]
        rs_plan.exec(ins, rs_out)
        ag_plan.exec(rs_out, ag_out)
        ev[0].record()
        PL.purlin_pack(x, ids, E, P, out=pack_out, workspace=ws, dev_status=st if with_status else None)
        ev[1].record()
        PL.purlin_unpack(y, pack_out["pos"], g, out=comb_out)
        torch.cuda.synchronize()
        if i >= 2:  # one untimed pass of each first
            ts[with_status].append(ev[0].elapsed_time(ev[1]) * 1e3)
    out = {name: {"avg_us": round(float(np.mean(ts[k])), 2), "median_us": round(float(np.median(ts[k])), 2)}
           for name, k in (("without_status", False), ("with_status", True))}
    out["status"] = int(st.item())
    out["cost_us"] = round(out["with_status"]["avg_us"] - out["without_status"]["avg_us"], 2)
    return out


def _round_robin_fraction(recs):
    """Fraction of workgroups b on XCD (b + c) % 8 for the dispatch's most
    common offset c: the hardware deals consecutive workgroups to consecutive
    XCDs, starting where the previous dispatch stopped."""
    off = (recs[:, 0] - np.arange(recs.shape[0])) % 8
    return float(np.bincount(off.astype(np.int64), minlength=8).max() / len(off))


def _xcd_summary(PL, rate, recs):
    fin = PL.xcd_finish_times(rate, recs)
    ends = [fin[k]["end_us"] for k in sorted(fin)]
    return {"span_us": round(max(ends), 2),
            "xcd_round_robin": _round_robin_fraction(recs),
            "xcd_end_us": {str(k): round(fin[k]["end_us"], 2) for k in sorted(fin)},
            "xcd_meta_us": {str(k): round(fin[k]["meta_us"], 2) for k in sorted(fin)},
            "mean_xcd_end_us": round(float(np.mean(ends)), 2),
            "first_to_last_xcd": round(max(ends) - min(ends), 2)}


def measure_xcd_balance(torch, PL, rs_plan, ag_plan, ins, rs_out, ag_out, x, ids, y, g, pack_out, comb_out, T, H,
                        E, K, P, reps=6):
    """When each of the chip's XCDs (accelerator dies, dealt consecutive
    workgroups round-robin) finishes its share of the pack, in the pack's place in the step
    (after the same ReduceScatter and AllGather; the one-launch pack with its
    timing record, purlin_pack_timed), and of plain streams of the pack's and
    the combine's access mix of the same size run back to back.  Each
    workgroup's end is the wall clock once all its stores have completed; an
    XCD's end is its last workgroup's; times from the first workgroup's
    entry, the median over `reps` runs per XCD."""
    log("bench: XCD finishing times")
    if not PL.purlin_pack_single_launch(T, H, K, E):
        return None
    runs = []
    rec = None
    for i in range(reps + 1):
        rs_plan.exec(ins, rs_out)
        ag_plan.exec(rs_out, ag_out)
        rec, groups = PL.purlin_pack_timed(x, ids, E, P, pack_out, rec=rec)
        PL.purlin_unpack(y, pack_out["pos"], g, out=comb_out)
        torch.cuda.synchronize()
        if i:  # the first run is a warm-up
            runs.append(_xcd_summary(PL, *PL._timed_records(rec, groups)))
    out = {"pack_in_step": _median_runs(runs)}
    nb = T * H * 2
    dsts = [pack_out["packed"][i * T:(i + 1) * T] for i in range(K)]
    srcs = [y[i * T:(i + 1) * T] for i in range(K)]
    for name, dd, ss, ntl, nts in (("stream_1to8_pack_size", dsts, [x], False, True),
                                   ("stream_8to1_combine_size", [comb_out], srcs, True, True),
                                   ("stream_write_only_packed_size", [pack_out["packed"]], [], False, True)):
        nbytes = nb * K if name.startswith("stream_write") else nb
        runs = []
        for i in range(reps + 1):
            r = PL.purlin_stream_timed(dd, ss, nbytes=nbytes, nt_load=ntl, nt_store=nts)
            if i:
                runs.append(_xcd_summary(PL, *r))
        out[name] = _median_runs(runs)
    return out


def _median_runs(runs):
    """Per-field medians of several _xcd_summary results."""
    m = {k: round(float(np.median([r[k] for r in runs])), 2) for k in ("span_us", "mean_xcd_end_us",
                                                                        "first_to_last_xcd")}
    m["xcd_round_robin"] = min(r["xcd_round_robin"] for r in runs)
    for key in ("xcd_end_us", "xcd_meta_us"):
        m[key] = {x: round(float(np.median([r[key][x] for r in runs])), 2) for x in runs[0][key]}
    m["runs"] = len(runs)
    return m


def measure_latency(torch, PL, W, graph_latency_us, sweep_sizes):
    # The floor: the smallest launch the library makes (a 16-byte copy, one
    # wavefront's worth of a workgroup), timed like the collectives below.
    a16 = torch.zeros(16, dtype=torch.uint8, device="cuda")
    b16 = torch.empty_like(a16)
    floor_us = graph_call_us(torch, lambda st: PL.purlin_stream_copy(b16, a16, stream=st))
    c1 = W.AR_P4_FP32_256K
    in1 = [to_dev(torch, a) for a in W.collective_inputs(c1)]
    out1 = [torch.empty(c1.count, dtype=torch.float32, device="cuda") for _ in range(c1.P)]
    ar1 = PL.Plan("allreduce", c1.P, c1.count, "fp32", c1.chunk)
    lat1_us = graph_latency_us(ar1, in1, out1)
    del in1, out1
    c2 = W.AR_P8_BF16_DECODE
    lat_in = [to_dev(torch, a) for a in W.collective_inputs(c2)]
    lat_out = [torch.empty(c2.count, dtype=torch.int16, device="cuda") for _ in range(c2.P)]
    ar2 = PL.Plan("allreduce", c2.P, c2.count, "bf16", c2.chunk)
    lat_us = graph_latency_us(ar2, lat_in, lat_out)
    # without a graph (plan bound to its buffers once): back-to-back eager
    # calls, and one call after the stream drained
    run = ar2.bind(lat_in, lat_out)
    run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(100):
        run()
    e1.record()
    torch.cuda.synchronize()
    eager_us = e0.elapsed_time(e1) * 1e3 / 100
    singles = []
    for _ in range(20):
        torch.cuda.synchronize()
        e0.record()
        run()
        e1.record()
        torch.cuda.synchronize()
        singles.append(e0.elapsed_time(e1) * 1e3)
    latency = {
        "launch_floor_us": round(floor_us, 2),
        "launch_floor": "purlin_stream_copy of 16 bytes, graph of 128 calls, 8 replays (time / 1024)",
        "allreduce_p4_fp32_262144": {
            "us": round(lat1_us, 2),
            "over_floor_us": round(lat1_us - floor_us, 2),
            "GBps_min": round(collective_bytes("allreduce", c1.P, c1.count, 4) / (lat1_us * 1e-6) / 1e9, 1),
            "algbw_GBps": round(c1.count * 4 / (lat1_us * 1e-6) / 1e9, 1),
            "timing": "graph of 128 calls, 8 replays after one warm-up replay (time / 1024)",
        },
        "allreduce_p8_bf16_128x8192": {
            "us": round(lat_us, 2),
            "over_floor_us": round(lat_us - floor_us, 2),
            "GBps_min": round(collective_bytes("allreduce", c2.P, c2.count, 2) / (lat_us * 1e-6) / 1e9, 1),
            "algbw_GBps": round(c2.count * 2 / (lat_us * 1e-6) / 1e9, 1),
            "timing": "graph of 128 calls, 8 replays after one warm-up replay (time / 1024)",
            "eager_via": "Plan.bind (buffers validated once)",
            "eager_back_to_back_us": round(eager_us, 2),
            "single_call_us": round(float(np.median(singles)), 2),
        }
    }
    if sweep_sizes:
        # the paper's latency sweep (Section 5): 1 KiB..512 KiB per rank (the
        # scattered side: AllReduce/ReduceScatter/AllToAll input, AllGather
        # output), P = 8, bf16, chunk 64 KiB; graph-replayed as above
        sweep = {}
        for op in ("allreduce", "reduce_scatter", "allgather", "alltoall"):
            row = {}
            for kib in (1, 2, 4, 8, 16, 32, 64, 128, 256, 512):
                n = kib * 1024 // 2
                li = [torch.randn(n, device="cuda").to(torch.bfloat16).view(torch.int16) for _ in range(8)]
                lo = [torch.empty(n, dtype=torch.int16, device="cuda") for _ in range(8)]
                if op == "reduce_scatter":
                    lo = [t[: n // 8] for t in lo]
                elif op == "allgather":
                    li = [t[: n // 8] for t in li]
                pl = PL.Plan(op, 8, n, "bf16", 65536)
                row[f"{kib}KiB"] = round(graph_latency_us(pl, li, lo), 2)
            sweep[op] = row
        latency["sweep_p8_bf16_us"] = sweep
        latency["sweep_p8_bf16_over_floor_us"] = {op: {k: round(v - floor_us, 2) for k, v in row.items()}
                                                  for op, row in sweep.items()}
    del lat_in, lat_out
    return latency


def emit(args, value, ms_per_step, step_bytes, P, N, T, H, E, K, roofline, cpu, per_op, latency, plan_ms, dev_name,
         src_hash, extra, ceilings=None, in_step=None):
    result = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "accumulate": "f32",  # reductions and the combine add in binary32; copies move bf16 bits
        "data": "synthetic (seeded; shapes of the paper's prefill collectives and MoE dispatch/combine)",
        "config": {
            "workload": "ReduceScatter then AllGather P=8 bf16 256MiB/rank chunk 1MiB; MoE pack + combine "
                        "4096x7168 bf16, E=256 over P=8, top-8 Zipf(1.1)",
            "ranks_simulated": P,
            "elements_per_rank": N,
            "moe": {"T": T, "H": H, "E": E, "K": K},
            "step_bytes_min": step_bytes,
        },
        "frac_of_hbm_peak": round(value / HBM_PEAK_GBS, 4),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "ops": per_op,
        "latency_us": latency,
        "other_ops_256MiB_per_rank": extra,
        "copy_ceilings": ceilings,
        "in_step_streams": in_step,
        "plan_ms": round(plan_ms, 3),
        "device": dev_name,
        "kernel_source_hash": src_hash,
    }
    print(json.dumps(result), flush=True)
    return 0


def cpu_baseline(torch, ins_np, rs_out, ag_out, x_np, ids_np, y_np, g_np, pack_out, comb_out, P, N, M, E, K):
    """Time the oracle (as it stands, single-threaded numpy) on a bounded
    sample of the same step, and compare the GPU's outputs on that sample."""
    import oracle

    def down(t, dt):
        return t.contiguous().view(torch.uint8).cpu().numpy().view(dt)

    log("bench: cpu baseline (oracle on a sample)")
    from paper_2609_36954_amd import workloads as W

    t_start = time.perf_counter()
    max_ulp = 0

    def ulp_gap(got, want):
        """Largest distance in bf16 ulps (both as bf16 encodings)."""
        def ordered(b):
            b = b.astype(np.int32)
            return np.where(b & 0x8000, 0x8000 - (b & 0x7FFF), 0x8000 + b)
        return int(np.abs(ordered(got) - ordered(want)).max()) if got.size else 0
    frac = 1  # the whole of each partition of the collectives
    m = M // frac
    ok = True
    t_total, bytes_total = 0.0, 0
    reps = 3  # every op: the median of three runs

    def median_time(fn):
        times, res = [], None
        for _ in range(reps):
            t = time.perf_counter()
            res = fn()
            times.append(time.perf_counter() - t)
        return sorted(times)[reps // 2], res

    # ReduceScatter on the first m elements of every partition
    sub = [np.concatenate([a[k * M:k * M + m] for k in range(P)]) for a in ins_np]
    dt, rs_want = median_time(lambda: oracle.reduce_scatter(sub, "bf16"))
    t_total += dt
    bytes_total += collective_bytes("reduce_scatter", P, P * m, 2)
    per_op = {"reduce_scatter": {"bytes": collective_bytes("reduce_scatter", P, P * m, 2), "seconds": dt}}
    for r in range(P):
        got = down(rs_out[r][:m], np.uint16)
        ok &= bool(np.array_equal(got, rs_want[r]))
        max_ulp = max(max_ulp, ulp_gap(got, rs_want[r]))
    # AllGather of those
    dt, ag_want = median_time(lambda: oracle.all_gather(rs_want, "bf16"))
    t_total += dt
    bytes_total += collective_bytes("allgather", P, P * m, 2)
    per_op["allgather"] = {"bytes": collective_bytes("allgather", P, P * m, 2), "seconds": dt}
    for r in (0, P - 1):
        got = np.concatenate([down(ag_out[r][k * M:k * M + m], np.uint16) for k in range(P)])
        ok &= bool(np.array_equal(got, ag_want[r]))
    # MoE pack and combine of all 4096 tokens
    T = ids_np.shape[0]
    Ts = T
    H = x_np.shape[1]
    dt, pw = median_time(lambda: oracle.pack(x_np, ids_np, E, P))
    t_pack_single = dt
    t_total += dt
    bytes_total += pack_bytes(T, H, K, E, P)
    per_op["moe_pack"] = {"bytes": pack_bytes(T, H, K, E, P), "seconds": dt}
    pos_want = pw["pos"]
    ok &= bool(np.array_equal(down(pack_out["pos"], np.int32).reshape(-1, K), pos_want))
    for key in ("dest_counts", "dest_offsets", "expert_counts", "expert_offsets"):
        ok &= bool(np.array_equal(down(pack_out[key], np.int32), pw[key]))
    rows = np.random.default_rng(0).choice(T * K, 256, replace=False)
    ok &= bool(np.array_equal(down(pack_out["packed"], np.uint16).reshape(T * K, H)[rows], pw["packed"][rows]))
    del pw
    dt, cw = median_time(lambda: oracle.unpack(y_np, pos_want[:Ts], g_np[:Ts]))
    t_total += dt
    bytes_total += unpack_bytes(Ts, H, K)
    per_op["moe_combine"] = {"bytes": unpack_bytes(Ts, H, K), "seconds": dt}
    got = down(comb_out[:Ts], np.uint16).reshape(Ts, H)
    ok &= bool(np.array_equal(got, cw))
    max_ulp = max(max_ulp, ulp_gap(got, cw))
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()

    # (ii) the same oracle functions over element blocks in a thread pool, one
    # thread per core this process may run on (numpy releases the GIL inside
    # its loops).  The per-element order is unchanged, so the results are the
    # single-threaded ones bit for bit.  Pack's positions come from a scan over
    # all tokens, so pack runs single-threaded in both.
    from concurrent.futures import ThreadPoolExecutor

    from oracle.collectives import rank_order_sum

    nthr = max(1, min(cores, 64))
    nblk = 4 * nthr

    def cuts(n):
        return [(n * j // nblk, n * (j + 1) // nblk) for j in range(nblk)]

    def pooled(jobs):
        with ThreadPoolExecutor(nthr) as ex:
            return list(ex.map(lambda f: f(), jobs))

    rs_jobs = [(r, lo, hi) for r in range(P) for lo, hi in cuts(m)]
    dt_rs, rs_blocks = median_time(lambda: pooled(
        [lambda r=r, lo=lo, hi=hi: rank_order_sum([sub[p][r * m + lo:r * m + hi] for p in range(P)], "bf16")
         for r, lo, hi in rs_jobs]))
    thr_ok = all(np.array_equal(b, rs_want[r][lo:hi]) for (r, lo, hi), b in zip(rs_jobs, rs_blocks))
    del rs_blocks
    ag_jobs = cuts(m)
    dt_ag, ag_blocks = median_time(lambda: pooled(
        [lambda lo=lo, hi=hi: oracle.all_gather([rs_want[p][lo:hi] for p in range(P)], "bf16") for lo, hi in ag_jobs]))
    for (lo, hi), b in zip(ag_jobs, ag_blocks):
        for r in (0, P - 1):
            thr_ok &= bool(np.array_equal(b[r], ag_want[r].reshape(P, m)[:, lo:hi].reshape(-1)))
    del ag_blocks
    un_jobs = cuts(Ts)
    dt_un, un_blocks = median_time(lambda: pooled(
        [lambda lo=lo, hi=hi: oracle.unpack(y_np, pos_want[lo:hi], g_np[lo:hi]) for lo, hi in un_jobs]))
    thr_ok &= all(np.array_equal(b, cw[lo:hi]) for (lo, hi), b in zip(un_jobs, un_blocks))
    del un_blocks
    t_pack = t_pack_single
    t_threaded = dt_rs + dt_ag + t_pack + dt_un
    for name, dt_thr in (("reduce_scatter", dt_rs), ("allgather", dt_ag), ("moe_pack", t_pack),
                         ("moe_combine", dt_un)):
        e = per_op[name]
        e["seconds_threaded"] = dt_thr
        e["GBps"] = round(e["bytes"] / e["seconds"] / 1e9, 3)
        e["GBps_threaded"] = round(e["bytes"] / dt_thr / 1e9, 3)
        e["seconds"] = round(e["seconds"], 4)
        e["seconds_threaded"] = round(dt_thr, 4)

    # the two small AllReduce workloads, whole, single-threaded (not in the step)
    small = {}
    for cfg in (W.AR_P4_FP32_256K, W.AR_P8_BF16_DECODE):
        ins_c = W.collective_inputs(cfg)
        es = 4 if cfg.dtype == "fp32" else 2
        dt_c, _ = median_time(lambda: oracle.all_reduce(ins_c, cfg.dtype))
        small[cfg.name] = {"seconds": round(dt_c, 4),
                           "GBps": round(collective_bytes("allreduce", cfg.P, cfg.count, es) / dt_c / 1e9, 3)}

    def sha(arrays):
        h = hashlib.sha256()
        for a in arrays:
            h.update(np.ascontiguousarray(a).view(np.uint8).reshape(-1))
        return h.hexdigest()

    return {
        "value": round(bytes_total / t_total / 1e9, 3),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"the whole step: ReduceScatter+AllGather of 256 MiB/rank (P=8, bf16) and MoE pack and "
                  f"combine of all {T} tokens; each op the median of {reps} runs",
        "seconds": round(t_total, 3),
        "cpu_seconds_spent": round(time.perf_counter() - t_start, 1),
        "host_cores_available": cores,
        "os_cpu_count": os.cpu_count(),
        "cpu": cpu_model(),
        "numpy": np.__version__,
        "gpu_matches_oracle_on_sample": ok,
        "max_bf16_ulp_on_sample": max_ulp,  # ReduceScatter and combine outputs against the oracle
        "small_allreduce": small,
        "per_op": per_op,  # single-threaded and pooled seconds of each op's sample (pack single-threaded in both)
        "threaded": {
            "value": round(bytes_total / t_threaded / 1e9, 3),
            "unit": "GB/s",
            "cores": nthr,
            "seconds": round(t_threaded, 3),
            "how": f"ReduceScatter, AllGather and combine over {nblk} element blocks each in a pool of {nthr} "
                   "threads; pack single-threaded (its positions need a scan over all tokens); median of 3",
            "identical_to_single_threaded": bool(thr_ok),
        },
        "input_sha256": {
            "rs_inputs_8_ranks": sha(ins_np),
            "moe_x": sha([x_np]),
            "moe_ids": sha([ids_np]),
            "moe_y": sha([y_np]),
            "moe_gates": sha([g_np]),
        },
    }


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo where there is one)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


if __name__ == "__main__":
    sys.exit(main())
