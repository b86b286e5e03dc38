"""The library driven from a plain C program on the GPU.

``tests/c_abi_gpu_program.c`` includes only ``include/purlin.h`` and the HIP
runtime's C API; it is built here with the system C compiler and linked
against ``libpurlin.so``, so no Python and no torch sit between the caller
and the kernels.  It runs the two small AllReduce workloads whole, a
ReduceScatter, an AllGather and an AllToAll with ragged partitions, and a
pack followed by a combine, on inputs this test writes; every output must
equal the oracle's bit for bit.
"""

import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from paper_2609_36954_amd import purlin as PL
from paper_2609_36954_amd import workloads as W

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.fixture(scope="module")
def program(tmp_path_factory):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    assert os.path.exists(PL.LIB_PATH), "library not built"
    exe = tmp_path_factory.mktemp("c_program") / "purlin_c"
    cmd = [gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c_abi_gpu_program.c"), PL.LIB_PATH,
           f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-Wl,-rpath," + os.path.dirname(PL.LIB_PATH),
           "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    return str(exe)


def _inputs(P, n, dtype, seed):
    rng = np.random.default_rng(seed)
    if dtype == "fp32":
        return [rng.uniform(-1, 1, n).astype(np.float32) for _ in range(P)]
    return [oracle.narrow(rng.standard_normal(n).astype(np.float32)) for _ in range(P)]


def _want(op, ins, dtype):
    if op == "allgather":
        M = len(ins[0]) // len(ins)
        return oracle.all_gather([a[:M] for a in ins], dtype)
    return {"allreduce": oracle.all_reduce, "reduce_scatter": oracle.reduce_scatter,
            "alltoall": oracle.all_to_all}[op](ins, dtype)


def test_c_program_matches_oracle(program, tmp_path):
    cases = [
        ("allreduce", W.AR_P4_FP32_256K.P, W.AR_P4_FP32_256K.count, "fp32", W.AR_P4_FP32_256K.chunk,
         W.collective_inputs(W.AR_P4_FP32_256K)),
        ("allreduce", W.AR_P8_BF16_DECODE.P, W.AR_P8_BF16_DECODE.count, "bf16", W.AR_P8_BF16_DECODE.chunk,
         W.collective_inputs(W.AR_P8_BF16_DECODE)),
        ("reduce_scatter", 8, 8 * 1003, "bf16", 96, _inputs(8, 8 * 1003, "bf16", 1)),
        ("allgather", 3, 3 * 1001, "fp32", 64, _inputs(3, 3 * 1001, "fp32", 2)),
        ("alltoall", 5, 5 * 777, "bf16", 256, _inputs(5, 5 * 777, "bf16", 3)),
    ]
    jobs = []
    for i, (op, P, count, dtype, chunk, ins) in enumerate(cases):
        in_elems = count // P if op == "allgather" else count
        for p, a in enumerate(ins):
            (tmp_path / f"c{i}_in{p}.bin").write_bytes(np.ascontiguousarray(a[:in_elems]).tobytes())
        jobs.append(f"coll {op} {P} {count} {dtype} {chunk} {tmp_path}/c{i}_")

    T, H, K, E, PM = 300, 520, 8, 64, 8
    rng = np.random.default_rng(4)
    x = oracle.narrow(rng.standard_normal((T, H)).astype(np.float32))
    ids = W.zipf_topk_ids(T, E, K, 1.1, seed=4).astype(np.int32)
    y = oracle.narrow(rng.standard_normal((T * K, H)).astype(np.float32))
    g = W.softmax_gates(T, K, 5).astype(np.float32)
    for name, a in (("x", x), ("ids", ids), ("y", y), ("g", g)):
        (tmp_path / f"m_{name}.bin").write_bytes(np.ascontiguousarray(a).tobytes())
    jobs.append(f"moe {T} {H} {K} {E} {PM} {tmp_path}/m_")

    r = subprocess.run([program], input="\n".join(jobs) + "\n", capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr

    for i, (op, P, count, dtype, chunk, ins) in enumerate(cases):
        want = _want(op, ins, dtype)
        bits = np.uint32 if dtype == "fp32" else np.uint16
        for q in range(P):
            got = np.frombuffer((tmp_path / f"c{i}_out{q}.bin").read_bytes(), dtype=bits)
            assert np.array_equal(got, want[q].view(bits)), (op, P, q)

    pw = oracle.pack(x, ids, E, PM)
    packed = np.frombuffer((tmp_path / "m_packed.bin").read_bytes(), dtype=np.uint16).reshape(T * K, H)
    pos = np.frombuffer((tmp_path / "m_pos.bin").read_bytes(), dtype=np.int32).reshape(T, K)
    meta = np.frombuffer((tmp_path / "m_meta.bin").read_bytes(), dtype=np.int32)
    assert np.array_equal(packed, pw["packed"])
    assert np.array_equal(pos, pw["pos"])
    assert np.array_equal(meta[:PM], pw["dest_counts"])
    assert np.array_equal(meta[PM:2 * PM], pw["dest_offsets"])
    assert np.array_equal(meta[2 * PM:2 * PM + E], pw["expert_counts"])
    assert np.array_equal(meta[2 * PM + E:2 * PM + 2 * E], pw["expert_offsets"])
    assert meta[-1] == 0
    out = np.frombuffer((tmp_path / "m_out.bin").read_bytes(), dtype=np.uint16).reshape(T, H)
    assert np.array_equal(out, oracle.unpack(y, pw["pos"], g))
