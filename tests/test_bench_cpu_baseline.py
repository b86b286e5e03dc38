"""bench.py's CPU-baseline leg, run on the CPU with small shapes.

Given outputs that hold the oracle's own results it must report a match at
0 ulp and a per-op breakdown whose bytes and seconds add up to the step's
figure; one wrong bf16 code in the combine output must flip the verdict
and show as a nonzero ulp gap.  (Seconds are rounded in the report, so
the bytes are checked exactly and the times only for their sum.)
"""

import numpy as np
import torch

import bench
import oracle
from paper_2609_36954_amd import workloads as W


def _case():
    P, M = 4, 96
    N = P * M
    rng = np.random.default_rng(5)
    ins = [W.normal_bf16(rng, N) for _ in range(P)]
    rs = oracle.reduce_scatter(ins, "bf16")
    ag = oracle.all_gather(rs, "bf16")
    T, H, E, K = 160, 32, 8, 2  # T * K >= the 256 packed rows the baseline samples
    ids = W.zipf_topk_ids(T, E, K, 1.1, seed=1)
    x = W.normal_bf16(rng, T * H).reshape(T, H)
    y = W.normal_bf16(rng, T * K * H).reshape(T * K, H)
    g = W.softmax_gates(T, K, 2)
    pw = oracle.pack(x, ids, E, P)
    cw = oracle.unpack(y, pw["pos"], g)

    def t16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16).copy())

    pack_out = {k: torch.from_numpy(np.ascontiguousarray(pw[k]).astype(np.int32))
                for k in ("dest_counts", "dest_offsets", "expert_counts", "expert_offsets", "pos")}
    pack_out["packed"] = t16(pw["packed"])
    args = dict(ins_np=ins, rs_out=[t16(r) for r in rs], ag_out=[t16(a) for a in ag], x_np=x, ids_np=ids, y_np=y,
                g_np=g, pack_out=pack_out, comb_out=t16(cw), P=P, N=N, M=M, E=E, K=K)
    return args


def test_baseline_reports_a_match_and_a_consistent_breakdown():
    a = _case()
    r = bench.cpu_baseline(torch, **a)
    assert r["kind"] == "oracle" and r["cores"] == 1
    assert r["gpu_matches_oracle_on_sample"] is True
    assert r["max_bf16_ulp_on_sample"] == 0
    assert r["threaded"]["identical_to_single_threaded"] is True
    per = r["per_op"]
    assert set(per) == {"reduce_scatter", "allgather", "moe_pack", "moe_combine"}
    total_bytes = sum(e["bytes"] for e in per.values())
    total_s = sum(e["seconds"] for e in per.values())
    assert abs(total_s - r["seconds"]) < 1e-3 + 1e-3 * r["seconds"]
    P, N, E, K = a["P"], a["N"], a["E"], a["K"]
    T, H = a["x_np"].shape
    assert total_bytes == (bench.collective_bytes("reduce_scatter", P, N, 2) + bench.collective_bytes("allgather", P, N, 2)
                           + bench.pack_bytes(T, H, K, E, P) + bench.unpack_bytes(T, H, K))
    assert per["moe_pack"]["seconds_threaded"] == per["moe_pack"]["seconds"]  # pack runs single-threaded in both


def test_one_wrong_code_flips_the_verdict():
    a = _case()
    a["comb_out"][3, 5] ^= 1  # one bf16 ulp away in the last place
    r = bench.cpu_baseline(torch, **a)
    assert r["gpu_matches_oracle_on_sample"] is False
    assert r["max_bf16_ulp_on_sample"] >= 1
