"""GPU parity of the de-duplicated dispatch (one row per token and
destination rank) and its combine with the oracle, alone and as an
expert-parallel round trip over P simulated ranks through AllToAllV.

Dispatch is integer and bit-copy work: bit-exact.  The combine adds bf16
rows in rank order in FP32 on both sides: bit-exact as well.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_util import Guarded, assert_bits_equal, to_device, to_host
from paper_2609_36954_amd import purlin as PL
from paper_2609_36954_amd import workloads as W

pytestmark = pytest.mark.gpu


def _distinct_ids(rng, T, K, E):
    return np.stack([rng.permutation(E)[:K] for _ in range(T)]).astype(np.int32) if T else np.zeros((0, K), np.int32)


def run_pack_dedup(x_np, ids_np, E, P):
    T, H = x_np.shape
    K = ids_np.shape[1]
    R = T * min(K, P)
    packed = Guarded(R * H * 2, torch.int16)
    row_of = Guarded(T * P * 4, torch.int32)
    st = torch.full((4,), 7, dtype=torch.int32, device="cuda")
    out = dict(packed=packed.t.view(R, H), row_of=row_of.t.view(T, P))
    r = PL.purlin_pack_dedup(to_device(x_np), to_device(ids_np), E, P, out=out, dev_status=st)
    torch.cuda.synchronize()
    assert packed.intact() and row_of.intact()
    got = {k: to_host(v, np.uint16 if k == "packed" else np.int32) for k, v in r.items()}
    got["packed"] = got["packed"].reshape(R, H)
    got["row_of"] = got["row_of"].reshape(T, P)
    return got, int(st[0].item())


@pytest.mark.parametrize("T,H,K,E,P,seed", [
    (0, 8, 2, 4, 2, 0),
    (1, 8, 1, 1, 1, 1),
    (5, 16, 2, 4, 2, 2),
    (63, 24, 4, 16, 4, 3),
    (65, 7, 3, 9, 3, 4),  # H not a multiple of 8; ragged last tile
    (130, 520, 8, 64, 8, 5),
    (200, 1000, 6, 96, 16, 6),
    (100, 64, 8, 8, 8, 7),  # E = P: nothing to de-duplicate
    (129, 64, 1, 32, 4, 8),  # K = 1
    # K of 4 to 64, P = 16, larger shapes
    (1, 8, 4, 4, 2, 9),
    (2047, 48, 16, 64, 16, 10),  # K = 16, P = 16
    (512, 16, 64, 64, 16, 11),  # K = 64
    (8192, 16, 4, 64, 16, 12),
    (4700, 7168, 4, 256, 8, 13),  # 64 MiB token matrix
    (300, 520, 8, 64, 4, 14),
    (1000, 64, 32, 128, 8, 15),  # K = 32
    (64, 128, 8, 8, 8, 16),  # E = P
])
def test_pack_dedup_matches_oracle(T, H, K, E, P, seed):
    print(f"pack_dedup T={T} H={H} K={K} E={E} P={P}", flush=True)
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
    ids = _distinct_ids(rng, T, K, E)
    got, status = run_pack_dedup(x, ids, E, P)
    want = oracle.pack_dedup(x, ids, E, P)
    assert status == 0
    for key in ("dest_counts", "dest_offsets", "row_of"):
        assert np.array_equal(got[key], want[key]), key
    R = len(want["packed"])
    assert np.array_equal(got["packed"][:R], want["packed"])


def test_pack_dedup_zipf_routing_matches_oracle():
    T, H, E, P, K = 1000, 256, 256, 8, 8
    ids = W.zipf_topk_ids(T, E, K, 1.1, seed=4)
    x = W.normal_bf16(np.random.default_rng(1), T * H).reshape(T, H)
    got, status = run_pack_dedup(x, ids, E, P)
    want = oracle.pack_dedup(x, ids, E, P)
    assert status == 0
    assert np.array_equal(got["row_of"], want["row_of"])
    assert np.array_equal(got["dest_counts"], want["dest_counts"])
    assert np.array_equal(got["packed"][:len(want["packed"])], want["packed"])


def test_pack_dedup_flags_bad_routing_and_stays_in_bounds():
    T, H, K, E, P = 70, 16, 3, 8, 4
    rng = np.random.default_rng(3)
    ids = _distinct_ids(rng, T, K, E)
    ids[5, 1] = E + 3  # out of range
    ids[66, 2] = ids[66, 0]  # repeated within a token
    ids[10, 0] = -1
    _, status = run_pack_dedup(rng.integers(0, 0x10000, (T, H)).astype(np.uint16), ids, E, P)
    assert status == 1


@pytest.mark.parametrize("T,K,E,P", [(70, 4, 8, 4), (4096, 8, 256, 8)])
def test_pack_dedup_flags_bad_routing_and_ignores_bad_ids(T, K, E, P):
    """Out-of-range ids (positive, negative) are ignored and flagged, a
    repeated id is flagged; the destination sets (and so every output) are
    those of the ids with the bad ones left out."""
    H = 16
    rng = np.random.default_rng(T + K)
    ids = _distinct_ids(rng, T, K, E)
    x = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
    bad = ids.copy()
    bad[5, 1] = E + 3
    bad[10, 0] = -1
    bad[T - 1, 2] = bad[T - 1, 0]  # repeated in the last token: the same set
    got, status = run_pack_dedup(x, bad, E, P)
    assert status == 1
    # the same destination sets without the bad ids: drop them, pad with a kept id of the token
    L = E // P
    want_sets = [set(int(e) // L for e in row if 0 <= e < E) for row in bad]
    counts = np.zeros(P, np.int64)
    row_of = np.full((T, P), -1, np.int64)
    for r in range(P):
        for t in range(T):
            if r in want_sets[t]:
                row_of[t, r] = counts[r]
                counts[r] += 1
    offs = np.concatenate([[0], np.cumsum(counts)[:-1]])
    row_of = np.where(row_of >= 0, row_of + offs[None, :], -1)
    assert np.array_equal(got["dest_counts"], counts)
    assert np.array_equal(got["row_of"], row_of)
    for t in (0, 5, 10, T - 1):
        for r in range(P):
            if row_of[t, r] >= 0:
                assert np.array_equal(got["packed"][row_of[t, r]], x[t])


def run_unpack_dedup(y_np, row_of_np):
    T, P = row_of_np.shape
    H = y_np.shape[1]
    out = Guarded(T * H * 2, torch.int16)
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    PL.purlin_unpack_dedup(to_device(y_np), to_device(row_of_np), out=out.t.view(T, H), dev_status=st)
    torch.cuda.synchronize()
    assert out.intact()
    return to_host(out.t, np.uint16).reshape(T, H), int(st.item())


@pytest.mark.parametrize("T,H,K,E,P,seed", [(1, 8, 1, 2, 2, 0), (64, 520, 8, 64, 8, 1), (77, 7, 3, 12, 4, 2),
                                            (300, 1024, 8, 256, 16, 3), (40, 64, 2, 2, 1, 4)])
def test_unpack_dedup_matches_oracle(T, H, K, E, P, seed):
    rng = np.random.default_rng(seed)
    ids = _distinct_ids(rng, T, K, E)
    row_of = oracle.pack_dedup(np.zeros((T, 1), np.uint16), ids, E, P)["row_of"]
    R = int((row_of >= 0).sum())
    y = oracle.narrow((rng.standard_normal((R, H)) * np.exp2(rng.integers(-30, 30, (R, H)))).astype(np.float32))
    y.reshape(-1)[:: 97] = 0x8000  # negative zeros
    y.reshape(-1)[1:: 89] = 0x0001  # denormals
    got, status = run_unpack_dedup(y, row_of)
    assert status == 0
    assert_bits_equal(got, oracle.unpack_dedup(y, row_of), "bf16", f"unpack_dedup T={T} H={H} P={P}")


def test_unpack_dedup_special_values_and_bad_entries():
    H = 64
    y = np.zeros((6, H), np.uint16)
    y[0] = 0x7F80  # +inf
    y[1] = 0xFF80  # -inf
    y[2] = 0x7FC1  # NaN
    y[3] = 0x7F7F  # largest finite
    y[4] = 0x7F7F
    y[5] = 0x3F80
    # tokens: inf + 1 = inf; inf + -inf = NaN; NaN + 1 = NaN; max + max = inf; no rows = +0
    row_of = np.array([[0, -1, 5], [0, 1, -1], [2, 5, -1], [3, 4, -1], [-1, -1, -1]], np.int32)
    got, status = run_unpack_dedup(y, row_of)
    assert status == 0
    want = oracle.unpack_dedup(y, row_of)
    assert np.array_equal(got[[0, 3, 4]], want[[0, 3, 4]])
    assert got[0, 0] == 0x7F80 and got[3, 0] == 0x7F80 and got[4, 0] == 0
    for t in (1, 2):  # NaN on both sides (the NaN's sign and payload are not compared)
        assert np.all((got[t] & 0x7FFF) > 0x7F80) and np.all((want[t] & 0x7FFF) > 0x7F80)
    bad = row_of.copy()
    bad[1, 2] = 6  # beyond the rows
    bad[3, 2] = -2
    got, status = run_unpack_dedup(y, bad)
    assert status == 1
    assert np.array_equal(got[[0, 3, 4]], want[[0, 3, 4]])  # valid entries still summed


def test_pack_dedup_full_size():
    """T = 4096, H = 7168, E = 256 over P = 8, top-8 Zipf(1.1): metadata
    against the oracle, every row by the row_of property, and the combine of
    the packed rows on sampled tokens."""
    T, H, E, P, K = 4096, 7168, 256, 8, 8
    ids_np = W.zipf_topk_ids(T, E, K, 1.1, seed=4)
    x_np = W.normal_bf16(np.random.default_rng(40), T * H).reshape(T, H)
    x = to_device(x_np)
    r = PL.purlin_pack_dedup(x, to_device(ids_np), E, P)
    torch.cuda.synchronize()
    meta = oracle.pack_dedup(x_np[:, :8], ids_np, E, P)
    assert np.array_equal(to_host(r["row_of"], np.int32).reshape(T, P), meta["row_of"])
    assert np.array_equal(to_host(r["dest_counts"], np.int32), meta["dest_counts"])
    assert np.array_equal(to_host(r["dest_offsets"], np.int32), meta["dest_offsets"])
    row_of = r["row_of"]
    t_idx, r_idx = torch.nonzero(row_of >= 0, as_tuple=True)
    assert torch.equal(r["packed"][row_of[t_idx, r_idx].long()], x[t_idx])
    R = int(meta["dest_counts"].sum())
    out = PL.purlin_unpack_dedup(r["packed"][:R], row_of)
    torch.cuda.synchronize()
    ts = np.sort(np.random.default_rng(2).choice(T, 64, replace=False))
    sub = meta["row_of"][ts]
    rows = sorted(set(sub[sub >= 0].tolist()))
    remap = {q: i for i, q in enumerate(rows)}
    y = to_host(r["packed"], np.uint16).reshape(-1, H)[rows]
    sub2 = np.vectorize(lambda q: remap.get(q, -1))(sub).astype(np.int32)
    assert_bits_equal(to_host(out, np.uint16).reshape(T, H)[ts], oracle.unpack_dedup(y, sub2), "bf16", "sampled")


def test_expert_parallel_dedup_round_trip():
    """P = 8 ranks: de-duplicated pack, AllToAllV of the rows (sizes =
    dest_counts on the device), a stand-in expert per rank (bit flip by
    r + 1), the reverse AllToAllV (counts read column-major) and the
    de-duplicated combine, against the oracle."""
    P, T, H, K, E = 8, 300, 520, 8, 64
    rngs = W.rank_rngs(77, P)
    xs_np = [W.normal_bf16(rngs[p], T * H).reshape(T, H) for p in range(P)]
    ids_np = [W.zipf_topk_ids(T, E, K, 1.1, 700 + p) for p in range(P)]
    rows_in, rows_out = T * min(K, P), P * T * min(K, P)
    counts = torch.zeros((P, P), dtype=torch.int32, device="cuda")
    packs = []
    for p in range(P):
        packs.append(PL.purlin_pack_dedup(to_device(xs_np[p]), to_device(ids_np[p]), E, P,
                                          out=dict(dest_counts=counts[p])))
    fwd = PL.purlin_plan_v("alltoallv", P, rows_in * H, "bf16", 1 << 16, unit=H, out_capacity=rows_out * H)
    bwd = PL.purlin_plan_v("alltoallv", P, rows_out * H, "bf16", 1 << 16, unit=H, out_capacity=rows_in * H,
                           counts_transposed=True)
    recv = [torch.empty(rows_out * H, dtype=torch.int16, device="cuda") for _ in range(P)]
    back = [torch.empty(rows_in * H, dtype=torch.int16, device="cuda") for _ in range(P)]
    fwd.exec_v([pk["packed"].view(-1) for pk in packs], recv, counts.view(-1))
    torch.cuda.synchronize()
    m = to_host(counts, np.int32).reshape(P, P)
    for r in range(P):
        n = int(m[:, r].sum())
        recv[r][: n * H].bitwise_xor_(r + 1)
    bwd.exec_v(recv, back, counts.view(-1))
    outs = [PL.purlin_unpack_dedup(back[p].view(rows_in, H), packs[p]["row_of"]) for p in range(P)]
    torch.cuda.synchronize()
    for p in range(P):
        d = oracle.pack_dedup(xs_np[p], ids_np[p], E, P)
        assert np.array_equal(m[p], d["dest_counts"])
        dest = np.repeat(np.arange(P), d["dest_counts"]).astype(np.uint16)
        y = d["packed"] ^ (dest + 1)[:, None]
        R = len(y)
        assert np.array_equal(to_host(back[p], np.uint16).reshape(rows_in, H)[:R], y), f"rank {p} exchange"
        assert_bits_equal(to_host(outs[p], np.uint16).reshape(T, H), oracle.unpack_dedup(y, d["row_of"]), "bf16",
                          f"rank {p} combine")


def test_dedup_dispatch_and_combine_in_one_graph():
    """pack_dedup and unpack_dedup captured once and replayed with new
    routing: sizes and row indices are formed on the device each replay."""
    T, H, K, E, P = 200, 136, 4, 32, 8
    x = torch.empty((T, H), dtype=torch.int16, device="cuda")
    ids = torch.empty((T, K), dtype=torch.int32, device="cuda")
    packed = torch.empty((T * min(K, P), H), dtype=torch.int16, device="cuda")
    out = dict(packed=packed, dest_counts=torch.empty(P, dtype=torch.int32, device="cuda"),
               dest_offsets=torch.empty(P, dtype=torch.int32, device="cuda"),
               row_of=torch.empty((T, P), dtype=torch.int32, device="cuda"))
    ws = torch.empty(max(PL.purlin_pack_dedup_workspace_size(T, P), 16), dtype=torch.uint8, device="cuda")
    comb = torch.empty((T, H), dtype=torch.int16, device="cuda")
    st = torch.zeros(2, dtype=torch.int32, device="cuda")

    def step(stream=None):
        PL.purlin_pack_dedup(x, ids, E, P, out=out, workspace=ws, dev_status=st[0:1], stream=stream)
        PL.purlin_unpack_dedup(packed, out["row_of"], out=comb, dev_status=st[1:2], stream=stream)

    def load(seed):
        rng = np.random.default_rng(seed)
        xn = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
        xn[(xn & 0x7F80) == 0x7F80] = 0x3F80  # finite values
        idn = _distinct_ids(rng, T, K, E)
        x.copy_(to_device(xn))
        ids.copy_(to_device(idn))
        return xn, idn

    load(0)
    step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            step(stream=side)
    for seed in (1, 2, 3):
        xn, idn = load(seed)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        want = oracle.pack_dedup(xn, idn, E, P)
        assert not st.any().item()
        assert np.array_equal(to_host(out["row_of"], np.int32).reshape(T, P), want["row_of"])
        R = len(want["packed"])
        assert np.array_equal(to_host(packed, np.uint16).reshape(-1, H)[:R], want["packed"])
        assert_bits_equal(to_host(comb, np.uint16).reshape(T, H), oracle.unpack_dedup(want["packed"], want["row_of"]),
                          "bf16", f"replay seed {seed}")
