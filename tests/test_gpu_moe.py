"""GPU parity of MoE pack (dispatch) and unpack (combine) with the oracle.

Pack is integer and bit-copy work: counts, offsets, positions and rows must
match exactly.  Combine follows the slot-order FP32 sum with separately
rounded multiply and add on both sides: bit-exact as well.
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


def run_pack(x_np, ids_np, E, P, status=True):
    T, H = x_np.shape
    K = ids_np.shape[1]
    x = to_device(x_np)
    ids = to_device(ids_np)
    packed = Guarded(T * K * H * 2, torch.int16)
    pos = Guarded(T * K * 4, torch.int32)
    st = torch.full((4,), 7, dtype=torch.int32, device="cuda")
    out = dict(packed=packed.t.view(T * K, H), pos=pos.t.view(T, K))
    r = PL.purlin_pack(x, ids, E, P, out=out, dev_status=st if status else None)
    torch.cuda.synchronize()
    assert packed.intact() and pos.intact()
    host = {k: to_host(v, np.uint16 if k == "packed" else np.int32) for k, v in r.items()}
    host["packed"] = host["packed"].reshape(T * K, H)
    host["pos"] = host["pos"].reshape(T, K)
    return host, int(st[0].item())


def check_pack(x_np, ids_np, E, P):
    got, status = run_pack(x_np, ids_np, E, P)
    want = oracle.pack(x_np, ids_np, E, P)
    assert status == 0
    for key in ("dest_counts", "dest_offsets", "expert_counts", "expert_offsets", "pos"):
        assert np.array_equal(got[key], want[key]), key
    assert np.array_equal(got["packed"], want["packed"])


@pytest.mark.parametrize(
    "T,H,K,E,P,seed",
    [
        (1, 8, 1, 1, 1, 0),
        (5, 16, 2, 4, 2, 1),
        (63, 24, 4, 16, 4, 2),
        (64, 128, 8, 256, 8, 3),
        (65, 7, 3, 9, 3, 4),  # H not a multiple of 8: element path
        (200, 520, 8, 64, 8, 5),
        (333, 1000, 6, 120, 4, 6),
        (130, 64, 64, 64, 8, 7),  # K = 64 (every expert)
        (97, 16, 2, 4096, 16, 8),  # E = 4096
        (0, 64, 8, 256, 8, 9),  # no tokens
        (4096, 24, 8, 256, 8, 12),  # 64 token tiles
        (4097, 24, 8, 256, 8, 13),  # 65 tiles, the last one a single token
        (300, 24, 8, 512, 8, 14),  # 512 experts
        (32768, 8, 1, 16, 4, 15),  # one slot: 512 token tiles
        (1023, 40, 32, 128, 8, 16),  # K = 32: 32736 ids
        (2500, 48, 13, 200, 8, 17),  # K = 13, E = 200, ragged last tile
        (32769, 8, 1, 16, 4, 18),  # 513 tiles, the last one a single token
        (100, 24, 4, 264, 8, 19),  # E = 264
        (600, 7171, 8, 256, 8, 24),  # 8.2 MiB token matrix read ahead, odd rows (element path)
        (4100, 1030, 8, 256, 8, 25),  # 8.1 MiB read ahead, rows not a multiple of 16 bytes
        (8192, 8192, 2, 64, 8, 26),  # 128 MiB: the largest matrix read ahead
        # one launch: limits and ragged edges
        (1, 8, 4, 4, 2, 27),  # T*K = 4, the smallest
        (2499, 48, 13, 200, 8, 28),  # 32487 ids: three after the last 4-id vector
        (100, 24, 4, 1024, 8, 29),  # E = 1024, the largest
        (16448, 16, 1, 256, 4, 30),  # 64 tokens per workgroup, 257 workgroups (two rounds)
        (4700, 7168, 4, 256, 8, 31),  # 18 rows per workgroup (registers), 262 workgroups
        (260, 131072, 8, 256, 8, 32),  # one 256 KiB row per workgroup: 16 vectors per thread
        (512, 8200, 64, 256, 8, 33),  # rows of 1025 vectors (more than the threads), K = 64
        (8000, 24, 4, 1000, 8, 34),  # 32 tokens per workgroup, 250 workgroups
    ],
)
def test_pack_matches_oracle(T, H, K, E, P, seed):
    print(f"pack T={T} H={H} K={K} E={E} P={P} one launch={PL.purlin_pack_single_launch(T, H, K, E)}", flush=True)
    rng = np.random.default_rng(seed)
    ids = _distinct_ids(rng, T, K, E)
    x = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
    check_pack(x, ids, E, P)


@pytest.mark.parametrize("T", [1000, 4096, 4100])
def test_pack_zipf_routing_skewed(T):
    rng = np.random.default_rng(10)
    H, E, P, K = 256, 256, 8, 8
    ids = W.zipf_topk_ids(T, E, K, 1.1, seed=10)
    x = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
    check_pack(x, ids, E, P)


@pytest.mark.parametrize("T,E", [(70, 16), (4200, 16), (70, 1024), (8000, 256), (9000, 256)])
def test_pack_reports_bad_routing(T, E):
    rng = np.random.default_rng(11)
    H, K, P = 16, 4, 4
    x = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
    ids = _distinct_ids(rng, T, K, E)
    rep = ids.copy()
    rep[3, 2] = rep[3, 0]  # repeated id within a token
    _, status = run_pack(x, rep, E, P)
    assert status == 1
    rep = ids.copy()
    rep[T - 1, 1] = rep[T - 1, 0]  # ... in the last (partial) tile
    _, status = run_pack(x, rep, E, P)
    assert status == 1
    oob = ids.copy()
    oob[66, 1] = E  # out of range
    got, status = run_pack(x, oob, E, P)
    assert status == 1
    assert got["pos"][66, 1] == -1
    oob[T - 1, 3] = -5  # negative, in the last token
    got, status = run_pack(x, oob, E, P)
    assert status == 1
    assert got["pos"][66, 1] == -1 and got["pos"][T - 1, 3] == -1
    _, status = run_pack(x, ids, E, P)
    assert status == 0


@pytest.mark.parametrize("T,K,E", [(4096, 8, 256), (500, 6, 64), (2000, 3, 16), (8192, 4, 64), (300, 12, 64)])
def test_pack_one_launch_reports_repeated_ids(T, K, E):
    """The one-launch form checks every token for repeated ids (loaded a
    round of tokens at a time for K <= 8, a plain loop above): a repeat in
    any slot pair of any token, including the first and last token and
    tokens on either side of a round, sets the status word; distinct ids
    leave it 0."""
    H, P = 8, 4
    assert PL.purlin_pack_single_launch(T, H, K, E)
    rng = np.random.default_rng(1000 + T + K)
    x = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
    ids = _distinct_ids(rng, T, K, E)
    _, status = run_pack(x, ids, E, P)
    assert status == 0
    cases = [(0, 1, 0), (T // 2, K - 1, 0), (T - 1, K - 1, K - 2), (min(T - 1, 4095), K - 1, 1), (min(T - 1, 4096), 1, 0)]
    for t, k, k2 in cases:
        rep = ids.copy()
        rep[t, k] = rep[t, k2]
        print(f"repeat at token {t}: slot {k} = slot {k2}", flush=True)
        _, status = run_pack(x, rep, E, P)
        assert status == 1


@pytest.mark.parametrize("T,H,K,E,P,seed", [(4096, 512, 8, 256, 8, 21), (333, 1000, 6, 120, 4, 22), (0, 64, 8, 256, 8, 23)])
def test_pack_split_on_two_streams_matches_pack(T, H, K, E, P, seed):
    """purlin_pack_meta on a side stream, an event, purlin_pack_rows on the
    current stream: every output equals purlin_pack's and the oracle's."""
    rng = np.random.default_rng(seed)
    ids_np = W.zipf_topk_ids(T, E, K, 1.1, seed) if T else np.zeros((0, K), np.int32)
    x_np = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
    want, status = run_pack(x_np, ids_np, E, P)
    assert status == 0
    x, ids = to_device(x_np), to_device(ids_np)
    ws = torch.empty(max(16, PL.purlin_pack_workspace_size(T, K, E)), dtype=torch.uint8, device="cuda")
    g = {"packed": Guarded(T * K * H * 2, torch.int16), "pos": Guarded(T * K * 4, torch.int32),
         "dest_counts": Guarded(P * 4, torch.int32), "dest_offsets": Guarded(P * 4, torch.int32),
         "expert_counts": Guarded(E * 4, torch.int32), "expert_offsets": Guarded(E * 4, torch.int32)}
    out = {k: v.t for k, v in g.items()}
    out["packed"] = out["packed"].view(T * K, H)
    out["pos"] = out["pos"].view(T, K)
    st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    PL.purlin_pack_meta(ids, E, P, out, ws, dev_status=st, stream=side)
    done = torch.cuda.Event()
    done.record(side)
    torch.cuda.current_stream().wait_event(done)
    PL.purlin_pack_rows(x, ids, E, out, ws)
    torch.cuda.synchronize()
    assert all(v.intact() for v in g.values())
    assert int(st[0].item()) == 0
    for key in want:
        got = to_host(g[key].t, np.uint16 if key == "packed" else np.int32).reshape(want[key].shape)
        assert np.array_equal(got, want[key]), key
    ref = oracle.pack(x_np, ids_np, E, P)
    assert np.array_equal(want["packed"], ref["packed"]) and np.array_equal(want["pos"], ref["pos"])


@pytest.mark.parametrize("fill", [0xFF, 0x00, 0x5A])
def test_pack_on_uncleared_workspace_and_again(fill):
    """The workspace's contents on entry do not matter: filled with a byte
    pattern, then reused for a second routing; each call matches the oracle."""
    T, H, K, E, P = 1000, 256, 8, 256, 8
    ws = torch.full((PL.purlin_pack_workspace_size(T, K, E),), fill, dtype=torch.uint8, device="cuda")
    for seed in (31, 32):
        rng = np.random.default_rng(seed)
        ids_np = W.zipf_topk_ids(T, E, K, 1.1, seed)
        x_np = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
        st = torch.full((1,), 7, dtype=torch.int32, device="cuda")
        r = PL.purlin_pack(to_device(x_np), to_device(ids_np), E, P, workspace=ws, dev_status=st)
        torch.cuda.synchronize()
        assert int(st[0].item()) == 0
        want = oracle.pack(x_np, ids_np, E, P)
        for key in ("dest_counts", "dest_offsets", "expert_counts", "expert_offsets", "pos"):
            assert np.array_equal(to_host(r[key], np.int32).reshape(want[key].shape), want[key]), (seed, key)
        assert np.array_equal(to_host(r["packed"], np.uint16).reshape(T * K, H), want["packed"]), seed


def test_pack_in_a_graph_replayed_with_new_routing():
    """One purlin_pack captured in a graph, replayed three times with new
    tokens and routing loaded eagerly between the replays: every replay
    matches the oracle."""
    T, H, K, E, P = 4096, 512, 8, 256, 8
    x = torch.empty((T, H), dtype=torch.int16, device="cuda")
    ids = torch.empty((T, K), dtype=torch.int32, device="cuda")
    ws = torch.empty(PL.purlin_pack_workspace_size(T, K, E), dtype=torch.uint8, device="cuda")
    out = dict(packed=torch.empty((T * K, H), dtype=torch.int16, device="cuda"),
               dest_counts=torch.empty(P, dtype=torch.int32, device="cuda"),
               dest_offsets=torch.empty(P, dtype=torch.int32, device="cuda"),
               expert_counts=torch.empty(E, dtype=torch.int32, device="cuda"),
               expert_offsets=torch.empty(E, dtype=torch.int32, device="cuda"),
               pos=torch.empty((T, K), dtype=torch.int32, device="cuda"))

    def load(seed):
        rng = np.random.default_rng(seed)
        ids_np = W.zipf_topk_ids(T, E, K, 1.1, seed)
        x_np = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
        x.copy_(to_device(x_np))
        ids.copy_(to_device(ids_np))
        return x_np, ids_np

    load(40)
    PL.purlin_pack(x, ids, E, P, out=out, workspace=ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=side):
            PL.purlin_pack(x, ids, E, P, out=out, workspace=ws, stream=side)
    for rep, seed in enumerate((41, 42, 43)):
        x_np, ids_np = load(seed)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        want = oracle.pack(x_np, ids_np, E, P)
        for key in ("dest_counts", "dest_offsets", "expert_counts", "pos"):
            assert np.array_equal(to_host(out[key], np.int32).reshape(want[key].shape), want[key]), (rep, key)
        assert np.array_equal(to_host(out["packed"], np.uint16).reshape(T * K, H), want["packed"]), rep


def run_unpack(y_np, pos_np, g_np, status=True):
    T, K = pos_np.shape
    H = y_np.shape[1]
    out = Guarded(T * H * 2, torch.int16)
    st = torch.full((4,), 7, dtype=torch.int32, device="cuda")
    PL.purlin_unpack(to_device(y_np), to_device(pos_np), to_device(g_np), out=out.t.view(T, H),
                     dev_status=st if status else None)
    torch.cuda.synchronize()
    assert out.intact()
    return to_host(out.t, np.uint16).reshape(T, H), int(st[0].item())


@pytest.mark.parametrize(
    "T,H,K,seed",
    [(1, 8, 1, 0), (5, 16, 2, 1), (64, 1024, 8, 2), (65, 7, 3, 3), (129, 520, 8, 4), (50, 64, 17, 5), (3, 4096, 64, 6),
     (0, 64, 8, 7)],
)
def test_unpack_matches_oracle(T, H, K, seed):
    rng = np.random.default_rng(seed)
    y = oracle.narrow((rng.standard_normal((T * K, H)) * np.exp2(rng.integers(-10, 10, (T * K, H)))).astype(np.float32))
    pos = rng.permutation(T * K).reshape(T, K).astype(np.int32)
    g = rng.uniform(0, 1, (T, K)).astype(np.float32)
    got, status = run_unpack(y, pos, g)
    assert status == 0
    assert_bits_equal(got, oracle.unpack(y, pos, g), "bf16", "unpack")


def test_unpack_never_fuses_and_keeps_slot_order():
    g0 = np.float32(-(1 + 2.0**-7 + 2.0**-23))
    g1 = np.float32(1 + 2.0**-23)
    v0 = oracle.narrow(np.array([1.0], np.float32))[0]
    v1 = oracle.narrow(np.array([1 + 2.0**-7], np.float32))[0]
    H = 64
    y = np.array([[v0] * H, [v1] * H], np.uint16)
    got, _ = run_unpack(y, np.array([[0, 1]], np.int32), np.array([[g0, g1]], np.float32))
    assert np.all(got == 0)  # a fused multiply-add would give 0x3080
    vals = oracle.narrow(np.array([2.0**24, 1.0, -(2.0**24)], np.float32))
    y = np.repeat(vals[:, None], H, axis=1)
    got, _ = run_unpack(y, np.array([[0, 1, 2]], np.int32), np.ones((1, 3), np.float32))
    assert np.all(got == 0)  # slot order 0, 1, 2


def test_unpack_reports_bad_positions():
    rng = np.random.default_rng(12)
    T, H, K = 9, 32, 2
    y = rng.integers(0, 0x4000, (T * K, H)).astype(np.uint16)
    pos = rng.permutation(T * K).reshape(T, K).astype(np.int32)
    g = np.ones((T, K), np.float32)
    bad = pos.copy()
    bad[4, 1] = T * K
    got, status = run_unpack(y, bad, g)
    assert status == 1
    _, status = run_unpack(y, pos, g)
    assert status == 0


def test_pack_then_unpack_round_trip():
    cfg = W.MOE_CONFIG
    T, H = 512, 256
    ids = W.zipf_topk_ids(T, cfg.E, cfg.K, cfg.zipf_s, seed=21)
    rng = np.random.default_rng(21)
    x = oracle.narrow(rng.standard_normal((T, H)).astype(np.float32))
    r = PL.purlin_pack(to_device(x), to_device(ids), cfg.E, cfg.P)
    out = PL.purlin_unpack(r["packed"], r["pos"], torch.full((T, cfg.K), 1.0 / cfg.K, device="cuda"))
    torch.cuda.synchronize()
    assert np.array_equal(to_host(out, np.uint16).reshape(T, H), x)


def test_pack_and_combine_4096x7168_top8_of_256_full_size():
    """4096 tokens x 7168 hidden, E=256 over P=8, top-8 Zipf(1.1); then combine."""
    cfg = W.MOE_CONFIG
    assert PL.purlin_pack_single_launch(cfg.T, cfg.H, cfg.K, cfg.E)
    ids = W.zipf_topk_ids(cfg.T, cfg.E, cfg.K, cfg.zipf_s, cfg.seed_ids)
    x = W.moe_tokens(cfg)
    got, status = run_pack(x, ids, cfg.E, cfg.P)
    want = oracle.pack(x, ids, cfg.E, cfg.P)
    assert status == 0
    for key in ("dest_counts", "dest_offsets", "expert_counts", "expert_offsets", "pos"):
        assert np.array_equal(got[key], want[key]), key
    assert np.array_equal(got["packed"], want["packed"])
    del got
    y = W.moe_expert_outputs(cfg)
    g = W.softmax_gates(cfg.T, cfg.K, cfg.seed_gates)
    out, status = run_unpack(y, want["pos"], g)
    assert status == 0
    assert_bits_equal(out, oracle.unpack(y, want["pos"], g), "bf16", "combine 4096 x 7168")


def test_binding_rejects_undersized_outputs_before_launch():
    """The C ABI cannot see tensor sizes, so the binding checks every output
    the kernels would write; nothing is enqueued on a rejection."""
    T, H, K, E, P = 64, 32, 4, 16, 4
    rng = np.random.default_rng(8)
    x = to_device(rng.integers(0, 0x10000, (T, H)).astype(np.uint16))
    ids = to_device(_distinct_ids(rng, T, K, E))
    small = torch.empty(T * K * H - 1, dtype=torch.int16, device="cuda")
    with pytest.raises(PL.PurlinError):
        PL.purlin_pack(x, ids, E, P, out=dict(packed=small))
    with pytest.raises(PL.PurlinError):
        PL.purlin_pack(x, ids, E, P, out=dict(pos=torch.empty(T * K - 1, dtype=torch.int32, device="cuda")))
    with pytest.raises(PL.PurlinError):
        PL.purlin_pack_dedup(x, ids, E, P, out=dict(row_of=torch.empty(T * P - 1, dtype=torch.int32, device="cuda")))
    r = PL.purlin_pack(x, ids, E, P)
    g = torch.ones((T, K), dtype=torch.float32, device="cuda")
    with pytest.raises(PL.PurlinError):
        PL.purlin_unpack(r["packed"][: T * K - 1], r["pos"], g)
    with pytest.raises(PL.PurlinError):
        PL.purlin_unpack(r["packed"], r["pos"], g, out=torch.empty(T * H - 1, dtype=torch.int16, device="cuda"))
    torch.cuda.synchronize()


def test_pack_and_combine_beyond_4GiB():
    """40960 tokens x 7168, top-8 of 256: the packed matrix is 4.7 GB, so row
    offsets pass 2^32 bytes in pack and combine.  Positions and counts are
    compared with the oracle's (computed on 8 columns of the same tokens),
    sampled rows bit for bit, and the combine of the packed rows with gates
    1/8 returns every token exactly (K equal rows weighted 1/K)."""
    T, H, K, E, P = 40960, 7168, 8, 256, 8
    ids = W.zipf_topk_ids(T, E, K, 1.1, seed=31).astype(np.int32)
    rng = np.random.default_rng(31)
    x_d = torch.randn(T, H, device="cuda").to(torch.bfloat16).view(torch.int16)
    r = PL.purlin_pack(x_d, to_device(ids), E, P)
    torch.cuda.synchronize()
    want = oracle.pack(np.zeros((T, 8), np.uint16), ids, E, P)
    assert np.array_equal(to_host(r["pos"], np.int32).reshape(T, K), want["pos"])
    assert np.array_equal(to_host(r["dest_counts"], np.int32), want["dest_counts"])
    assert np.array_equal(to_host(r["expert_offsets"], np.int32), want["expert_offsets"])
    assert int(want["pos"].max()) * H * 2 > (1 << 32)
    # the rows that land past 4 GiB and a random sample
    far = np.argwhere(want["pos"].astype(np.int64) * H * 2 >= (1 << 32))
    pick = np.concatenate([far[rng.choice(len(far), 128, replace=False)],
                           np.argwhere(want["pos"] >= 0)[rng.choice(T * K, 128, replace=False)]])
    for t, k in pick:
        assert torch.equal(r["packed"][int(want["pos"][t, k])], x_d[t]), (t, k)
    g = torch.full((T, K), 1.0 / K, device="cuda")
    out = PL.purlin_unpack(r["packed"], r["pos"], g)
    torch.cuda.synchronize()
    assert torch.equal(out.view(T, H), x_d)


def test_short_names():
    """plan / pack / unpack: the same calls under the wrapper's short names."""
    rng = np.random.default_rng(40)
    T, H, K, E, P = 100, 64, 4, 16, 4
    x = to_device(rng.integers(0, 0x7F00, (T, H)).astype(np.uint16))
    ids = to_device(_distinct_ids(rng, T, K, E))
    packed, dest_counts, dest_offsets, expert_counts, pos = PL.pack(x, ids, E, P)
    out = PL.unpack(packed, pos, torch.full((T, K), 1.0 / K, device="cuda"))
    torch.cuda.synchronize()
    assert torch.equal(out.view(T, H), x.view(T, H))
    assert int(dest_counts.sum().item()) == T * K and int(expert_counts.sum().item()) == T * K
    pl = PL.plan("allreduce", 2, 64, "fp32", 64)
    a = [torch.ones(64, device="cuda"), torch.full((64,), 2.0, device="cuda")]
    o = [torch.empty(64, device="cuda") for _ in range(2)]
    pl.exec(a, o)
    torch.cuda.synchronize()
    assert bool((o[0] == 3).all()) and bool((o[1] == 3).all())
