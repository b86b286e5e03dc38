"""Pins of the expert-parallel dispatch / combine oracle (``oracle.ep``):
a hand-worked two-rank example, the placement of every row, and the
combine against ``oracle.unpack`` of each rank's own pack (pinned in
test_oracle_pins.py) with identity and marked experts."""

import numpy as np
import pytest

import oracle
from oracle.ep import ep_combine, ep_dispatch


def test_ep_dispatch_hand_worked_example():
    """P=2, E=2 (one expert per rank), T=3, K=1.

    rank 0: ids [1, 0, 1] -> packed [a1 | a0 a2], counts [1, 2]
    rank 1: ids [0, 0, 1] -> packed [b0 b1 | b2], counts [2, 1]
    rank 0 receives a1 (from 0), then b0 b1 (from 1); rank 1 receives a0 a2, then b2.
    """
    a = np.array([[10, 11], [20, 21], [30, 31]], np.uint16)
    b = np.array([[40, 41], [50, 51], [60, 61]], np.uint16)
    ids = [np.array([[1], [0], [1]], np.int32), np.array([[0], [0], [1]], np.int32)]
    d = ep_dispatch([a, b], ids, E=2, P=2)
    assert d["counts"].tolist() == [[1, 2], [2, 1]]
    assert np.array_equal(d["recv"][0], np.stack([a[1], b[0], b[1]]))
    assert np.array_equal(d["recv"][1], np.stack([a[0], a[2], b[2]]))
    assert d["recv_pos"].reshape(2, 3).tolist() == [[0, 0, 1], [1, 2, 2]]


def _inputs(P, T, H, K, E, seed):
    rng = np.random.default_rng(seed)
    xs = [rng.integers(0, 0x4700, (T, H)).astype(np.uint16) for _ in range(P)]  # finite, |x| < 2^15
    idss = [np.stack([rng.permutation(E)[:K] for _ in range(T)]).astype(np.int32) for _ in range(P)]
    gates = [rng.random((T, K)).astype(np.float32) for _ in range(P)]
    return xs, idss, gates


@pytest.mark.parametrize("P,T,H,K,E,seed", [(2, 9, 3, 2, 4, 0), (3, 20, 5, 3, 9, 1), (4, 33, 2, 4, 16, 2)])
def test_every_row_lands_once_where_recv_pos_says(P, T, H, K, E, seed):
    xs, idss, _ = _inputs(P, T, H, K, E, seed)
    d = ep_dispatch(xs, idss, E, P)
    L = E // P
    seen = [[] for _ in range(P)]
    for p in range(P):
        for t in range(T):
            for k in range(K):
                r = int(idss[p][t, k]) // L
                q = int(d["recv_pos"][p, t, k])
                assert np.array_equal(d["recv"][r][q], xs[p][t])
                seen[r].append((q, p, int(idss[p][t, k]), t))
    for r in range(P):
        assert len(d["recv"][r]) == int(d["counts"][:, r].sum())
        rows = sorted(seen[r])
        assert [q for q, *_ in rows] == list(range(len(rows)))  # a bijection onto the buffer
        keys = [(p, e, t) for _, p, e, t in rows]
        assert keys == sorted(keys)  # sender ascending, then expert, then token


def test_ep_dispatch_on_zipf_routing_matches_pack_counts():
    from paper_2609_36954_amd import workloads as W

    P, T, H, K, E = 8, 128, 2, 8, 64
    xs = [np.full((T, H), p, np.uint16) for p in range(P)]
    idss = [W.zipf_topk_ids(T, E, K, 1.1, 900 + p) for p in range(P)]
    d = ep_dispatch(xs, idss, E, P)
    for p in range(P):
        assert np.array_equal(d["counts"][p], oracle.pack(xs[p], idss[p], E, P)["dest_counts"])
    for r in range(P):  # rows arrive grouped by sender, in sender order
        assert np.array_equal(d["recv"][r][:, 0], np.repeat(np.arange(P), d["counts"][:, r]).astype(np.uint16))


@pytest.mark.parametrize("P,T,H,K,E,seed", [(2, 9, 3, 2, 4, 3), (4, 33, 6, 4, 16, 4)])
def test_ep_combine_identity_experts_equals_unpack_of_pack(P, T, H, K, E, seed):
    xs, idss, gates = _inputs(P, T, H, K, E, seed)
    d = ep_dispatch(xs, idss, E, P)
    outs = ep_combine(d["recv"], idss, d["recv_pos"], gates, E, P)
    for p in range(P):
        pk = oracle.pack(xs[p], idss[p], E, P)
        assert np.array_equal(outs[p], oracle.unpack(pk["packed"], pk["pos"], gates[p]))


def test_ep_combine_marked_experts():
    """Expert rank r returns row ^ (r + 1): the combine must pick each slot's
    output from the rank owning that slot's expert."""
    P, T, H, K, E = 4, 40, 5, 3, 12
    xs, idss, gates = _inputs(P, T, H, K, E, 5)
    d = ep_dispatch(xs, idss, E, P)
    ys = [d["recv"][r] ^ np.uint16(r + 1) for r in range(P)]
    outs = ep_combine(ys, idss, d["recv_pos"], gates, E, P)
    L = E // P
    for p in range(P):
        rows = np.repeat(xs[p], K, axis=0) ^ ((idss[p].reshape(-1) // L) + 1).astype(np.uint16)[:, None]
        want = oracle.unpack(rows, np.arange(T * K).reshape(T, K), gates[p])
        assert np.array_equal(outs[p], want)


def test_ep_dispatch_dedup_hand_worked_example():
    """P=2, E=4 (experts 0,1 on rank 0; 2,3 on rank 1), T=3, K=2.

    rank 0: ids [[0,2],[1,0],[3,2]] -> ranks {0,1}, {0}, {1}: rows to 0: a0 a1; to 1: a0 a2
    rank 1: ids [[2,3],[0,3],[1,0]] -> ranks {1}, {0,1}, {0}: rows to 0: b1 b2; to 1: b0 b1
    rank 0 receives a0 a1 b1 b2; rank 1 receives a0 a2 b0 b1.
    """
    a = np.array([[1, 1], [2, 2], [3, 3]], np.uint16)
    b = np.array([[4, 4], [5, 5], [6, 6]], np.uint16)
    ids = [np.array([[0, 2], [1, 0], [3, 2]], np.int32), np.array([[2, 3], [0, 3], [1, 0]], np.int32)]
    d = oracle.ep_dispatch_dedup([a, b], ids, E=4, P=2)
    assert d["counts"].tolist() == [[2, 2], [2, 2]]
    assert np.array_equal(d["recv"][0], np.stack([a[0], a[1], b[1], b[2]]))
    assert np.array_equal(d["recv"][1], np.stack([a[0], a[2], b[0], b[1]]))
    assert d["recv_row"].tolist() == [[[0, 0], [1, -1], [-1, 1]], [[-1, 2], [2, 3], [3, -1]]]


@pytest.mark.parametrize("P,T,H,K,E,seed", [(2, 9, 3, 2, 4, 6), (4, 40, 5, 4, 16, 7), (3, 25, 2, 3, 12, 8)])
def test_ep_dedup_rows_land_once_and_combine_equals_unpack_dedup(P, T, H, K, E, seed):
    xs, idss, _ = _inputs(P, T, H, K, E, seed)
    d = oracle.ep_dispatch_dedup(xs, idss, E, P)
    L = E // P
    for r in range(P):
        got = sorted(int(d["recv_row"][p, t, r]) for p in range(P) for t in range(T) if d["recv_row"][p, t, r] >= 0)
        assert got == list(range(len(d["recv"][r])))
    for p in range(P):
        for t in range(T):
            owners = {int(e) // L for e in idss[p][t]}
            for r in range(P):
                q = int(d["recv_row"][p, t, r])
                assert (q >= 0) == (r in owners)
                if q >= 0:
                    assert np.array_equal(d["recv"][r][q], xs[p][t])
    ys = [d["recv"][r] ^ np.uint16(r + 1) for r in range(P)]  # marked partial outputs
    outs = oracle.ep_combine_dedup(ys, d["recv_row"], P)
    for p in range(P):
        pk = oracle.pack_dedup(xs[p], idss[p], E, P)
        mark = np.repeat(np.arange(P), pk["dest_counts"]).astype(np.uint16) + 1
        assert np.array_equal(outs[p], oracle.unpack_dedup(pk["packed"] ^ mark[:, None], pk["row_of"]))
