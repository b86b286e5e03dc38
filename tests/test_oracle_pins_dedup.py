"""Pins of the de-duplicated dispatch / combine oracle (``oracle.moe_dedup``)
against things other than itself: a hand-worked example, a brute force by
explicit sorting, the cases where it must coincide with ``oracle.pack`` /
``oracle.unpack`` (themselves pinned in test_oracle_pins.py), scalar brute
force of the combine, and an order-sensitive sum that tells rank order from
any other."""

import numpy as np
import pytest

import brute
import oracle


def _distinct_ids(rng, T, K, E):
    return np.stack([rng.permutation(E)[:K] for _ in range(T)]).astype(np.int32)


def test_pack_dedup_hand_worked_example():
    """T=4, K=2, E=4 over P=2 (L=2: experts 0,1 on rank 0, experts 2,3 on rank 1).

    ids = [[1,3],[0,1],[3,2],[1,0]]
      dests: t0 {0,1}  t1 {0}  t2 {1}  t3 {0}
      dest_counts = [3, 2], dest_offsets = [0, 3]
      rank 0 rows: t0, t1, t3 -> rows 0, 1, 2;  rank 1 rows: t0, t2 -> rows 3, 4
      row_of = [[0,3],[1,-1],[-1,4],[2,-1]]
    """
    ids = np.array([[1, 3], [0, 1], [3, 2], [1, 0]], np.int32)
    x = np.arange(4 * 3, dtype=np.uint16).reshape(4, 3) + 100
    r = oracle.pack_dedup(x, ids, E=4, P=2)
    assert r["dest_counts"].tolist() == [3, 2]
    assert r["dest_offsets"].tolist() == [0, 3]
    assert r["row_of"].tolist() == [[0, 3], [1, -1], [-1, 4], [2, -1]]
    assert np.array_equal(r["packed"], x[[0, 1, 3, 0, 2]])


def _brute_pack_dedup(ids, E, P):
    """The rows are the sorted set of (destination, token) pairs."""
    L = E // P
    pairs = sorted({(e // L, t) for t, row in enumerate(ids) for e in row})
    row_of = [[-1] * P for _ in ids]
    for i, (r, t) in enumerate(pairs):
        row_of[t][r] = i
    counts = [sum(1 for (r, _) in pairs if r == q) for q in range(P)]
    return pairs, row_of, counts


@pytest.mark.parametrize("T,K,E,P,seed", [(5, 2, 4, 2, 0), (9, 3, 12, 4, 1), (33, 4, 16, 4, 2), (64, 8, 64, 8, 3),
                                          (7, 1, 3, 1, 4), (20, 6, 48, 16, 5)])
def test_pack_dedup_matches_sort_brute_force(T, K, E, P, seed):
    rng = np.random.default_rng(seed)
    ids = _distinct_ids(rng, T, K, E)
    x = rng.integers(0, 0x10000, (T, 5)).astype(np.uint16)
    r = oracle.pack_dedup(x, ids, E, P)
    pairs, row_of, counts = _brute_pack_dedup(ids.tolist(), E, P)
    assert r["row_of"].tolist() == row_of
    assert r["dest_counts"].tolist() == counts
    assert r["dest_offsets"].tolist() == [sum(counts[:q]) for q in range(P)]
    assert len(r["packed"]) == len(pairs)
    for i, (_, t) in enumerate(pairs):
        assert np.array_equal(r["packed"][i], x[t])


@pytest.mark.parametrize("T,K,P,seed", [(30, 3, 4, 0), (64, 8, 8, 1), (17, 2, 16, 2)])
def test_pack_dedup_is_pack_when_each_rank_owns_one_expert(T, K, P, seed):
    """E = P: a token's experts are on distinct ranks, nothing is de-duplicated,
    and (expert, token) order is (rank, token) order."""
    rng = np.random.default_rng(seed)
    ids = _distinct_ids(rng, T, K, P)
    x = rng.integers(0, 0x10000, (T, 4)).astype(np.uint16)
    d = oracle.pack_dedup(x, ids, P, P)
    p = oracle.pack(x, ids, P, P)
    assert np.array_equal(d["packed"], p["packed"])
    assert np.array_equal(d["dest_counts"], p["dest_counts"])
    assert np.array_equal(d["dest_offsets"], p["dest_offsets"])
    for t in range(T):
        for k in range(K):
            assert d["row_of"][t, ids[t, k]] == p["pos"][t, k]


@pytest.mark.parametrize("E,P,seed", [(8, 2, 0), (64, 8, 1), (12, 3, 2)])
def test_pack_dedup_is_pack_for_one_slot(E, P, seed):
    rng = np.random.default_rng(seed)
    T = 40
    ids = rng.integers(0, E, (T, 1)).astype(np.int32)
    x = rng.integers(0, 0x10000, (T, 3)).astype(np.uint16)
    d = oracle.pack_dedup(x, ids, E, P)
    p = oracle.pack(x, ids, E, P)
    # one row per token either way; pack orders a rank's rows by expert first
    assert np.array_equal(d["dest_counts"], p["dest_counts"])
    L = E // P
    for t in range(T):
        assert d["row_of"][t].tolist().count(-1) == P - 1
        assert np.array_equal(d["packed"][d["row_of"][t, ids[t, 0] // L]], x[t])


def test_pack_dedup_invariants_on_zipf_routing():
    from paper_2609_36954_amd import workloads as W

    T, E, P, K = 512, 256, 8, 8
    ids = W.zipf_topk_ids(T, E, K, 1.1, seed=4)
    x = np.arange(T, dtype=np.uint16)[:, None].repeat(2, axis=1)
    r = oracle.pack_dedup(x, ids, E, P)
    L = E // P
    n_dests = [len(set(int(e) // L for e in row)) for row in ids]
    assert r["dest_counts"].sum() == sum(n_dests) < T * K
    rows = r["row_of"][r["row_of"] >= 0]
    assert sorted(rows.tolist()) == list(range(sum(n_dests)))  # a bijection
    for q in range(P):  # each segment: its tokens in ascending order
        lo, n = r["dest_offsets"][q], r["dest_counts"][q]
        toks = r["packed"][lo:lo + n, 0].tolist()
        assert toks == sorted(toks)
        assert all(q in {int(e) // L for e in ids[t]} for t in toks)


def test_pack_dedup_rejects_bad_routing():
    x = np.zeros((2, 4), np.uint16)
    for ids, E in (([[0, 0], [1, 2]], 4), ([[0, 4], [1, 2]], 4), ([[0, 1], [1, 2]], 3)):
        with pytest.raises(ValueError):
            oracle.pack_dedup(x, np.array(ids, np.int32), E=E, P=2)


def _brute_unpack_dedup(y, row_of):
    out = []
    for t in range(len(row_of)):
        line = []
        for h in range(len(y[0])):
            acc = 0.0
            for r in range(len(row_of[t])):
                if row_of[t][r] >= 0:
                    acc = brute.f32(acc + brute.bf16_widen(int(y[row_of[t][r]][h])))
            line.append(brute.bf16_narrow(acc))
        out.append(line)
    return out


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_unpack_dedup_matches_scalar_brute_force(seed):
    rng = np.random.default_rng(seed)
    T, E, P, K, H = 12, 16, 4, 3, 6
    ids = _distinct_ids(rng, T, K, E)
    d = oracle.pack_dedup(np.zeros((T, 1), np.uint16), ids, E, P)
    R = len(d["packed"])
    y = oracle.narrow((rng.standard_normal((R, H)) * np.exp2(rng.integers(-8, 8, (R, H)))).astype(np.float32))
    got = oracle.unpack_dedup(y, d["row_of"])
    assert got.tolist() == _brute_unpack_dedup(y.tolist(), d["row_of"].tolist())


def test_unpack_dedup_sums_in_rank_order():
    """bf16 2^24, 1, -2^24 from ranks 0, 1, 2: rank order gives
    ((0 + 2^24) + 1) - 2^24 = 0 (2^24 + 1 rounds to 2^24); any order that
    adds rank 2 before rank 1 gives 1."""
    big, one = oracle.narrow(np.float32([2.0 ** 24, 1.0]))
    y = np.array([[big], [one], [big | 0x8000]], np.uint16)
    row_of = np.array([[0, 1, 2]], np.int32)
    assert oracle.widen(oracle.unpack_dedup(y, row_of))[0, 0] == 0.0
    assert oracle.widen(oracle.unpack_dedup(y[[0, 2, 1]], np.array([[0, 2, 1]], np.int32)))[0, 0] == 0.0
    assert oracle.widen(oracle.unpack_dedup(y[[0, 2, 1]], np.array([[0, 1, 2]], np.int32)))[0, 0] == 1.0


def test_unpack_dedup_single_row_is_the_row_up_to_the_sign_of_zero():
    rng = np.random.default_rng(9)
    y = rng.integers(0, 0x10000, (20, 7)).astype(np.uint16)
    y[(y & 0x7F80) == 0x7F80] = 0x3F80  # keep NaN payloads out
    row_of = np.full((20, 3), -1, np.int32)
    row_of[np.arange(20), rng.integers(0, 3, 20)] = np.arange(20)[::-1]
    got = oracle.unpack_dedup(y, row_of)
    want = y[::-1].copy()
    want[want == 0x8000] = 0x0000  # +0 + -0 = +0 (the sum starts at +0)
    assert np.array_equal(got, want)


def test_unpack_dedup_two_rows_is_one_float32_add():
    rng = np.random.default_rng(3)
    a, b = (oracle.narrow(rng.standard_normal(64).astype(np.float32)) for _ in range(2))
    y = np.stack([a, b], axis=1).reshape(-1, 1)  # rows alternate a_i, b_i
    row_of = np.stack([np.arange(0, 128, 2), np.arange(1, 128, 2)], axis=1).astype(np.int32)
    got = oracle.unpack_dedup(y, row_of)[:, 0]
    assert np.array_equal(got, oracle.narrow(np.float32(oracle.widen(a) + oracle.widen(b))))


def test_unpack_dedup_is_unpack_with_unit_gates_when_slots_follow_ranks():
    """E = P and ids ascending within each token: slot order is rank order
    and pack == pack_dedup, so with gates 1 the two combines coincide."""
    rng = np.random.default_rng(4)
    T, P, K, H = 25, 8, 4, 9
    ids = np.sort(_distinct_ids(rng, T, K, P), axis=1)
    d = oracle.pack_dedup(np.zeros((T, 1), np.uint16), ids, P, P)
    p = oracle.pack(np.zeros((T, 1), np.uint16), ids, P, P)
    y = oracle.narrow(rng.standard_normal((T * K, H)).astype(np.float32))
    assert np.array_equal(oracle.unpack_dedup(y, d["row_of"]), oracle.unpack(y, p["pos"], np.ones((T, K), np.float32)))


def test_unpack_dedup_starts_from_positive_zero():
    """A token with no rows gives +0; negative zeros sum to +0 (the sum starts at +0)."""
    y = np.array([[0x8000, 0x8000], [0x8000, 0x3F80]], np.uint16)
    row_of = np.array([[0, 1], [-1, -1], [1, -1]], np.int32)
    got = oracle.unpack_dedup(y, row_of)
    assert got.tolist() == [[0x0000, 0x3F80], [0x0000, 0x0000], [0x0000, 0x3F80]]
