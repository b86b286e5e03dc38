"""Pins of the oracle against what the paper and the mathematics fix.

Each test checks ``oracle/`` against something other than itself: the
paper's worked layout example (tests/golden/fig2_layouts.txt), a pure-Python
brute force with its own rounding (tests/brute.py), closed forms, special
cases that reduce to a textbook routine, and invariants.  A plausible slip
in the oracle (a dropped rank, a swapped index, a transposed operand, a
wrong rounding direction, a fused multiply-add, a different summation order)
fails at least one of them.
"""

import os
import struct

import numpy as np
import pytest

import brute
import oracle
from oracle import collectives as C
from oracle import moe as MOE

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def f32_from_bits(bits):
    return np.asarray(bits, dtype=np.uint32).view(np.float32)


# ---------------------------------------------------------------------------
# bf16 conversions
# ---------------------------------------------------------------------------

TIE_VECTORS = [
    # (float32 encoding, expected bf16 encoding, why)
    (0x3F808000, 0x3F80, "tie, lower candidate even -> stays"),
    (0x3F818000, 0x3F82, "tie, lower candidate odd -> rounds up to even"),
    (0x3F808001, 0x3F81, "just above the tie -> up"),
    (0x3F807FFF, 0x3F80, "just below the tie -> down"),
    (0xBF818000, 0xBF82, "negative tie -> away from zero to the even one"),
    (0x7F7F8000, 0x7F80, "tie at max finite + half ulp -> +inf"),
    (0x7F7F7FFF, 0x7F7F, "below max finite + half ulp -> max finite"),
    (0xFF7FFFFF, 0xFF80, "negative overflow -> -inf"),
    (0x7F800000, 0x7F80, "+inf"),
    (0xFF800000, 0xFF80, "-inf"),
    (0x00000000, 0x0000, "+0"),
    (0x80000000, 0x8000, "-0"),
    (0x00008000, 0x0000, "denormal tie, lower even -> 0"),
    (0x00018000, 0x0002, "denormal tie, lower odd -> up"),
    (0x00010001, 0x0001, "denormal below tie"),
    (0x007FFFFF, 0x0080, "largest denormal rounds up into the normal range"),
    (0x7FA00000, 0x7FE0, "signalling NaN -> quiet NaN, payload top bits kept"),
    (0xFFC00001, 0xFFC0, "negative quiet NaN keeps its sign"),
]


@pytest.mark.parametrize("f32bits,expect,why", TIE_VECTORS)
def test_narrow_vectors(f32bits, expect, why):
    got = int(oracle.narrow(f32_from_bits([f32bits]))[0])
    assert got == expect, f"{why}: {f32bits:#010x} -> {got:#06x}, want {expect:#06x}"


def test_narrow_matches_fraction_brute_force():
    rng = np.random.default_rng(11)
    bits = rng.integers(0, 2**32, size=20000, dtype=np.uint64).astype(np.uint32)
    # every exponent, with low halves at and around the tie
    hi = np.arange(0, 0x10000, 7, dtype=np.uint32) << np.uint32(16)
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    bits = np.concatenate([bits, (hi[:, None] | lows[None, :]).ravel()])
    x = f32_from_bits(bits)
    got = oracle.narrow(x)
    for b, g in zip(bits.tolist(), got.tolist()):
        want = brute.bf16_narrow(brute.f32_from_bits(b))
        assert g == want, f"{b:#010x}: oracle {g:#06x} brute {want:#06x}"


def test_narrow_matches_torch_cpu_cast():
    """Run (only run) torch's CPU float32 -> bfloat16 cast as a second opinion."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(12)
    bits = rng.integers(0, 2**32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    x = f32_from_bits(bits)
    ours = oracle.narrow(x)
    theirs = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    nan = np.isnan(x)
    assert np.array_equal(ours[~nan], theirs[~nan])
    assert np.all(np.isnan(oracle.widen(ours[nan])))


def test_widen_all_encodings():
    h = np.arange(0x10000, dtype=np.uint32).astype(np.uint16)
    got = oracle.widen(h).view(np.uint32)
    want = np.array([brute.f32_bits(brute.bf16_widen(int(v))) for v in range(0x10000)], dtype=np.uint32)
    # NaN encodings: compare bits directly (struct may quiet them); others must match exactly
    assert np.array_equal(got, (np.arange(0x10000, dtype=np.uint32) << 16))
    finite = ~np.isnan(oracle.widen(h))
    assert np.array_equal(got[finite], want[finite])


def test_widen_narrow_round_trip():
    h = np.arange(0x10000, dtype=np.uint32).astype(np.uint16)
    w = oracle.widen(h)
    ok = ~np.isnan(w)
    assert np.array_equal(oracle.narrow(w)[ok], h[ok])


# ---------------------------------------------------------------------------
# Collectives: the paper's worked example
# ---------------------------------------------------------------------------


def _load_fig2():
    rows = []
    with open(os.path.join(GOLDEN, "fig2_layouts.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            lhs, rhs = line.split(":")
            op, rank = lhs.split()
            rows.append((op, int(rank), rhs.split()))
    return rows


FIG2 = _load_fig2()
FIG_P, FIG_M = 3, 4


def _sum_code(p, k):
    # distinct powers of two: a sum of any subset is exact in binary32 and
    # names the subset
    return np.float32(2.0 ** (8 * p + k))


def _decode_sum(v):
    v = float(v)
    terms = set()
    for p in range(FIG_P):
        for k in range(FIG_P):
            e = 2.0 ** (8 * p + k)
            if v >= e and int(v // e) % 2 == 1:
                terms.add((p, k))
    return terms


def _copy_code(p, k, i, dtype):
    if dtype == "fp32":
        return 0x3F800000 | (p << 12) | (k << 8) | i
    return (p << 12) | (k << 8) | i


def _decode_copy(bits, dtype):
    b = int(bits) & (0xFFFF if dtype == "bf16" else 0xFFFFFFFF)
    if dtype == "fp32":
        b &= 0xFFFF
    return (b >> 12) & 0xF, (b >> 8) & 0xF, b & 0xFF


def _as_bits(a, dtype):
    return a.view(np.uint32) if dtype == "fp32" else a


def _from_bits(codes, dtype):
    if dtype == "fp32":
        return np.asarray(codes, dtype=np.uint32).view(np.float32)
    return np.asarray(codes, dtype=np.uint16)


def _symbol_of_sum_block(block):
    terms = {frozenset(_decode_sum(v)) for v in block}
    assert len(terms) == 1, "a block mixes different sums"
    (t,) = terms
    ks = {k for (_, k) in t}
    ps = {p for (p, _) in t}
    assert len(ks) == 1 and ps == set(range(FIG_P)), f"not a full column sum: {sorted(t)}"
    return f"y{ks.pop()}"


@pytest.mark.parametrize("row", FIG2, ids=lambda r: f"{r[0]}-{r[1]}")
def test_fig2_layouts(row):
    op, rank, want = row
    P, M = FIG_P, FIG_M
    if op in ("reduce_scatter", "all_reduce"):
        ins = [np.concatenate([np.full(M, _sum_code(p, k), np.float32) for k in range(P)]) for p in range(P)]
        outs = getattr(oracle, op)(ins, "fp32")
        out = outs[rank]
        got = [_symbol_of_sum_block(out[j * M:(j + 1) * M]) for j in range(len(out) // M)]
        assert got == want
        return
    for dtype in ("fp32", "bf16"):
        if op == "all_gather":
            # inputs: the packed y_k held by rank k, coded as (k, k, i)
            ins = [_from_bits([_copy_code(k, k, i, dtype) for i in range(M)], dtype) for k in range(P)]
            out = _as_bits(oracle.all_gather(ins, dtype)[rank], dtype)
            got = []
            for j in range(P):
                dec = [_decode_copy(v, dtype) for v in out[j * M:(j + 1) * M]]
                assert [d[2] for d in dec] == list(range(M)), "elements out of order"
                assert len({d[:2] for d in dec}) == 1
                got.append(f"y{dec[0][0]}")
        else:  # all_to_all
            ins = [
                _from_bits([_copy_code(p, k, i, dtype) for k in range(P) for i in range(M)], dtype)
                for p in range(P)
            ]
            out = _as_bits(oracle.all_to_all(ins, dtype)[rank], dtype)
            got = []
            for j in range(P):
                dec = [_decode_copy(v, dtype) for v in out[j * M:(j + 1) * M]]
                assert [d[2] for d in dec] == list(range(M)), "elements out of order"
                assert len({d[:2] for d in dec}) == 1
                got.append(f"x{dec[0][0]}{dec[0][1]}")
        assert got == want, dtype


# ---------------------------------------------------------------------------
# Collectives: brute force on tiny inputs
# ---------------------------------------------------------------------------


def _rand_inputs(P, n, dtype, seed):
    rng = np.random.default_rng(seed)
    if dtype == "fp32":
        # wide magnitudes and both signs, so that rounding happens
        mag = rng.uniform(-1, 1, (P, n)) * np.exp2(rng.integers(-30, 30, (P, n)))
        return [mag[p].astype(np.float32) for p in range(P)]
    bits = rng.integers(0, 0x10000, (P, n)).astype(np.uint16)
    # keep finite values only (NaN payload propagation is not pinned)
    exp_all_ones = (bits & 0x7F80) == 0x7F80
    bits[exp_all_ones] &= 0xBFFF
    return [bits[p] for p in range(P)]


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P,n", [(2, 16), (3, 12), (4, 8), (1, 5)])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_collectives_brute_force(dtype, P, n, seed):
    ins = _rand_inputs(P, n, dtype, seed)
    as_list = [a.tolist() for a in ins]

    def same(oracle_outs, brute_outs):
        for o, b in zip(oracle_outs, brute_outs):
            if dtype == "fp32":
                assert o.view(np.uint32).tolist() == [brute.f32_bits(v) for v in b]
            else:
                assert o.tolist() == b

    same(oracle.reduce_scatter(ins, dtype), brute.reduce_scatter(as_list, dtype))
    same(oracle.all_reduce(ins, dtype), brute.all_reduce(as_list, dtype))
    same(oracle.all_to_all(ins, dtype), brute.all_to_all(as_list))
    packed = [a[: n // P] for a in ins]
    same(oracle.all_gather(packed, dtype), brute.all_gather([a.tolist() for a in packed]))


# ---------------------------------------------------------------------------
# Collectives: closed forms, special cases, invariants
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P", [1, 2, 3, 8, 16])
def test_reduce_scatter_then_all_gather_is_all_reduce(dtype, P):
    ins = _rand_inputs(P, P * 257, dtype, 100 + P)
    if dtype == "bf16":
        ins = [a & np.uint16(0xBFFF) for a in ins]  # keep |x| < 2, no overflow to inf
    rs = oracle.reduce_scatter(ins, dtype)
    ag = oracle.all_gather(rs, dtype)
    ar = oracle.all_reduce(ins, dtype)
    for a, b in zip(ag, ar):
        assert np.array_equal(_as_bits(a, dtype), _as_bits(b, dtype))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("c", [0.75, -1.5, 0.125])
@pytest.mark.parametrize("P", [1, 2, 3, 5, 8, 16])
def test_constant_fill_sums_to_P_times_c(dtype, c, P):
    """With every rank holding c, the result is exactly P*c.

    Holds because every partial sum k*c (k <= 16) of these c is a short
    binary fraction, exact in binary32, and P*c needs at most 8 significant
    bits, so it is exact in bf16 as well.
    """
    n = P * 64
    if dtype == "fp32":
        ins = [np.full(n, c, np.float32) for _ in range(P)]
        want = np.float32(P * c)
        for out in oracle.all_reduce(ins, dtype):
            assert np.all(out == want)
    else:
        cb = oracle.narrow(np.array([c], np.float32))[0]
        ins = [np.full(n, cb, np.uint16) for _ in range(P)]
        for out in oracle.all_reduce(ins, dtype):
            assert np.all(oracle.widen(out) == np.float32(P * c))


def test_rank_order_not_a_tree():
    """[2**24, 1, -2**24] summed in rank order is 0; other orders give 1."""
    ins = [np.full(3, v, np.float32) for v in (2.0**24, 1.0, -(2.0**24))]
    outs = {float(v) for o in oracle.all_reduce(ins, "fp32") for v in o}
    assert outs == {0.0}
    # the two other association orders (the point of the test)
    assert (np.float32(2.0**24) + (np.float32(1.0) + np.float32(-(2.0**24)))) == np.float32(1.0)
    assert ((np.float32(2.0**24) + np.float32(-(2.0**24))) + np.float32(1.0)) == np.float32(1.0)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_sum_of_negative_zeros_is_positive_zero(dtype):
    """The accumulator starts at +0.0 (Eq. 2 starts from zero); +0 + -0 = +0."""
    P = 4
    if dtype == "fp32":
        ins = [np.full(8, -0.0, np.float32) for _ in range(P)]
        out = oracle.all_reduce(ins, dtype)[0]
        assert np.all(out.view(np.uint32) == 0)
    else:
        ins = [np.full(8, 0x8000, np.uint16) for _ in range(P)]
        out = oracle.all_reduce(ins, dtype)[0]
        assert np.all(out == 0)


def test_denormals_are_kept():
    tiny = np.float32(2.0**-140)
    out = oracle.all_reduce([np.full(4, tiny), np.full(4, tiny)], "fp32")[0]
    assert np.all(out == np.float32(2.0**-139))
    outb = oracle.all_reduce([np.full(4, 1, np.uint16), np.full(4, 1, np.uint16)], "bf16")[0]
    assert np.all(outb == 2)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_single_rank_is_identity(dtype):
    ins = _rand_inputs(1, 64, dtype, 7)
    nz = _as_bits(ins[0], dtype) != (0x80000000 if dtype == "fp32" else 0x8000)
    out = oracle.all_reduce(ins, dtype)[0]
    assert np.array_equal(_as_bits(out, dtype)[nz], _as_bits(ins[0], dtype)[nz])


def test_two_ranks_fp32_is_one_add():
    ins = _rand_inputs(2, 4096, "fp32", 8)
    want = ins[0] + ins[1]
    got = oracle.all_reduce(ins, "fp32")[0]
    assert np.array_equal(got.view(np.uint32), (np.float32(0.0) + want).view(np.uint32))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P", [2, 5, 8])
def test_all_gather_and_all_to_all_are_permutations(dtype, P):
    """Coded inputs: every output element maps back to exactly one input element.

    AllGather copies each input element to P places; AllToAll moves each
    input element to exactly one place.
    """
    M = 6
    n = P * M
    code_max = 0x10000 if dtype == "bf16" else 0x1000000
    assert P * n < code_max
    ins = [_from_bits([(0x3F000000 if dtype == "fp32" else 0) | (p * n + j) for j in range(n)], dtype) for p in range(P)]
    idx = lambda v: int(v) & 0xFFFFFF if dtype == "fp32" else int(v)  # noqa: E731

    a2a = oracle.all_to_all(ins, dtype)
    seen = {}
    for r, out in enumerate(a2a):
        for pos, v in enumerate(_as_bits(out, dtype)):
            seen.setdefault(idx(v), []).append((r, pos))
    assert sorted(seen) == list(range(P * n))
    assert all(len(v) == 1 for v in seen.values())
    for code, [(r, pos)] in seen.items():
        p, j = divmod(code, n)  # element j of rank p's input
        assert j // M == r and pos == p * M + j % M

    packed = [a[:M] for a in ins]
    ag = oracle.all_gather(packed, dtype)
    seen = {}
    for r, out in enumerate(ag):
        assert len(out) == P * M
        for pos, v in enumerate(_as_bits(out, dtype)):
            seen.setdefault(idx(v), []).append((r, pos))
    assert sorted(seen) == sorted(p * n + i for p in range(P) for i in range(M))
    for code, places in seen.items():
        p, i = divmod(code, n)
        assert sorted(places) == [(r, p * M + i) for r in range(P)]


def test_oracle_rejects_nonuniform_slices():
    with pytest.raises(ValueError):
        oracle.reduce_scatter([np.zeros(10, np.float32)] * 3, "fp32")
    with pytest.raises(ValueError):
        oracle.all_to_all([np.zeros(10, np.uint16)] * 4, "bf16")


# ---------------------------------------------------------------------------
# MoE pack
# ---------------------------------------------------------------------------


def test_pack_hand_worked_example():
    """T=4, K=2, E=4 experts over P=2 ranks (L=2 experts per rank).

    ids = [[1,3],[0,1],[3,2],[1,0]]
      tokens per expert, in token order: e0: t1 t3 | e1: t0 t1 t3 | e2: t2 | e3: t0 t2
      expert_counts = [2,3,1,2], expert_offsets = [0,2,5,6]
      dest 0 = experts 0,1 -> 5 rows at 0; dest 1 = experts 2,3 -> 3 rows at 5
      pos[t,k] = expert_offsets[e] + (# earlier tokens that chose e):
        t0: e1 -> 2+0, e3 -> 6+0      t1: e0 -> 0+0, e1 -> 2+1
        t2: e3 -> 6+1, e2 -> 5+0      t3: e1 -> 2+2, e0 -> 0+1
      packed rows 0..7 come from tokens 1,3,0,1,3,2,0,2
    """
    ids = np.array([[1, 3], [0, 1], [3, 2], [1, 0]], np.int32)
    x = np.arange(4 * 3, dtype=np.uint16).reshape(4, 3) + 100
    r = oracle.pack(x, ids, E=4, P=2)
    assert r["expert_counts"].tolist() == [2, 3, 1, 2]
    assert r["expert_offsets"].tolist() == [0, 2, 5, 6]
    assert r["dest_counts"].tolist() == [5, 3]
    assert r["dest_offsets"].tolist() == [0, 5]
    assert r["pos"].tolist() == [[2, 6], [0, 3], [7, 5], [4, 1]]
    assert np.array_equal(r["packed"], x[[1, 3, 0, 1, 3, 2, 0, 2]])


def _distinct_ids(rng, T, K, E):
    return np.stack([rng.permutation(E)[:K] for _ in range(T)]).astype(np.int32)


@pytest.mark.parametrize("T,K,E,P,seed", [(5, 2, 4, 2, 0), (5, 2, 4, 2, 1), (33, 4, 16, 4, 2), (64, 8, 64, 8, 3), (7, 1, 3, 1, 4)])
def test_pack_matches_sort_brute_force(T, K, E, P, seed):
    rng = np.random.default_rng(seed)
    ids = _distinct_ids(rng, T, K, E)
    x = rng.integers(0, 0x10000, (T, 5)).astype(np.uint16)
    r = oracle.pack(x, ids, E, P)
    pos, ec, dc, do = brute.pack(ids.tolist(), E, P)
    assert r["pos"].tolist() == pos
    assert r["expert_counts"].tolist() == ec
    assert r["dest_counts"].tolist() == dc
    assert r["dest_offsets"].tolist() == do
    for t in range(T):
        for k in range(K):
            assert np.array_equal(r["packed"][pos[t][k]], x[t])


def test_pack_invariants_on_zipf_routing():
    from paper_2609_36954_amd import workloads as W

    T, E, P, K = 512, 256, 8, 8
    ids = W.zipf_topk_ids(T, E, K, 1.1, seed=4)
    assert all(len(set(row)) == K for row in ids.tolist())
    x = np.arange(T, dtype=np.uint16)[:, None].repeat(3, axis=1)
    r = oracle.pack(x, ids, E, P)
    dc, do, pos = r["dest_counts"], r["dest_offsets"], r["pos"]
    assert dc.sum() == T * K
    assert do.tolist() == np.concatenate([[0], np.cumsum(dc)[:-1]]).tolist()
    assert sorted(pos.ravel().tolist()) == list(range(T * K))  # a bijection
    # rows sorted by (expert, token)
    rows = sorted((int(pos[t, k]), int(ids[t, k]), t) for t in range(T) for k in range(K))
    keys = [(e, t) for (_, e, t) in rows]
    assert keys == sorted(keys)
    # each destination segment holds exactly that rank's experts
    L = E // P
    for (p_, e, t) in rows:
        rank = e // L
        assert do[rank] <= p_ < do[rank] + dc[rank]
    assert np.array_equal(r["packed"][:, 0], np.array([t for (_, _, t) in rows], np.uint16))


def test_pack_rejects_bad_routing():
    x = np.zeros((2, 4), np.uint16)
    with pytest.raises(ValueError):
        oracle.pack(x, np.array([[0, 0], [1, 2]], np.int32), E=4, P=2)
    with pytest.raises(ValueError):
        oracle.pack(x, np.array([[0, 4], [1, 2]], np.int32), E=4, P=2)
    with pytest.raises(ValueError):
        oracle.pack(x, np.array([[0, 1], [1, 2]], np.int32), E=3, P=2)


# ---------------------------------------------------------------------------
# MoE unpack (combine)
# ---------------------------------------------------------------------------


def test_unpack_single_slot_unit_gate_is_inverse_permutation():
    rng = np.random.default_rng(5)
    T, H = 37, 16
    y = rng.integers(0, 0x10000, (T, H)).astype(np.uint16)
    y[(y & 0x7F80) == 0x7F80] &= 0xBFFF  # finite only
    y[y == 0x8000] = 0  # -0 becomes +0 through the +0 accumulator
    perm = rng.permutation(T).astype(np.int32)[:, None]
    out = oracle.unpack(y, perm, np.ones((T, 1), np.float32))
    assert np.array_equal(out, y[perm[:, 0]])


@pytest.mark.parametrize("K", [1, 2, 4, 8])
def test_unpack_equal_rows_with_gate_one_over_K(K):
    """K copies of a row with gate 1/K sum back to the row exactly (K a power of two)."""
    rng = np.random.default_rng(6)
    T, H = 9, 32
    base = oracle.narrow(rng.standard_normal((T, H)).astype(np.float32))
    y = np.repeat(base, K, axis=0)  # rows t*K .. t*K+K-1 hold token t's row
    pos = (np.arange(T)[:, None] * K + np.arange(K)[None, :]).astype(np.int32)
    out = oracle.unpack(y, pos, np.full((T, K), 1.0 / K, np.float32))
    assert np.array_equal(out, base)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_unpack_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    T, K, H = 4, 3, 6
    y = oracle.narrow((rng.standard_normal((T * K, H)) * np.exp2(rng.integers(-8, 8, (T * K, H)))).astype(np.float32))
    pos = rng.permutation(T * K).reshape(T, K).astype(np.int32)
    g = rng.uniform(0, 1, (T, K)).astype(np.float32)
    got = oracle.unpack(y, pos, g)
    want = brute.unpack(y.tolist(), pos.tolist(), g.tolist())
    assert got.tolist() == want


def test_unpack_does_not_fuse_multiply_add():
    """g1*v1 rounds away 2**-30 before the add; a fused multiply-add would keep it.

    slot 0: g = -(1 + 2**-7 + 2**-23), v = 1      -> acc = g exactly
    slot 1: g = 1 + 2**-23,           v = 1 + 2**-7
            exact product 1 + 2**-7 + 2**-23 + 2**-30 rounds to 1 + 2**-7 + 2**-23
    separate rounding: acc = 0 -> bf16 0x0000;  fused: 2**-30 -> bf16 0x3080
    """
    g0 = np.float32(-(1 + 2.0**-7 + 2.0**-23))
    g1 = np.float32(1 + 2.0**-23)
    assert float(g0) == -(1 + 2.0**-7 + 2.0**-23) and float(g1) == 1 + 2.0**-23
    v0 = oracle.narrow(np.array([1.0], np.float32))[0]
    v1 = oracle.narrow(np.array([1 + 2.0**-7], np.float32))[0]
    y = np.array([[v0], [v1]], np.uint16)
    out = oracle.unpack(y, np.array([[0, 1]], np.int32), np.array([[g0, g1]], np.float32))
    assert int(out[0, 0]) == 0x0000
    fused = struct.unpack("<I", struct.pack("<f", 2.0**-30))[0] >> 16
    assert fused == 0x3080


def test_unpack_sums_slots_in_ascending_order():
    """Rows [2**24, 1, -2**24] with unit gates give 0 in slot order 0,1,2.

    Other orders give 1: (-2**24 + 1) + 2**24 = 1, while 2**24 + 1 rounds back
    to 2**24 in binary32.
    """
    vals = oracle.narrow(np.array([2.0**24, 1.0, -(2.0**24)], np.float32))
    assert oracle.widen(vals).tolist() == [2.0**24, 1.0, -(2.0**24)]
    y = vals[:, None].repeat(4, axis=1)
    out = oracle.unpack(y, np.array([[0, 1, 2]], np.int32), np.ones((1, 3), np.float32))
    assert np.all(out == 0)
    out_rev = oracle.unpack(y, np.array([[2, 1, 0]], np.int32), np.ones((1, 3), np.float32))
    assert np.all(oracle.widen(out_rev) == 1.0)


def test_pack_then_unpack_of_the_tokens_returns_them():
    """Combining the dispatched rows of x with gates 1/K returns x exactly."""
    from paper_2609_36954_amd import workloads as W

    T, E, P, K, H = 64, 32, 4, 4, 24
    ids = W.zipf_topk_ids(T, E, K, 1.1, seed=9)
    rng = np.random.default_rng(9)
    x = oracle.narrow(rng.standard_normal((T, H)).astype(np.float32))
    r = oracle.pack(x, ids, E, P)
    out = oracle.unpack(r["packed"], r["pos"], np.full((T, K), 1.0 / K, np.float32))
    assert np.array_equal(out, x)


def test_rank_order_sum_helper_is_eq2():
    # a direct check that the shared helper is the rank-order sum, with +0 start
    cols = [np.array([1.0, -0.0], np.float32), np.array([2.0**-24, -0.0], np.float32)]
    out = C.rank_order_sum(cols, "fp32")
    assert out[0] == np.float32(1.0) and out.view(np.uint32)[1] == 0
    assert MOE.unpack is oracle.unpack
