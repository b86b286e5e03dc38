"""Pins of the rooted collectives of the oracle (Appendix A of the paper).

* brute force in pure Python (tests/brute.py) on tiny inputs;
* the compositions the paper gives: broadcast = compose<scatter, allGather>,
  reduce = compose<reduceScatter, gather>;
* coded inputs: every output element maps back to the input element the
  definition names.
"""

import numpy as np
import pytest

import brute
import oracle

from test_oracle_pins import _as_bits, _rand_inputs


def _same(o, b, dtype):
    if o is None or b is None:
        assert o is None and b is None
        return
    if dtype == "fp32":
        assert o.view(np.uint32).tolist() == [brute.f32_bits(v) for v in b]
    else:
        assert o.tolist() == b


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P,n", [(1, 4), (2, 16), (3, 12), (4, 8)])
@pytest.mark.parametrize("seed", [0, 1])
def test_rooted_brute_force(dtype, P, n, seed):
    ins = _rand_inputs(P, n, dtype, 50 + seed)
    as_list = [a.tolist() for a in ins]
    for root in range(P):
        for o, b in zip(oracle.broadcast(ins, root, dtype), brute.broadcast(as_list, root)):
            _same(o, b, dtype)
        for o, b in zip(oracle.scatter(ins, root, dtype), brute.scatter(as_list, root)):
            _same(o, b, dtype)
        packed = [a[: n // P] for a in ins]
        for o, b in zip(oracle.gather(packed, root, dtype), brute.gather([a.tolist() for a in packed], root)):
            _same(o, b, dtype)
        for o, b in zip(oracle.reduce(ins, root, dtype), brute.reduce(as_list, root, dtype)):
            _same(o, b, dtype)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("P", [1, 2, 5, 8])
def test_paper_compositions(dtype, P):
    """Appendix A: broadcast = compose<scatter, allGather>; reduce = compose<reduceScatter, gather>."""
    ins = _rand_inputs(P, P * 33, dtype, 70 + P)
    if dtype == "bf16":
        ins = [a & np.uint16(0xBFFF) for a in ins]  # no overflow to inf
    for root in range(P):
        bc = oracle.broadcast(ins, root, dtype)
        via = oracle.all_gather(oracle.scatter(ins, root, dtype), dtype)
        for a, b in zip(bc, via):
            assert np.array_equal(_as_bits(a, dtype), _as_bits(b, dtype))
        red = oracle.reduce(ins, root, dtype)
        via = oracle.gather(oracle.reduce_scatter(ins, dtype), root, dtype)
        assert np.array_equal(_as_bits(red[root], dtype), _as_bits(via[root], dtype))
        assert all(red[r] is None and via[r] is None for r in range(P) if r != root)


@pytest.mark.parametrize("P", [2, 3, 8])
def test_scatter_and_gather_move_the_named_elements(P):
    M = 5
    root = P - 1
    ins = [np.arange(p * 1000, p * 1000 + P * M, dtype=np.uint16) for p in range(P)]
    sc = oracle.scatter(ins, root, "bf16")
    for r in range(P):
        assert sc[r].tolist() == [root * 1000 + r * M + i for i in range(M)]
    packed = [a[:M] for a in ins]
    g = oracle.gather(packed, root, "bf16")
    assert g[root].tolist() == [p * 1000 + i for p in range(P) for i in range(M)]
    assert all(g[r] is None for r in range(P) if r != root)


def test_root_out_of_range():
    with pytest.raises(ValueError):
        oracle.broadcast([np.zeros(4, np.float32)] * 2, 2, "fp32")
