"""The four fixed-size collectives, written as their definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper passages followed (Purlin, arXiv 2609.36954):

* Section 2.1, "Stable communication semantics": AllGather concatenates the
  contribution of every rank; ReduceScatter reduces uniform slices and rank
  ``r`` receives slice ``r``; AllReduce leaves the whole reduced result at
  every rank; AllToAll gives rank ``r`` the ``r``-th partition of every rank.
* Section 3.1, "Buffer Layouts": ``packed`` (one contiguous contribution),
  ``scattered`` (contiguous partitions indexed by rank), ``transposed``
  (destination ``r`` holds partition ``r`` of every source, in source order);
  Listing 1 pairs each collective with its consume op and layouts.
* Section 3.3, Eq. 2: ``y[i] = sum_{p=0}^{n-1} x_p[i]``, starting from zero,
  adding rank 0, then rank 1, ..., rank n-1; each term converted from the
  element type to FP32, the sum kept in FP32 and converted back once.

Conventions:

* ``ins`` is a sequence of P one-dimensional arrays, rank order.  fp32 data
  is ``float32``; bf16 data is ``uint16`` encodings.
* ``count`` (N) is the per-rank element count on the scattered side, the
  paper's message-size convention (Section 5, "Microbenchmark
  methodology"): AllReduce N in / N out, ReduceScatter N in / N/P out,
  AllGather N/P in / N out, AllToAll N in / N out.  N must be a multiple of
  P: the fixed-size collectives use uniform slices.
"""

import numpy as np

from .bf16 import narrow, widen

_DTYPES = {"fp32": np.float32, "bf16": np.uint16}


def _check(ins, dtype):
    if dtype not in _DTYPES:
        raise ValueError(f"unknown dtype {dtype!r}")
    ins = [np.asarray(a) for a in ins]
    if not ins:
        raise ValueError("need at least one rank")
    n = ins[0].shape[0]
    for a in ins:
        if a.ndim != 1 or a.shape[0] != n:
            raise ValueError("every rank must hold a 1-D buffer of the same length")
        if a.dtype != _DTYPES[dtype]:
            raise ValueError(f"{dtype} data must be {np.dtype(_DTYPES[dtype]).name}")
    return ins, n


def _to_f32(a, dtype):
    return widen(a) if dtype == "bf16" else a.astype(np.float32)


def _from_f32(a, dtype):
    return narrow(a) if dtype == "bf16" else a.astype(np.float32)


def rank_order_sum(columns, dtype):
    """Eq. 2 over equally long arrays ``columns[0..P-1]``.

    ``acc`` starts at +0.0 and adds rank 0's term, then rank 1's, ... in
    binary32; the result is converted back to the element type once.
    """
    acc = np.zeros(np.asarray(columns[0]).shape[0], dtype=np.float32)  # +0.0
    for col in columns:  # p = 0, 1, ..., P-1
        acc = np.add(acc, _to_f32(np.asarray(col), dtype), dtype=np.float32)
    return _from_f32(acc, dtype)


def reduce_scatter(ins, dtype):
    """ReduceScatter: scattered input -> packed output (consume op: reduce).

    Rank ``r`` receives partition ``r`` reduced over all ranks:
    ``out_r[i] = narrow(sum_p widen(in_p[r*M + i]))`` with ``M = N/P``.
    """
    ins, n = _check(ins, dtype)
    P = len(ins)
    if n % P:
        raise ValueError("count must be a multiple of P")
    M = n // P
    return [rank_order_sum([ins[p][r * M:(r + 1) * M] for p in range(P)], dtype) for r in range(P)]


def all_gather(ins, dtype):
    """AllGather: packed input -> scattered output (consume op: copy).

    Every rank ``r`` receives the contributions of all ranks in rank order:
    ``out_r[p*M + i] = in_p[i]`` (the self slot included).  A bit copy, so
    the element type does not matter beyond its width.
    """
    ins, M = _check(ins, dtype)
    P = len(ins)
    gathered = np.concatenate([ins[p] for p in range(P)])
    return [gathered.copy() for _ in range(P)]


def all_reduce(ins, dtype):
    """AllReduce: scattered input -> scattered output, complete result everywhere.

    Every rank receives the whole reduction:
    ``out_r[j] = narrow(sum_p widen(in_p[j]))`` for all ``j < N``.  Written
    from the definition (Section 2.1), not as compose<ReduceScatter,
    AllGather> (Section 3.1, Listing 1), so that the identity
    ``AllGather(ReduceScatter(x)) == AllReduce(x)`` is a real check of the
    partition bookkeeping of the other two functions.
    """
    ins, n = _check(ins, dtype)
    P = len(ins)
    if n % P:
        raise ValueError("count must be a multiple of P")
    full = rank_order_sum(ins, dtype)
    return [full.copy() for _ in range(P)]


def all_to_all(ins, dtype):
    """AllToAll: scattered input -> transposed output (consume op: copy).

    Destination ``r`` receives partition ``r`` of every source ``p`` and
    arranges them in source order: ``out_r[p*M + i] = in_p[r*M + i]``.
    """
    ins, n = _check(ins, dtype)
    P = len(ins)
    if n % P:
        raise ValueError("count must be a multiple of P")
    M = n // P
    return [np.concatenate([ins[p][r * M:(r + 1) * M] for p in range(P)]) for r in range(P)]
