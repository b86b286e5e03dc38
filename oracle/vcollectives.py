"""Variable-size collectives, written as their definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 3.1 of the paper: the V variants keep the packed / scattered /
transposed relationships but take partition sizes at run time
(AllGatherV, ReduceScatterV, AllToAllV in Listing 1; sizes of the
evaluation in Appendix C.4).  Sizes here are element counts:

* AllGatherV (packedV -> scatteredV): rank p contributes counts[p] elements;
  every rank receives the contributions in rank order,
  ``out_r[off_p + i] = in_p[i]`` with ``off_p = sum(counts[:p])``;
* ReduceScatterV (scatteredV -> packedV): every rank's input holds
  sum(counts) elements in partitions of counts[r]; rank r receives
  partition r reduced over all ranks in rank order (Eq. 2);
* AllToAllV (scatteredV -> transposedV): counts[p][r] elements go from rank p
  to rank r; rank p's input holds its partitions in destination order,
  rank r's output holds what it receives in source order.
"""

import numpy as np

from .collectives import _check, rank_order_sum


def _offsets(sizes):
    out, run = [], 0
    for n in sizes:
        out.append(run)
        run += int(n)
    return out, run


def all_gather_v(ins, counts, dtype):
    P = len(ins)
    if len(counts) != P:
        raise ValueError("one count per rank")
    parts = []
    for p in range(P):
        (a,), n = _check([ins[p]], dtype)
        if counts[p] < 0 or counts[p] > n:
            raise ValueError("count out of range")
        parts.append(a[: int(counts[p])])
    gathered = np.concatenate(parts) if parts else np.zeros(0)
    return [gathered.copy() for _ in range(P)]


def reduce_scatter_v(ins, counts, dtype):
    P = len(ins)
    if len(counts) != P or min(counts) < 0:
        raise ValueError("one non-negative count per rank")
    offs, total = _offsets(counts)
    ins, n = _check(ins, dtype)
    if total > n:
        raise ValueError("inputs shorter than the partitions")
    return [rank_order_sum([a[offs[r]:offs[r] + int(counts[r])] for a in ins], dtype) for r in range(P)]


def all_to_all_v(ins, counts, dtype):
    """counts[p][r]: elements rank p sends to rank r."""
    P = len(ins)
    if len(counts) != P or any(len(row) != P for row in counts):
        raise ValueError("counts must be P x P")
    outs = []
    for r in range(P):
        pieces = []
        for p in range(P):
            (a,), n = _check([ins[p]], dtype)
            send_offs, send_total = _offsets(counts[p])
            if send_total > n or min(counts[p]) < 0:
                raise ValueError("rank p's partitions do not fit its input")
            pieces.append(a[send_offs[r]:send_offs[r] + int(counts[p][r])])
        outs.append(np.concatenate(pieces))
    return outs
