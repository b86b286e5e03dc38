"""Rooted collectives, written as their definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Appendix A ("Rooted Collectives in SNAC") of the paper describes Broadcast,
Reduce, Scatter and Gather with the existing layouts plus a choice of which
ranks produce or consume:

* Broadcast copies the root's whole input to every rank (the root's own
  output included);
* Scatter gives rank ``r`` partition ``r`` of the root's input (scattered
  input -> packed output, only the root produces);
* Gather concatenates every rank's contribution, in rank order, at the root
  (packed input -> scattered output, only the root consumes);
* Reduce combines every rank's contribution at the root (Eq. 2 order).

The paper also composes them: broadcast = compose<scatter, allGather>,
reduce = compose<reduceScatter, gather> (Appendix A listing); the pins check
those identities against the direct definitions below.

``ins`` holds P one-dimensional arrays in rank order (entries of ranks that
contribute nothing may be ``None``).  Outputs of ranks that receive nothing
are ``None``.  ``count`` (N) is the root-side scattered size: Broadcast and
Reduce move N elements per rank, Scatter splits the root's N elements into
P partitions, Gather assembles P contributions of N/P elements.
"""

import numpy as np

from .collectives import _check, rank_order_sum


def _rooted_check(P, root):
    if not 0 <= root < P:
        raise ValueError("root out of range")


def broadcast(ins, root, dtype):
    P = len(ins)
    _rooted_check(P, root)
    (src,), _ = _check([ins[root]], dtype)
    return [src.copy() for _ in range(P)]


def scatter(ins, root, dtype):
    P = len(ins)
    _rooted_check(P, root)
    (src,), n = _check([ins[root]], dtype)
    if n % P:
        raise ValueError("count must be a multiple of P")
    M = n // P
    return [src[r * M:(r + 1) * M].copy() for r in range(P)]


def gather(ins, root, dtype):
    P = len(ins)
    _rooted_check(P, root)
    ins, _ = _check(ins, dtype)
    out = [None] * P
    out[root] = np.concatenate([ins[p] for p in range(P)])
    return out


def reduce(ins, root, dtype):
    P = len(ins)
    _rooted_check(P, root)
    ins, n = _check(ins, dtype)
    if n % P:
        raise ValueError("count must be a multiple of P")
    out = [None] * P
    out[root] = rank_order_sum(ins, dtype)
    return out
