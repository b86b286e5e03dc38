"""De-duplicated MoE dispatch and its combine, written as their definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper names expert-parallel dispatch and combine only as uses of
AllToAll(V) (Section 2, Table 2) and says nothing of de-duplication.  This
variant sends a token once to each rank that owns at least one of its
experts, instead of once per (token, slot); the receiving rank applies all
of its local experts to that one row and returns one partial output per
(token, rank).  The contract below is this library's reading.

Dispatch, for ``ids[T, K]`` expert ids, ``E`` experts split evenly over
``P`` ranks (``L = E / P``, ``dest(e) = e // L``):

* ``dests(t)``           = the set ``{dest(ids[t, k]) : k < K}``;
* ``dest_counts[r]``     = number of tokens t with ``r in dests(t)``;
* ``dest_offsets``       = exclusive prefix sum of ``dest_counts``;
* ``row_of[t, r]``       = ``dest_offsets[r] + #{t' < t : r in dests(t')}``
  when ``r in dests(t)``, else -1;
* ``packed[row_of[t, r], :] = x[t, :]`` (bit copy), for every ``r in dests(t)``.

Rows are grouped by destination rank, then token ascending.  Ids must lie in
[0, E) and be distinct within a token (as for ``pack``).

Combine, for partial outputs ``y[R, H]`` in the de-duplicated layout (row
``row_of[t, r]`` holds what rank r computed for token t, gate weights
already applied there):

    acc = +0.0
    for r = 0 .. P-1, r in dests(t):  acc = acc (+) widen(y[row_of[t, r], h])
    out[t, h] = narrow(acc)

binary32 adds, each rounded, ranks in ascending order (the rank order of
Eq. 2, Section 3.3).
"""

import numpy as np

from .bf16 import narrow, widen


def _check_routing(ids, E, P):
    ids = np.asarray(ids)
    T, K = ids.shape
    if E % P:
        raise ValueError("E must be a multiple of P")
    if ids.size and (ids.min() < 0 or ids.max() >= E):
        raise ValueError("expert id out of range")
    for t in range(T):
        if len(set(int(e) for e in ids[t])) != K:
            raise ValueError(f"token {t} repeats an expert id")
    return ids


def pack_dedup(x, ids, E, P):
    """``x``: uint16 [T, H] (bf16 encodings); ``ids``: int [T, K].

    Returns ``packed`` (uint16 [R, H], R = sum of ``dest_counts``),
    ``dest_counts`` [P], ``dest_offsets`` [P] and ``row_of`` [T, P], all
    int32.
    """
    x = np.asarray(x)
    ids = _check_routing(ids, E, P)
    T = ids.shape[0]
    if x.shape[0] != T:
        raise ValueError("x and ids disagree on T")
    L = E // P
    dests = [set(int(e) // L for e in ids[t]) for t in range(T)]

    dest_counts = np.zeros(P, dtype=np.int64)
    for t in range(T):
        for r in dests[t]:
            dest_counts[r] += 1
    dest_offsets = np.zeros(P, dtype=np.int64)
    running = 0
    for r in range(P):
        dest_offsets[r] = running
        running += dest_counts[r]

    row_of = np.full((T, P), -1, dtype=np.int64)
    seen = np.zeros(P, dtype=np.int64)  # #{t' < t : r in dests(t')}
    for t in range(T):
        for r in range(P):
            if r in dests[t]:
                row_of[t, r] = dest_offsets[r] + seen[r]
                seen[r] += 1

    packed = np.zeros((running,) + x.shape[1:], dtype=x.dtype)
    for t in range(T):
        for r in range(P):
            if row_of[t, r] >= 0:
                packed[row_of[t, r]] = x[t]

    i32 = np.int32
    return {
        "packed": packed,
        "dest_counts": dest_counts.astype(i32),
        "dest_offsets": dest_offsets.astype(i32),
        "row_of": row_of.astype(i32),
    }


def unpack_dedup(y, row_of):
    """``y``: uint16 [R, H]; ``row_of``: int [T, P] (-1 = no row).  Returns uint16 [T, H]."""
    y = np.asarray(y)
    row_of = np.asarray(row_of)
    T, P = row_of.shape
    H = y.shape[1]
    acc = np.zeros((T, H), dtype=np.float32)  # +0.0
    with np.errstate(over="ignore", invalid="ignore"):  # IEEE overflow to inf, inf - inf = NaN
        for r in range(P):  # rank order
            sel = row_of[:, r] >= 0
            acc[sel] = np.add(acc[sel], widen(y[row_of[sel, r]]), dtype=np.float32)
    return narrow(acc)
