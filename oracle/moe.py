"""MoE dispatch (pack) and combine (unpack), written as their definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper names these operations only as the expert-parallel use of
AllGather(V) / ReduceScatter(V) / AllToAll(V), "dispatch tokens and combine
expert outputs" (Section 2, Table 2), and the variable-size layouts of
Section 3.1 (``scatteredV``).  The contract below is this library's reading:

Pack (dispatch), for ``ids[T, K]`` expert ids, ``E`` experts split evenly
over ``P`` ranks (``L = E / P`` consecutive experts per rank,
``dest(e) = e // L``):

* ``expert_counts[e]``  = number of (t, k) with ``ids[t, k] == e``;
* ``expert_offsets``    = exclusive prefix sum of ``expert_counts`` in
  global expert order;
* ``dest_counts[r]``    = sum of ``expert_counts`` over rank ``r``'s experts,
  ``dest_offsets[r] = expert_offsets[r * L]``;
* ``pos[t, k]``         = ``expert_offsets[e] + #{t' < t : e in ids[t', :]}``
  with ``e = ids[t, k]``;
* ``packed[pos[t, k], :] = x[t, :]`` (bit copy).

Rows are grouped by destination rank, then expert ascending, then token
ascending; one row per (t, k), no per-destination de-duplication.  Ids must
lie in [0, E) and be distinct within a token.

Unpack (combine), for expert outputs ``y[T*K, H]`` in the packed layout and
fp32 gate weights ``g[T, K]``:

    acc = +0.0
    for k = 0 .. K-1:  acc = acc (+) ( g[t, k] (x) widen(y[pos[t, k], h]) )
    out[t, h] = narrow(acc)

with (x) and (+) binary32 multiply and add, each rounded, never fused, and
the slots summed in ascending order -- the slot analogue of the rank order
of Eq. 2 (Section 3.3).
"""

import numpy as np

from .bf16 import narrow, widen


def pack(x, ids, E, P):
    """MoE dispatch.  ``x``: uint16 [T, H] (bf16 encodings); ``ids``: int [T, K].

    Returns a dict with ``packed`` (uint16 [T*K, H]), ``dest_counts`` [P],
    ``dest_offsets`` [P], ``expert_counts`` [E], ``expert_offsets`` [E] and
    ``pos`` [T, K], all counts/offsets/positions int32.
    """
    x = np.asarray(x)
    ids = np.asarray(ids)
    T, K = ids.shape
    if x.shape[0] != T:
        raise ValueError("x and ids disagree on T")
    if E % P:
        raise ValueError("E must be a multiple of P")
    if ids.size and (ids.min() < 0 or ids.max() >= E):
        raise ValueError("expert id out of range")
    for t in range(T):
        if len(set(int(e) for e in ids[t])) != K:
            raise ValueError(f"token {t} repeats an expert id")
    L = E // P

    expert_counts = np.zeros(E, dtype=np.int64)
    for t in range(T):
        for k in range(K):
            expert_counts[int(ids[t, k])] += 1

    expert_offsets = np.zeros(E, dtype=np.int64)
    running = 0
    for e in range(E):
        expert_offsets[e] = running
        running += expert_counts[e]

    dest_counts = np.array([expert_counts[r * L:(r + 1) * L].sum() for r in range(P)], dtype=np.int64)
    dest_offsets = np.array([expert_offsets[r * L] if E else 0 for r in range(P)], dtype=np.int64)

    # #{t' < t : e in ids[t', :]}: walk tokens in order, counting per expert.
    seen = np.zeros(E, dtype=np.int64)
    pos = np.zeros((T, K), dtype=np.int64)
    for t in range(T):
        for k in range(K):
            e = int(ids[t, k])
            pos[t, k] = expert_offsets[e] + seen[e]
        for k in range(K):
            seen[int(ids[t, k])] += 1

    packed = np.zeros((T * K,) + x.shape[1:], dtype=x.dtype)
    for t in range(T):
        for k in range(K):
            packed[pos[t, k]] = x[t]

    i32 = np.int32
    return {
        "packed": packed,
        "dest_counts": dest_counts.astype(i32),
        "dest_offsets": dest_offsets.astype(i32),
        "expert_counts": expert_counts.astype(i32),
        "expert_offsets": expert_offsets.astype(i32),
        "pos": pos.astype(i32),
    }


def unpack(y, pos, gates):
    """MoE combine.  ``y``: uint16 [T*K, H]; ``pos``: int [T, K]; ``gates``: float32 [T, K].

    Returns uint16 [T, H] (bf16 encodings).
    """
    y = np.asarray(y)
    pos = np.asarray(pos)
    gates = np.asarray(gates, dtype=np.float32)
    T, K = pos.shape
    H = y.shape[1]
    acc = np.zeros((T, H), dtype=np.float32)  # +0.0
    with np.errstate(over="ignore", invalid="ignore"):  # IEEE overflow to inf, inf - inf = NaN
        for k in range(K):  # slot order
            term = np.multiply(gates[:, k:k + 1], widen(y[pos[:, k]]), dtype=np.float32)
            acc = np.add(acc, term, dtype=np.float32)
    return narrow(acc)
