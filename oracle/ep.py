"""Expert-parallel dispatch and combine over P ranks, as compositions of the
pinned definitions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Expert parallelism moves every token to the ranks owning its experts and
the expert outputs back (Section 2, Table 2: AllToAll(V)).  The contract
below is this library's reading; each step is an already-pinned oracle
function:

Dispatch: rank p packs its tokens (``moe.pack``), then the packed rows are
exchanged by AllToAllV (``vcollectives.all_to_all_v``, one row = one unit)
with ``counts[p][r]`` = rank p's ``dest_counts[r]``.  Rank r's receive
buffer holds the rows from rank 0, then rank 1, ..., each in its sender's
pack order.  ``recv_pos[p, t, k]`` is the row of token t's slot k of rank p
in the buffer of the rank owning expert ``ids_p[t, k]``:

    sum_{q < p} counts[q][r] + pos_p[t, k] - dest_offsets_p[r]

Combine: expert outputs ``y_r`` in rank r's receive layout go back the same
way and rank p finishes with ``moe.unpack`` of its own rows:

    out_p[t, h] = narrow( +0 (+) g[t, 0] (x) widen(y_{r0}[recv_pos[p, t, 0], h]) (+) ... )

in slot order, exactly as if the rows had been returned to p's pack order.
"""

import numpy as np

from .moe import pack, unpack
from .vcollectives import all_to_all_v


def ep_dispatch(xs, idss, E, P):
    """``xs``: P arrays uint16 [T, H]; ``idss``: P arrays int [T, K].

    Returns ``recv`` (P arrays uint16 [R_r, H]), ``counts`` (int32 [P, P])
    and ``recv_pos`` (int32 [P, T, K]).
    """
    if len(xs) != P or len(idss) != P:
        raise ValueError("need one token matrix and one id matrix per rank")
    packs = [pack(xs[p], idss[p], E, P) for p in range(P)]
    H = xs[0].shape[1]
    counts = np.array([[int(c) for c in pk["dest_counts"]] for pk in packs], dtype=np.int64)
    flat = all_to_all_v([pk["packed"].reshape(-1) for pk in packs], (counts * H).tolist(), "bf16")
    recv = [f.reshape(-1, H) for f in flat]
    L = E // P
    T, K = np.asarray(idss[0]).shape
    recv_pos = np.zeros((P, T, K), dtype=np.int64)
    for p in range(P):
        ids = np.asarray(idss[p])
        for t in range(T):
            for k in range(K):
                r = int(ids[t, k]) // L
                before = int(counts[:p, r].sum())  # rows rank r received from ranks < p
                recv_pos[p, t, k] = before + int(packs[p]["pos"][t, k]) - int(packs[p]["dest_offsets"][r])
    return {"recv": recv, "counts": counts.astype(np.int32), "recv_pos": recv_pos.astype(np.int32)}


def ep_combine(ys, idss, recv_pos, gatess, E, P):
    """``ys``: P arrays uint16 [>= R_r, H] (expert outputs in the receive
    layout); ``idss``, ``recv_pos`` as returned by ``ep_dispatch``;
    ``gatess``: P arrays float32 [T, K].  Returns P arrays uint16 [T, H]."""
    L = E // P
    outs = []
    for p in range(P):
        ids = np.asarray(idss[p])
        T, K = ids.shape
        H = ys[0].shape[1]
        rows = np.zeros((T * K, H), dtype=np.uint16)  # slot (t, k)'s expert output, in (t, k) order
        for t in range(T):
            for k in range(K):
                rows[t * K + k] = ys[int(ids[t, k]) // L][int(recv_pos[p, t, k])]
        outs.append(unpack(rows, np.arange(T * K, dtype=np.int64).reshape(T, K), gatess[p]))
    return outs


def ep_dispatch_dedup(xs, idss, E, P):
    """De-duplicated dispatch over P ranks: rank p's ``moe_dedup.pack_dedup``
    (one row per token and owning rank), then the AllToAllV of those rows.
    Returns ``recv`` (P arrays [R_r, H]), ``counts`` (int32 [P, P]) and
    ``recv_row`` (int32 [P, T, P]: row of rank p's token t in rank r's
    buffer, -1 where t has no expert on r)."""
    from .moe_dedup import pack_dedup

    packs = [pack_dedup(xs[p], idss[p], E, P) for p in range(P)]
    H = xs[0].shape[1]
    counts = np.array([[int(c) for c in pk["dest_counts"]] for pk in packs], dtype=np.int64)
    flat = all_to_all_v([pk["packed"].reshape(-1) for pk in packs], (counts * H).tolist(), "bf16")
    recv = [f.reshape(-1, H) for f in flat]
    T = np.asarray(idss[0]).shape[0]
    recv_row = np.full((P, T, P), -1, dtype=np.int64)
    for p in range(P):
        for t in range(T):
            for r in range(P):
                q = int(packs[p]["row_of"][t, r])
                if q >= 0:
                    recv_row[p, t, r] = int(counts[:p, r].sum()) + q - int(packs[p]["dest_offsets"][r])
    return {"recv": recv, "counts": counts.astype(np.int32), "recv_row": recv_row.astype(np.int32)}


def ep_combine_dedup(ys, recv_row, P):
    """Partial outputs ``ys`` (P arrays, rank r's receive layout) back to
    their tokens, summed in rank order as ``moe_dedup.unpack_dedup`` does.
    Returns P arrays uint16 [T, H]."""
    from .moe_dedup import unpack_dedup

    outs = []
    for p in range(P):
        T = recv_row.shape[1]
        H = ys[0].shape[1]
        rows = np.zeros((T * P, H), dtype=np.uint16)  # (t, r)'s partial row, in (t, r) order
        row_of = np.full((T, P), -1, dtype=np.int64)
        for t in range(T):
            for r in range(P):
                q = int(recv_row[p, t, r])
                if q >= 0:
                    rows[t * P + r] = ys[r][q]
                    row_of[t, r] = t * P + r
        outs.append(unpack_dedup(rows, row_of))
    return outs
