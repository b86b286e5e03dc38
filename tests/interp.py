"""CPU interpreter of a plan's work items (test infrastructure).

Executes the planner's table on host numpy byte buffers so the planner can be
checked against the oracle without a GPU.  It is not the oracle: it only
applies each item's copy / rank-order reduce to the bytes it names, with the
oracle's bf16 conversions.  Items of a phase run in a shuffled order, so a
schedule whose result depended on the order within a phase would show.
"""

import numpy as np

from oracle import narrow, widen

KIND_COPY, KIND_REDUCE = 0, 1


def _typed(buf, off, nbytes, dtype):
    raw = buf[off:off + nbytes]
    return raw.view(np.uint16) if dtype == "bf16" else raw.view(np.float32)


def apply_item(it, bufs, dtype):
    n = int(it["bytes"])
    so, do = int(it["src_off"]), int(it["dst_off"])
    if it["kind"] == KIND_COPY:
        data = bufs[int(it["src_buf"])][so:so + n].copy()
    else:
        acc = np.zeros(n // (2 if dtype == "bf16" else 4), dtype=np.float32)
        for p in range(int(it["nsrc"])):
            src = bufs[int(it["src_buf"]) + p * int(it["src_step"])]
            x = _typed(src, so, n, dtype)
            acc = np.add(acc, widen(x) if dtype == "bf16" else x, dtype=np.float32)
        data = (narrow(acc) if dtype == "bf16" else acc).view(np.uint8)
    for j in range(int(it["ndst"])):
        dst = bufs[int(it["dst_buf"]) + j * int(it["dst_step"])]
        dst[do:do + n] = data


def run(items, phase_begin, bufs, dtype, seed=0):
    rng = np.random.default_rng(seed)
    bounds = [(phase_begin[0], phase_begin[1]), (phase_begin[1], phase_begin[2])]
    for lo, hi in bounds:
        order = rng.permutation(np.arange(lo, hi))
        for i in order:
            apply_item(items[i], bufs, dtype)


def run_v(items, bufs, counts, op, P, unit, dtype, capacity, out_capacity=None, transposed=False):
    """The variable-size mapping on the CPU: every item covers a range of the
    virtual index space; the sizes decide which source / destination and
    offset each element belongs to.  Returns False (writing nothing) for
    sizes the device would reject."""
    s = 2 if dtype == "bf16" else 4
    in_cap, out_cap = capacity, capacity if out_capacity is None else out_capacity
    c = [int(x) * unit for x in counts]
    if op == "alltoallv" and transposed:
        c = [c[(i % P) * P + i // P] for i in range(P * P)]
    if op == "alltoallv":
        m = [c[p * P:(p + 1) * P] for p in range(P)]
        if any(x < 0 or x > max(in_cap, out_cap) for x in c):
            return False
        if any(sum(row) > in_cap for row in m) or any(sum(m[p][r] for p in range(P)) > out_cap for r in range(P)):
            return False
    elif op == "allgatherv":
        if any(x < 0 or x > in_cap for x in c) or sum(c) > out_cap:
            return False
    elif any(x < 0 or x > out_cap for x in c) or sum(c) > in_cap:
        return False
    for it in items:
        lo, hi = int(it["src_off"]) // s, (int(it["src_off"]) + int(it["bytes"])) // s
        if op == "allgatherv":
            off = 0
            for p in range(P):
                x, y = max(lo, off), min(hi, off + c[p])
                if x < y:
                    data = bufs[p][(x - off) * s:(y - off) * s].copy()
                    for r in range(P):
                        bufs[P + r][x * s:y * s] = data
                off += c[p]
        elif op == "reduce_scatterv":
            off = 0
            for r in range(P):
                x, y = max(lo, off), min(hi, off + c[r])
                if x < y:
                    acc = np.zeros(y - x, np.float32)
                    for p in range(P):
                        v = _typed(bufs[p], x * s, (y - x) * s, dtype)
                        acc = np.add(acc, widen(v) if dtype == "bf16" else v, dtype=np.float32)
                    out = narrow(acc) if dtype == "bf16" else acc
                    bufs[P + r][(x - off) * s:(y - off) * s] = out.view(np.uint8)
                off += c[r]
        elif int(it["dst_step"]) == 1:  # source-major: the item covers source `part`'s input
            p = int(it["part"])
            send = 0
            for r in range(P):
                recv = sum(m[q][r] for q in range(p))
                x, y = max(lo, send), min(hi, send + m[p][r])
                if x < y:
                    b0 = recv + (x - send)
                    bufs[P + r][b0 * s:(b0 + y - x) * s] = bufs[p][x * s:y * s]
                send += m[p][r]
        else:  # destination-major: the item covers destination `part`'s output
            r = int(it["part"])
            recv = 0
            for p in range(P):
                send = sum(m[p][:r])
                x, y = max(lo, recv), min(hi, recv + m[p][r])
                if x < y:
                    a0 = send + (x - recv)
                    bufs[P + r][x * s:y * s] = bufs[p][a0 * s:(a0 + y - x) * s]
                recv += m[p][r]
    return True
