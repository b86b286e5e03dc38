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
