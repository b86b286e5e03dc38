"""Pure-Python scalar brute force, used to pin the oracle on tiny inputs.

Independent of ``oracle/``: no numpy arithmetic, its own rounding.

* binary32 rounding of a Python float (binary64) goes through
  ``struct.pack('f')``, which rounds to nearest, ties to even.  For ``+``,
  ``-`` and ``*`` of two binary32 operands, computing in binary64 and then
  rounding to binary32 equals the correctly rounded binary32 result, because
  binary64 carries at least 2*24+2 significand bits (double rounding is
  innocuous; S. A. Figueroa, "When is double rounding innocuous?", 1995).
* bf16 narrowing is done with exact rationals (``fractions.Fraction``) and
  Python's ``round``, which rounds a Fraction half to even.
"""

import math
import struct
from fractions import Fraction


def f32(x):
    """Round a Python float to the nearest binary32 value (ties to even)."""
    return struct.unpack("<f", struct.pack("<f", x))[0]


def f32_bits(x):
    return struct.unpack("<I", struct.pack("<f", x))[0]


def f32_from_bits(b):
    return struct.unpack("<f", struct.pack("<I", b & 0xFFFFFFFF))[0]


def bf16_widen(h):
    return f32_from_bits((h & 0xFFFF) << 16)


def bf16_narrow(x):
    """binary32 value (Python float) -> bf16 encoding, round half to even."""
    if math.isnan(x):
        return (f32_bits(x) >> 16) | 0x0040
    if math.isinf(x) or x == 0.0:
        return f32_bits(x) >> 16
    sign = 0x8000 if x < 0 else 0
    a = Fraction(abs(x))
    _, e = math.frexp(abs(x))  # abs(x) in [2**(e-1), 2**e)
    # bf16 keeps 8 significant bits; below the normal range (2**-126) the
    # spacing stays at 2**-133.
    q = Fraction(2) ** (max(e, -125) - 8)
    r = round(a / q) * q  # ties to the even multiple of q
    if r >= Fraction(2) ** 128:
        return sign | 0x7F80
    return sign | (f32_bits(float(r)) >> 16)


def rank_order_reduce(columns, dtype):
    """Eq. 2 on scalars: acc = +0.0, add rank 0 .. P-1 in binary32, convert once."""
    n = len(columns[0])
    out = []
    for i in range(n):
        acc = 0.0
        for col in columns:
            v = bf16_widen(int(col[i])) if dtype == "bf16" else float(col[i])
            acc = f32(acc + v)
        out.append(bf16_narrow(acc) if dtype == "bf16" else acc)
    return out


def reduce_scatter(ins, dtype):
    P = len(ins)
    M = len(ins[0]) // P
    return [rank_order_reduce([list(ins[p][r * M:(r + 1) * M]) for p in range(P)], dtype) for r in range(P)]


def all_reduce(ins, dtype):
    P = len(ins)
    full = rank_order_reduce([list(a) for a in ins], dtype)
    return [list(full) for _ in range(P)]


def all_gather(ins):
    P = len(ins)
    M = len(ins[0])
    outs = []
    for r in range(P):
        o = [None] * (P * M)
        for p in range(P):
            for i in range(M):
                o[p * M + i] = ins[p][i]
        outs.append(o)
    return outs


def all_to_all(ins):
    P = len(ins)
    M = len(ins[0]) // P
    outs = []
    for r in range(P):
        o = [None] * (P * M)
        for p in range(P):
            for i in range(M):
                o[p * M + i] = ins[p][r * M + i]
        outs.append(o)
    return outs


def pack(ids, E, P):
    """Positions by an explicit sort of (expert, token) pairs.

    Returns (pos, expert_counts, dest_counts, dest_offsets) as Python lists.
    """
    T = len(ids)
    K = len(ids[0]) if T else 0
    entries = sorted((int(ids[t][k]), t, k) for t in range(T) for k in range(K))
    pos = [[None] * K for _ in range(T)]
    for row, (_, t, k) in enumerate(entries):
        pos[t][k] = row
    expert_counts = [sum(1 for (e, _, _) in entries if e == x) for x in range(E)]
    L = E // P
    dest_counts = [sum(expert_counts[r * L:(r + 1) * L]) for r in range(P)]
    dest_offsets = [sum(dest_counts[:r]) for r in range(P)]
    return pos, expert_counts, dest_counts, dest_offsets


def unpack(y, pos, gates):
    """out[t][h] = narrow(sum_k f32(g[t][k] * widen(y[pos[t][k]][h]))), slot order, no FMA."""
    T = len(pos)
    K = len(pos[0]) if T else 0
    H = len(y[0]) if len(y) else 0
    out = []
    for t in range(T):
        row = []
        for h in range(H):
            acc = 0.0
            for k in range(K):
                prod = f32(float(gates[t][k]) * bf16_widen(int(y[pos[t][k]][h])))
                acc = f32(acc + prod)
            row.append(bf16_narrow(acc))
        out.append(row)
    return out


def broadcast(ins, root):
    return [list(ins[root]) for _ in range(len(ins))]


def scatter(ins, root):
    P = len(ins)
    M = len(ins[root]) // P
    return [[ins[root][r * M + i] for i in range(M)] for r in range(P)]


def gather(ins, root):
    P = len(ins)
    out = [None] * P
    out[root] = [ins[p][i] for p in range(P) for i in range(len(ins[p]))]
    return out


def reduce(ins, root, dtype):
    out = [None] * len(ins)
    out[root] = rank_order_reduce([list(a) for a in ins], dtype)
    return out


def all_gather_v(ins, counts):
    out = []
    for p in range(len(ins)):
        for i in range(counts[p]):
            out.append(ins[p][i])
    return [list(out) for _ in ins]


def reduce_scatter_v(ins, counts, dtype):
    outs = []
    off = 0
    for r in range(len(ins)):
        cols = [list(a[off:off + counts[r]]) for a in ins]
        outs.append(rank_order_reduce(cols, dtype) if counts[r] else [])
        off += counts[r]
    return outs


def all_to_all_v(ins, counts):
    P = len(ins)
    outs = []
    for r in range(P):
        o = []
        for p in range(P):
            start = sum(counts[p][:r])
            o.extend(ins[p][start:start + counts[p][r]])
        outs.append(o)
    return outs
