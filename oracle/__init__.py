"""Oracle for the Purlin datapath executor: plain, slow CPU definitions.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package; only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
path (no kernels, headers, helpers, tables or pre/post-processing): every
function here is written from the paper's statement of what is computed.

Contents
--------
``bf16``         exact bf16 -> fp32 widening and fp32 -> bf16 round-to-nearest-
                 even narrowing, from the IEEE 754 binary32 encoding.
``collectives``  AllGather, ReduceScatter, AllReduce, AllToAll over P ranks
                 (Section 2.1 "Stable communication semantics"; layouts of
                 Section 3.1; rank-order reduction of Eq. 2, Section 3.3).
``rooted``       Broadcast, Scatter, Gather, Reduce (Appendix A).
``vcollectives`` AllGatherV, ReduceScatterV, AllToAllV (sizes at run time).
``moe``          MoE dispatch ``pack`` and combine ``unpack`` (the paper names
                 them only as the expert-parallel use of AllToAll, Table 2;
                 their contract is written out in ``moe``'s docstrings).
``moe_dedup``    De-duplicated dispatch ``pack_dedup`` (one row per token and
                 destination rank) and its combine ``unpack_dedup``.
``ep``           Expert-parallel dispatch / combine over P ranks: pack, then
                 AllToAllV of the rows (and back, then unpack), per slot and
                 de-duplicated, composed from the definitions above.

Representation: fp32 data is ``numpy.float32``; bf16 data is its 16-bit
encoding held in ``numpy.uint16``.  Floating-point arithmetic is numpy
float32 ufuncs, which round every operation to binary32 (round to nearest,
ties to even, denormals kept) and never contract a multiply and an add.

Parity status: every function has independent pins in
``tests/test_oracle_pins*.py`` (brute force, the paper's worked layout
example, closed forms, special cases); none is "parity unpinned".
"""

from .bf16 import narrow, widen
from .collectives import all_gather, all_reduce, all_to_all, reduce_scatter
from .moe import pack, unpack
from .moe_dedup import pack_dedup, unpack_dedup
from .ep import ep_combine, ep_combine_dedup, ep_dispatch, ep_dispatch_dedup
from .rooted import broadcast, gather, reduce, scatter
from .vcollectives import all_gather_v, all_to_all_v, reduce_scatter_v

__all__ = [
    "narrow",
    "widen",
    "all_gather",
    "all_reduce",
    "all_to_all",
    "reduce_scatter",
    "pack",
    "unpack",
    "pack_dedup",
    "unpack_dedup",
    "ep_dispatch",
    "ep_combine",
    "ep_dispatch_dedup",
    "ep_combine_dedup",
    "broadcast",
    "gather",
    "reduce",
    "scatter",
    "all_gather_v",
    "all_to_all_v",
    "reduce_scatter_v",
]
