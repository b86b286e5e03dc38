"""The reference streams (purlin_stream): XOR of the sources into every destination.

These are the access mixes (read-only, write-only, 1:1, 8-to-1, 1-to-8) that
the executor's kernels are measured against; the test checks the bytes they
move, including a ragged tail of vectors and a generic source/destination
count, against numpy.
"""

import numpy as np
import pytest
import torch

from gpu_util import Guarded, to_host
from paper_2609_36954_amd import purlin as PL

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("hints", [0, 3])
@pytest.mark.parametrize("nsrc,ndst", [(1, 1), (8, 1), (1, 8), (0, 1), (3, 5), (16, 2), (0, 3)])
@pytest.mark.parametrize("nvec", [1, 1023, 4096 + 17])
def test_stream_moves_the_xor_of_its_sources(nsrc, ndst, nvec, hints):
    rng = np.random.default_rng(nsrc * 100 + ndst * 10 + nvec)
    srcs_np = [rng.integers(0, 2**32, nvec * 4, dtype=np.uint64).astype(np.uint32) for _ in range(nsrc)]
    srcs = [torch.from_numpy(a.view(np.int32)).cuda() for a in srcs_np]
    outs = [Guarded(nvec * 16, torch.int32) for _ in range(ndst)]
    PL.purlin_stream([o.t for o in outs], srcs, nbytes=nvec * 16, nt_load=bool(hints & 1), nt_store=bool(hints & 2))
    torch.cuda.synchronize()
    if nsrc:
        want = srcs_np[0].copy()
        for a in srcs_np[1:]:
            want ^= a
    else:
        want = np.repeat(np.arange(nvec, dtype=np.uint32), 4)
    for o in outs:
        assert o.intact()
        assert np.array_equal(to_host(o.t, np.uint32), want)


def test_stream_read_only_writes_nothing_but_the_sink():
    src = torch.arange(4096 * 4, dtype=torch.int32, device="cuda")
    sink = Guarded(16, torch.int32)
    before = src.clone()
    PL.purlin_stream([], [src], sink=sink.t)
    torch.cuda.synchronize()
    assert sink.intact() and torch.equal(src, before)
