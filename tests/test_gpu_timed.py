"""The measurement entry points (purlin_stream_timed, purlin_pack_timed):
the same outputs as the untimed calls, and sane per-workgroup records."""

import numpy as np
import pytest
import torch

from paper_2609_36954_amd import purlin as PL
from paper_2609_36954_amd import workloads as W

pytestmark = pytest.mark.gpu


def _check_records(rate, recs, groups):
    assert rate > 0
    assert recs.shape == (groups, 4)
    assert set(recs[:, 0].tolist()) <= set(range(16))
    assert np.all(recs[:, 1] <= recs[:, 2]) and np.all(recs[:, 2] <= recs[:, 3])
    assert np.all(recs[:, 1] > 0)


def test_pack_timed_matches_pack():
    T, H, K, E, P = 1000, 512, 8, 256, 8
    ids = torch.from_numpy(W.zipf_topk_ids(T, E, K, 1.1, 5)).cuda()
    x = torch.from_numpy(np.random.default_rng(5).integers(0, 0x10000, (T, H)).astype(np.uint16).view(np.int16)).cuda()

    def outs():
        return dict(packed=torch.full((T * K, H), 7, dtype=torch.int16, device="cuda"),
                    dest_counts=torch.empty(P, dtype=torch.int32, device="cuda"),
                    dest_offsets=torch.empty(P, dtype=torch.int32, device="cuda"),
                    expert_counts=torch.empty(E, dtype=torch.int32, device="cuda"),
                    expert_offsets=torch.empty(E, dtype=torch.int32, device="cuda"),
                    pos=torch.empty((T, K), dtype=torch.int32, device="cuda"))

    want, got = outs(), outs()
    st_w = torch.full((1,), 5, dtype=torch.int32, device="cuda")
    st_g = torch.full((1,), 5, dtype=torch.int32, device="cuda")
    PL.purlin_pack(x, ids, E, P, out=want, dev_status=st_w)
    rec, groups = PL.purlin_pack_timed(x, ids, E, P, got, dev_status=st_g)
    torch.cuda.synchronize()
    for k in want:
        assert torch.equal(want[k], got[k]), k
    assert int(st_g.item()) == int(st_w.item()) == 0
    rate, recs = PL._timed_records(rec, groups)
    assert rec[1].item() == groups == (T + 3) // 4  # 4 tokens per workgroup, one per compute unit
    _check_records(rate, recs, groups)
    fin = PL.xcd_finish_times(rate, recs)
    assert sum(v["groups"] for v in fin.values()) == groups
    assert all(v["meta_us"] <= v["end_us"] for v in fin.values())


def test_pack_timed_rejects_three_launch_shapes():
    x = torch.zeros((4100, 1030), dtype=torch.int16, device="cuda")
    ids = torch.zeros((4100, 8), dtype=torch.int32, device="cuda")
    out = dict(packed=torch.empty((4100 * 8, 1030), dtype=torch.int16, device="cuda"),
               dest_counts=torch.empty(8, dtype=torch.int32, device="cuda"),
               dest_offsets=torch.empty(8, dtype=torch.int32, device="cuda"),
               expert_counts=torch.empty(256, dtype=torch.int32, device="cuda"),
               expert_offsets=torch.empty(256, dtype=torch.int32, device="cuda"),
               pos=torch.empty((4100, 8), dtype=torch.int32, device="cuda"))
    with pytest.raises(PL.PurlinError) as e:
        PL.purlin_pack_timed(x, ids, 256, 8, out)
    assert e.value.status == PL.PURLIN_ERR_UNSUPPORTED


@pytest.mark.parametrize("ns,nd", [(1, 8), (8, 1), (0, 1), (1, 0)])
def test_stream_timed_matches_stream(ns, nd):
    n = (3 << 20) + 48  # a ragged last workgroup
    g = torch.Generator(device="cuda").manual_seed(ns * 10 + nd)
    srcs = [torch.randint(-2**31, 2**31 - 1, (n // 4,), dtype=torch.int32, device="cuda", generator=g) for _ in range(ns)]
    want = [torch.zeros(n // 4, dtype=torch.int32, device="cuda") for _ in range(nd)]
    got = [torch.ones(n // 4, dtype=torch.int32, device="cuda") for _ in range(nd)]
    sink = torch.zeros(4, dtype=torch.int32, device="cuda") if nd == 0 else None
    PL.purlin_stream(want, srcs, nbytes=n, sink=sink)
    rate, recs = PL.purlin_stream_timed(got, srcs, nbytes=n, sink=sink, nt_store=True)
    for a, b in zip(want, got):
        assert torch.equal(a, b)
    per_block = 256 * (2 if ns >= 8 else 4) * 16
    groups = (n + per_block - 1) // per_block
    _check_records(rate, recs, groups)
    assert np.all(recs[:, 1] == recs[:, 2])
