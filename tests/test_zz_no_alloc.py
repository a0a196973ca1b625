"""The allocation-free selection entry point (static per-GPU scratch) gives
what the workspace entry point gives, bit for bit, on consecutive calls
that reuse the scratch (the second call smaller), and refuses requests past
its fixed maximum before launching anything."""

import numpy as np
import pytest
import torch

from paper_2609_09240_amd import tq

pytestmark = pytest.mark.gpu


def _both(energy, n_out, G, nnz):
    ed = torch.from_numpy(energy).cuda()
    ref = tq.tq_select_two_plane(ed, n_out, G, nnz)
    n = n_out * G
    out = (torch.full((n,), 0x5A5A5A5A, dtype=torch.int32, device="cuda"),
           torch.full((n_out + 1,), -7, dtype=torch.int32, device="cuda"),
           torch.full((max(nnz, 1),), 0x3C3C, dtype=torch.int16, device="cuda")[:nnz])
    got = tq.tq_select_two_plane_noalloc(ed, n_out, G, nnz, *out)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in ref], [t.cpu().numpy() for t in got]


@pytest.mark.parametrize("first,second", [((12288, 32, 0.1), (1000, 13, 0.036)),
                                          ((4096, 96, 0.5), (3, 7, 1.0))])
def test_noalloc_matches_workspace_call_twice(first, second):
    r = np.random.default_rng(21)
    for n_out, G, f2 in (first, second):
        n = n_out * G
        e = np.round(r.exponential(1.0, n) * 8) / 8          # ties across the cut
        nnz = int(np.floor(f2 * n))
        ref, got = _both(e, n_out, G, nnz)
        for name, a, b in zip(("rec_index", "rowptr1", "gidx1"), ref, got):
            np.testing.assert_array_equal(b, a, err_msg=f"{name} n_out={n_out} G={G} nnz={nnz}")
        assert got[1][-1] == nnz


def test_noalloc_refuses_past_its_maximum():
    e = torch.zeros(8, dtype=torch.float64, device="cuda")
    rec = torch.empty(8, dtype=torch.int32, device="cuda")
    rp = torch.empty(9, dtype=torch.int32, device="cuda")
    gi = torch.empty(8, dtype=torch.int16, device="cuda")
    with pytest.raises(tq.TqError) as err:
        # claims (2^24 / 128 + 1) * 128 groups: refused on the host, nothing launched
        tq.tq_select_two_plane_noalloc(e, (1 << 24) // 128 + 1, 128, 1, rec, rp, gi)
    assert err.value.status == 4
