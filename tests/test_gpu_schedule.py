"""Device schedule and tile classification, bit-exact against the oracle and brute force."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api
from parity_util import say

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _fixture_rows():
    import os
    rows = []
    path = os.path.join(os.path.dirname(__file__), "golden", "schedule_qwen3.txt")
    for line in open(path):
        line = line.split("#", 1)[0].strip()
        if line:
            rows.append([int(t) for t in line.split()])
    return rows


def test_device_schedule_bit_exact():
    for w in (1, 3, 7, 64, 512):
        lengths = np.arange(1, 4 * w + 2, dtype=np.int32)
        positions = np.arange(0, 4 * w + 1, dtype=np.int32)
        say("debug_schedule w=%d n_lengths=%d n_positions=%d" % (w, len(lengths), len(positions)))
        g, f, dlt = api.debug_schedule(torch.from_numpy(lengths).cuda(),
                                       torch.from_numpy(positions).cuda(), w)
        g, f, dlt = g.cpu().numpy(), f.cpu().numpy(), dlt.cpu().numpy()
        for i, Lx in enumerate(lengths):
            G = O.group_size(int(Lx), w)
            assert g[i] == G
            want_f = np.array([O.remote_position(int(x), G) for x in positions])
            assert np.array_equal(f[i], want_f)
            assert np.array_equal(dlt[i], want_f - positions)
    rows = _fixture_rows()
    lengths = np.array([r[0] for r in rows], dtype=np.int32)
    for w in sorted(set(r[1] for r in rows)):
        sel = [r for r in rows if r[1] == w]
        lens = np.array([r[0] for r in sel], dtype=np.int32)
        pos = lens - 1
        g, f, _ = api.debug_schedule(torch.from_numpy(lens).cuda(), torch.from_numpy(pos).cuda(), w)
        g, f = g.cpu().numpy(), f.cpu().numpy()
        for i, r in enumerate(sel):
            assert g[i] == r[2] and f[i, i] == r[3], r


def _brute_classes(L, BQ, BK, w0):
    nq, nk = -(-L // BQ), -(-L // BK)
    out = np.zeros((nq, nk), dtype=np.int8)
    for qb in range(nq):
        qs = np.arange(qb * BQ, min(qb * BQ + BQ, L))
        for kt in range(nk):
            ks = np.arange(kt * BK, min(kt * BK + BK, L))
            diff = qs[:, None] - ks[None, :]
            causal = diff >= 0
            local = (causal & (diff <= w0)).any()
            remote = (causal & (diff > w0)).any()
            out[qb, kt] = (1 if local else 0) + (2 if remote else 0)
    return out


@pytest.mark.parametrize("g", [1, 2, 4, 8])
def test_device_tile_classes_equal_element_aggregate(g):
    for L in (1, 63, 64, 65, 200, 777):
        for w0 in (0, 1, 63, 64, 65, 127, 128, 300, 4096):
            say("debug_prefill_tiles L=%d g=%d w0=%d" % (L, g, w0))
            cls, BQ, BK = api.debug_prefill_tiles(L, 2 * g, 2, w0)
            want = _brute_classes(L, BQ, BK, w0)
            assert np.array_equal(cls.cpu().numpy(), want), (L, g, w0)
