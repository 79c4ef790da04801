"""Chunked prefill over paged raw caches: jl_bifocal_prefill_chunk_paged against
the dense-cache chunk (bit for bit) and the fp64 oracle across G transitions."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import assert_close, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

NAN = np.uint16(0x7FC0)


def _pool(k, v, page_size, seed, max_pages=None, spare_pages=3):
    """Scatter [B, T, Hkv, d] keys/values into shuffled pages of a pool.  Rows
    past T in the last page and the spare pages hold NaN; table entries past a
    sequence's pages are -1."""
    B, T, Hkv, d = k.shape
    used = (T + page_size - 1) // page_size
    max_pages = max_pages or used
    n_pages = B * used + spare_pages
    order = np.random.default_rng(seed).permutation(n_pages)
    kp = np.full((n_pages, page_size, Hkv, d), NAN, dtype=np.uint16)
    vp = np.full((n_pages, page_size, Hkv, d), NAN, dtype=np.uint16)
    table = np.full((B, max_pages), -1, dtype=np.int32)
    nxt = 0
    for b in range(B):
        for j in range(used):
            pg = int(order[nxt])
            nxt += 1
            table[b, j] = pg
            lo, hi = j * page_size, min((j + 1) * page_size, T)
            kp[pg, :hi - lo] = k[b, lo:hi]
            vp[pg, :hi - lo] = v[b, lo:hi]
    return kp, vp, table


def _dense_of(kp, vp, table, n_rows):
    """The dense caches [B, n_rows, Hkv, d] that a table describes, its entries
    clamped into the pool as the kernels clamp them."""
    n_pages, page_size = kp.shape[:2]
    B = table.shape[0]
    kc = np.empty((B, n_rows) + kp.shape[2:], dtype=np.uint16)
    vc = np.empty_like(kc)
    for b in range(B):
        for x0 in range(0, n_rows, page_size):
            pg = min(max(int(table[b, x0 // page_size]), 0), n_pages - 1)
            n = min(page_size, n_rows - x0)
            kc[b, x0:x0 + n] = kp[pg, :n]
            vc[b, x0:x0 + n] = vp[pg, :n]
    return kc, vc


def _paged_chunk(q, kp, vp, table, P, w_pre, w0, bifocal=True):
    out = api.prefill_chunk_paged(to_dev(q), to_dev(kp), to_dev(vp),
                                  torch.from_numpy(table).cuda(), q_start=P, w_pretrained=w_pre,
                                  w_local=w0, bifocal=bifocal, want_lse=True)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("T,P,g,page_size,w_pre,w0", [
    (700, 300, 4, 64, 128, 40),     # G = 6, many pages, chunk starts mid-page
    (517, 0, 2, 128, 100, 128),     # the whole sequence as one chunk, ragged last page
    (1000, 999, 8, 1024, 256, 65),  # one query, one page holding the whole sequence
    (2100, 1500, 2, 256, 512, 200),
])
def test_paged_chunk_bit_identical_to_dense(T, P, g, page_size, w_pre, w0):
    """Shuffled pages, NaN in every row no one may read: the paged call's output
    and LSE equal the dense-cache chunk's bit for bit."""
    B, Hkv = 2, 2
    q, k, v = synth.prefill_inputs(B, g * Hkv, Hkv, T, 128, seed=T + page_size,
                                   outlier_channels=8)
    kp, vp, table = _pool(k, v, page_size, seed=T, max_pages=(T + page_size - 1) // page_size + 2)
    say("paged chunk T=%d P=%d page_size=%d pages=%d" % (T, P, page_size, kp.shape[0]))
    out, lse = _paged_chunk(q[:, P:], kp, vp, table, P, w_pre, w0)
    kc = np.full((B, T + 37, Hkv, 128), NAN, dtype=np.uint16)
    vc = kc.copy()
    kc[:, :T], vc[:, :T] = k, v
    say("dense chunk T=%d P=%d" % (T, P))
    want, want_lse = api.prefill_chunk(to_dev(q[:, P:]), to_dev(kc), to_dev(vc), q_start=P,
                                       w_pretrained=w_pre, w_local=w0, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), want.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), want_lse.view(torch.int32))
    rows = np.array([[b, h, x] for b in range(B) for h in range(g * Hkv)
                     for x in range(P, T, 29)], dtype=np.int64)
    ref, _ = O.prefill_rows(q, k, v, rows, theta=1e6, w_pretrained=w_pre, w_local=w0)
    assert_close(to_f64(out)[rows[:, 0], rows[:, 2] - P, rows[:, 1]], ref,
                 what="paged chunk T=%d P=%d" % (T, P))


def test_paged_chunks_across_g_transitions_on_one_pool():
    """A 2048-token sequence in four chunks of 512 over one paged pool that no
    call rewrites: G = 2, 4, 6, 8 from the growing length (w_pretrained = 256)."""
    B, Hq, Hkv, T, w_pre, w0, page_size = 2, 8, 2, 2048, 256, 100, 128
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, T, 128, seed=78, outlier_channels=8)
    kp, vp, table = _pool(k, v, page_size, seed=5)
    kp_d, vp_d, table_d = to_dev(kp), to_dev(vp), torch.from_numpy(table).cuda()
    kp0, vp0 = kp_d.clone(), vp_d.clone()
    for c in range(4):
        P, n = 512 * c, 512
        L = P + n
        say("paged chunk %d: P=%d L=%d G=%d" % (c, P, L, api.group_size(L, w_pre)))
        out = api.prefill_chunk_paged(to_dev(q[:, P:L]), kp_d, vp_d, table_d, q_start=P,
                                      w_pretrained=w_pre, w_local=w0)
        torch.cuda.synchronize()
        rows = np.array([[b, h, x] for b in range(B) for h in range(Hq) for x in range(P, L, 7)],
                        dtype=np.int64)
        want, _ = O.prefill_rows(q[:, :L], k[:, :L], v[:, :L], rows, theta=1e6,
                                 w_pretrained=w_pre, w_local=w0)
        o = to_f64(out)
        assert_close(o[rows[:, 0], rows[:, 2] - P, rows[:, 1]], want, what="paged chunk %d" % c)
        assert np.isfinite(o).all()
    assert torch.equal(kp_d.view(torch.int16), kp0.view(torch.int16))
    assert torch.equal(vp_d.view(torch.int16), vp0.view(torch.int16))


def test_vanilla_paged_chunk_matches_dense():
    B, Hq, Hkv, T, P, page_size = 1, 4, 2, 400, 150, 64
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, T, 128, seed=4)
    kp, vp, table = _pool(k, v, page_size, seed=9)
    say("vanilla paged chunk")
    out, lse = _paged_chunk(q[:, P:], kp, vp, table, P, 1, 0, bifocal=False)
    want, want_lse = api.prefill_chunk(to_dev(q[:, P:]), to_dev(k), to_dev(v), q_start=P,
                                       bifocal=False, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), want.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), want_lse.view(torch.int32))


def test_out_of_range_table_entries_are_clamped():
    """Entries outside [0, n_pages) read the nearest end page, as the dense
    cache built from the clamped table does; entries past the sequence's pages
    are never read."""
    B, Hq, Hkv, T, P, page_size, w_pre, w0 = 1, 4, 2, 640, 200, 64, 128, 30
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, T, 128, seed=12)
    kp, vp, table = _pool(k, v, page_size, seed=2, max_pages=14, spare_pages=0)
    kp[:] = np.where(kp == NAN, np.uint16(0), kp)  # every page finite
    vp[:] = np.where(vp == NAN, np.uint16(0), vp)
    table[0, 3] = -7
    table[0, 6] = 10 ** 6
    table[0, 10:] = [2 ** 31 - 1, -(2 ** 31), 5, -1]
    say("paged chunk with clamped entries")
    out, lse = _paged_chunk(q[:, P:], kp, vp, table, P, w_pre, w0)
    kc, vc = _dense_of(kp, vp, table, T)
    want, want_lse = api.prefill_chunk(to_dev(q[:, P:]), to_dev(kc), to_dev(vc), q_start=P,
                                       w_pretrained=w_pre, w_local=w0, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), want.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), want_lse.view(torch.int32))


def test_paged_chunk_checked_pass_equals_dense():
    """With the rescale bound lowered to 2^3 nearly every block of the chunk
    goes through the checked rerun, whose paged instance must give the dense
    chunk's bits too, and the oracle's values."""
    B, Hq, Hkv, T, P, page_size, w_pre, w0 = 1, 8, 2, 900, 400, 128, 200, 50
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, T, 128, seed=31, outlier_channels=8)
    kp, vp, table = _pool(k, v, page_size, seed=6)
    old = api.debug_prefill_rescale_log2(3.0)
    try:
        say("paged chunk, checked pass on every block")
        out, lse = _paged_chunk(q[:, P:], kp, vp, table, P, w_pre, w0)
        want, want_lse = api.prefill_chunk(to_dev(q[:, P:]), to_dev(k), to_dev(v), q_start=P,
                                           w_pretrained=w_pre, w_local=w0, want_lse=True)
        torch.cuda.synchronize()
    finally:
        api.debug_prefill_rescale_log2(old)
    assert torch.equal(out.view(torch.int16), want.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), want_lse.view(torch.int32))
    rows = np.array([[0, h, x] for h in range(Hq) for x in range(P, T, 13)], dtype=np.int64)
    ref, _ = O.prefill_rows(q, k, v, rows, theta=1e6, w_pretrained=w_pre, w_local=w0)
    assert_close(to_f64(out)[rows[:, 0], rows[:, 2] - P, rows[:, 1]], ref,
                 what="paged chunk, checked pass")
