"""Decode on a paged raw cache: jl_bifocal_decode_paged against the dense-cache
kernels and the fp64 oracle (which reads the same keys from a dense cache)."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import assert_close, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

NAN = np.uint16(0x7FC0)


def _paginate(kc, vc, lens, page_size, seed, spare_pages=3):
    """Scatter dense caches [B, max_len, Hkv, d] into shuffled pages of a pool;
    pages nobody uses (and rows past each length) hold NaN."""
    B, max_len, Hkv, d = kc.shape
    max_pages = (max_len + page_size - 1) // page_size
    n_used = sum((int(n) + page_size - 1) // page_size for n in lens)
    n_pages = n_used + spare_pages
    rng = np.random.default_rng(seed)
    order = rng.permutation(n_pages)
    kp = np.full((n_pages, page_size, Hkv, d), NAN, dtype=np.uint16)
    vp = np.full((n_pages, page_size, Hkv, d), NAN, dtype=np.uint16)
    table = np.full((B, max_pages), -1, dtype=np.int32)
    nxt = 0
    for b in range(B):
        for j in range((int(lens[b]) + page_size - 1) // page_size):
            pg = int(order[nxt])
            nxt += 1
            table[b, j] = pg
            lo, hi = j * page_size, min((j + 1) * page_size, int(lens[b]))
            kp[pg, :hi - lo] = kc[b, lo:hi]
            vp[pg, :hi - lo] = vc[b, lo:hi]
    return kp, vp, table


def _paged(bifocal, q, kp, vp, table, lens, w, w0):
    out = api.decode_paged(to_dev(q), to_dev(kp), to_dev(vp),
                           torch.from_numpy(table).cuda(),
                           torch.from_numpy(np.asarray(lens, dtype=np.int32)).cuda(),
                           w_pretrained=w, w_local=w0, bifocal=bifocal)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("page_size", [16, 64, 256])
def test_paged_decode_matches_oracle_across_g(page_size):
    Hq, Hkv, w_pre, w0 = 8, 2, 96, 20
    max_len = 4 * w_pre + 40
    lens = [1, w0 + 1, w_pre, w_pre + 1, 2 * w_pre + 1, 3 * w_pre + 7, max_len]
    B = len(lens)
    q, kc, vc, lens = synth.decode_inputs(B, Hq, Hkv, max_len, lens, seed=page_size,
                                          nan_tail=True)
    kp, vp, table = _paginate(kc, vc, lens, page_size, seed=page_size)
    say("paged decode page_size=%d pages=%d" % (page_size, kp.shape[0]))
    for bif in (True, False):
        out = _paged(bif, q, kp, vp, table, lens, w_pre, w0)
        want, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=w_pre, w_local=w0,
                              bifocal=bif)
        assert_close(to_f64(out), want, what="paged %d bifocal=%s" % (page_size, bif))


def test_paged_equals_dense_at_128k():
    """Same keys in the same order: the paged decode is bit-identical to the
    dense one on the Qwen3-4B-like 128K workload (pages of 256 keys)."""
    w = synth.WORKLOADS["qwen3_4b_decode_128k"]
    say("generating decode 4b 128k")
    q, kc, vc, lens = synth.make_inputs(w)
    kp, vp, table = _paginate(kc, vc, lens, 256, seed=1, spare_pages=1)
    say("dense decode")
    dense = api.bifocal_decode(to_dev(q), to_dev(kc), to_dev(vc),
                               torch.from_numpy(lens).cuda(), w_pretrained=w.w_pretrained,
                               w_local=w.w_local)
    del kc, vc
    say("paged decode, %d pages" % kp.shape[0])
    paged = _paged(True, q, kp, vp, table, lens, w.w_pretrained, w.w_local)
    assert torch.equal(dense.view(torch.int16), paged.view(torch.int16))


def test_paged_table_entries_out_of_range_are_clamped():
    """Entries below 0 or past the pool read the first or last page: wrong
    values, but every read stays inside the pool."""
    B, Hq, Hkv, page_size, n_pages = 2, 4, 2, 16, 5
    q = synth.prefill_inputs(1, B * Hq, 1, 1, 128, seed=4)[0].reshape(B, Hq, 128)
    kp = synth.prefill_inputs(1, 1, 1, n_pages * page_size * Hkv, 128, seed=5)[1].reshape(
        n_pages, page_size, Hkv, 128)
    vp = synth.prefill_inputs(1, 1, 1, n_pages * page_size * Hkv, 128, seed=6)[2].reshape(
        n_pages, page_size, Hkv, 128)
    table = np.array([[-7, 1, 10 ** 6], [2, -1, 4]], dtype=np.int32)
    lens = [40, 48]
    say("paged decode with clamped table entries")
    out = _paged(True, q, kp, vp, table, lens, 16, 4)
    clamped = np.clip(table, 0, n_pages - 1)
    kc = np.stack([np.concatenate([kp[p] for p in clamped[b]]) for b in range(B)])
    vc = np.stack([np.concatenate([vp[p] for p in clamped[b]]) for b in range(B)])
    want, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=16, w_local=4)
    assert_close(to_f64(out), want, what="clamped pages")


@pytest.mark.parametrize("page_size", [16, 128])
def test_paged_freq_map_decode(page_size):
    """jl_bifocal_decode_paged_map: the frequency map (Sec. 4.5) on shuffled
    pages equals the dense frequency-map decode bit for bit and matches the
    oracle, across factors s = L / w_pretrained; the alias choice is the plain
    paged decode."""
    Hq, Hkv, w_pre, w0 = 8, 2, 96, 20
    max_len = 4 * w_pre + 40
    lens = [1, w0 + 1, w_pre, w_pre + 1, 2 * w_pre + 1, 3 * w_pre + 7, max_len]
    B = len(lens)
    q, kc, vc, lens = synth.decode_inputs(B, Hq, Hkv, max_len, lens, seed=page_size + 7,
                                          nan_tail=True)
    kp, vp, table = _paginate(kc, vc, lens, page_size, seed=page_size + 1)
    ld = torch.from_numpy(np.asarray(lens, dtype=np.int32)).cuda()
    say("paged freq-map decode page_size=%d" % page_size)
    paged = api.decode_paged(to_dev(q), to_dev(kp), to_dev(vp), torch.from_numpy(table).cuda(),
                             ld, w_pretrained=w_pre, w_local=w0, remote_map="freq")
    dense = api.bifocal_decode(to_dev(q), to_dev(kc), to_dev(vc), ld, w_pretrained=w_pre,
                               w_local=w0, remote_map="freq")
    alias_map = api.decode_paged(to_dev(q), to_dev(kp), to_dev(vp),
                                 torch.from_numpy(table).cuda(), ld, w_pretrained=w_pre,
                                 w_local=w0, remote_map="alias")
    alias = _paged(True, q, kp, vp, table, lens, w_pre, w0)
    torch.cuda.synchronize()
    assert torch.equal(paged.view(torch.int16), dense.view(torch.int16))
    assert torch.equal(alias_map.view(torch.int16), alias.view(torch.int16))
    want, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=w_pre, w_local=w0,
                          bifocal=True, remote_map="freq")
    assert_close(to_f64(paged), want, what="paged freq map %d" % page_size)
