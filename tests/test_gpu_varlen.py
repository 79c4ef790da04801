"""Packed variable-length prefill: jl_bifocal_prefill_varlen against the fp64
oracle on each sequence's slice and against per-sequence calls of
jl_bifocal_prefill (same kernels, so bit-identical)."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import assert_close, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _pack(lens, Hq, Hkv, seed):
    """Sequences of the given lengths packed along one token axis."""
    T = int(sum(lens))
    q, k, v = synth.prefill_inputs(1, Hq, Hkv, T, 128, seed=seed, outlier_channels=8)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    return q[0], k[0], v[0], cu


def _varlen(q, k, v, cu, max_seqlen, bifocal, w, w0, want_lse=True):
    qd = to_dev(q)
    out = torch.full_like(qd, float("nan"))
    lse = torch.full((q.shape[1], q.shape[0]), float("nan"), device="cuda") if want_lse else None
    api.prefill_varlen(qd, to_dev(k), to_dev(v), torch.from_numpy(cu).cuda(),
                       max_seqlen=max_seqlen, w_pretrained=w, w_local=w0, bifocal=bifocal,
                       out=out, lse=lse)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("g", [1, 4, 8])
def test_varlen_matches_oracle_per_sequence(g):
    """Lengths around the tile and window edges, G = 1 .. 6 across sequences
    (w_pretrained = 100), an empty sequence in the middle."""
    Hkv, w, w0 = 2, 100, 30
    lens = [300, 1, 0, 64, 65, 517, 100, 129, 37]
    q, k, v, cu = _pack(lens, g * Hkv, Hkv, seed=g)
    say("varlen prefill g=%d T=%d lens=%s" % (g, cu[-1], lens))
    out, lse = _varlen(q, k, v, cu, max(lens), True, w, w0)
    o, ls = to_f64(out), lse.cpu().numpy()
    for s, L in enumerate(lens):
        if L == 0:
            continue
        a, b = cu[s], cu[s + 1]
        want, want_lse = O.prefill(q[None, a:b], k[None, a:b], v[None, a:b], theta=1e6,
                                   w_pretrained=w, w_local=w0)
        assert_close(o[a:b], want[0], what="seq %d L=%d G=%d" % (s, L, api.group_size(L, w)))
        assert_close(ls[:, a:b], want_lse[0], max_abs=5e-2, mean_abs=5e-3, what="lse %d" % s)


@pytest.mark.parametrize("bifocal", [True, False])
def test_varlen_equals_per_sequence_calls(bifocal):
    """Each sequence's rows (and LSE) are bit-identical to a call on that
    sequence alone; G = 1 sequences give the vanilla kernel's bits."""
    Hq, Hkv, w, w0 = 16, 4, 256, 64
    lens = [1000, 3, 256, 257, 2049, 64, 700]
    q, k, v, cu = _pack(lens, Hq, Hkv, seed=11)
    say("varlen vs per-sequence, bifocal=%s" % bifocal)
    out, lse = _varlen(q, k, v, cu, max(lens), bifocal, w, w0)
    for s, L in enumerate(lens):
        a, b = cu[s], cu[s + 1]
        one, one_lse = api._prefill(bifocal, to_dev(q[None, a:b]), to_dev(k[None, a:b]),
                                    to_dev(v[None, a:b]), w, w0, 1e6, None, None, True, None)
        torch.cuda.synchronize()
        assert torch.equal(out[a:b].view(torch.int16), one[0].view(torch.int16)), s
        assert torch.equal(lse[:, a:b], one_lse[0]), s


def test_varlen_malformed_offsets_are_clamped():
    """cu = [0, 100, 50, 300, 10**9] over T = 300: the third sequence is rows
    50 .. 299 (the decreasing step clamps), the second and fourth are empty.
    Rows 100 .. 299 hold that sequence's positions 50 .. 249."""
    Hq, Hkv, w, w0, T = 8, 2, 64, 16, 300
    q, k, v = (x[0] for x in synth.prefill_inputs(1, Hq, Hkv, T, 128, seed=5))
    cu = np.array([0, 100, 50, 300, 10 ** 9], dtype=np.int32)
    say("varlen with clamped offsets")
    out, _ = _varlen(q, k, v, cu, T, True, w, w0, want_lse=False)
    rows = np.array([[0, h, x] for h in range(Hq) for x in range(50, 250, 3)], dtype=np.int64)
    want, _ = O.prefill_rows(q[None, 50:], k[None, 50:], v[None, 50:], rows, theta=1e6,
                             w_pretrained=w, w_local=w0)
    o = to_f64(out)
    assert_close(o[rows[:, 2] + 50, rows[:, 1]], want, what="clamped sequence")


def test_varlen_overfull_lists_skip_sequence():
    """cu = [0, 300, 0, 300]: two full-length sequences cannot both fit the
    work lists sized for 300 tokens; the third is skipped and every row holds
    the first sequence's result, bit for bit."""
    Hq, Hkv, w, w0, T = 8, 2, 64, 16, 300
    q, k, v = (x[0] for x in synth.prefill_inputs(1, Hq, Hkv, T, 128, seed=6))
    cu = np.array([0, 300, 0, 300], dtype=np.int32)
    say("varlen with overfull work lists")
    out, _ = _varlen(q, k, v, cu, T, True, w, w0, want_lse=False)
    one = api.bifocal_prefill(to_dev(q[None]), to_dev(k[None]), to_dev(v[None]),
                              w_pretrained=w, w_local=w0)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), one[0].view(torch.int16))


def test_varlen_max_seqlen_cuts_sequences():
    """A sequence longer than max_seqlen is cut to its first max_seqlen rows;
    the rows past the cut keep their previous contents."""
    Hq, Hkv, w, w0 = 8, 2, 64, 16
    lens = [200, 90]
    q, k, v, cu = _pack(lens, Hq, Hkv, seed=8)
    say("varlen with max_seqlen 120")
    out, _ = _varlen(q, k, v, cu, 120, True, w, w0, want_lse=False)
    o = to_f64(out)
    assert np.isnan(o[120:200]).all()
    for a, L in ((0, 120), (200, 90)):
        want, _ = O.prefill(q[None, a:a + L], k[None, a:a + L], v[None, a:a + L], theta=1e6,
                            w_pretrained=w, w_local=w0)
        assert_close(o[a:a + L], want[0], what="cut seq at %d" % a)


def test_varlen_many_short_sequences():
    """1500 sequences (more than one planning chunk of 1024) of 0 .. 40 tokens."""
    Hq, Hkv, w, w0 = 8, 8, 16, 4
    rng = np.random.default_rng(3)
    lens = [int(x) for x in rng.integers(0, 41, size=1500)]
    q, k, v, cu = _pack(lens, Hq, Hkv, seed=9)
    say("varlen with %d short sequences, T=%d" % (len(lens), cu[-1]))
    out, _ = _varlen(q, k, v, cu, 40, True, w, w0, want_lse=False)
    o = to_f64(out)
    assert np.isfinite(o).all()
    for s in [0, 1, 2, 1023, 1024, 1025, 1499] + [int(x) for x in rng.integers(0, 1500, 8)]:
        a, b = cu[s], cu[s + 1]
        if a == b:
            continue
        want, _ = O.prefill(q[None, a:b], k[None, a:b], v[None, a:b], theta=1e6, w_pretrained=w,
                            w_local=w0)
        assert_close(o[a:b], want[0], what="short seq %d L=%d" % (s, b - a))


def test_varlen_mixed_long_batch_equals_per_sequence():
    """Qwen3-8B heads (32 / 8), w_pretrained 4096, w_local 1024: a 32K
    sequence beside 9K, 4K and short ones, each bit-identical to its own call."""
    Hq, Hkv, w, w0 = 32, 8, 4096, 1024
    lens = [32768, 9000, 4096, 4097, 129, 1]
    q, k, v, cu = _pack(lens, Hq, Hkv, seed=12)
    say("varlen mixed long batch T=%d" % cu[-1])
    out, _ = _varlen(q, k, v, cu, max(lens), True, w, w0, want_lse=False)
    for s, L in enumerate(lens):
        a, b = cu[s], cu[s + 1]
        one = api.bifocal_prefill(to_dev(q[None, a:b]), to_dev(k[None, a:b]),
                                  to_dev(v[None, a:b]), w_pretrained=w, w_local=w0)
        torch.cuda.synchronize()
        assert torch.equal(out[a:b].view(torch.int16), one[0].view(torch.int16)), s
    a = cu[0]
    rows = np.array([[0, h, x] for h in (0, 13, 31) for x in (0, 1023, 1024, 1025, 4095, 4096,
                                                           20000, 32767)], dtype=np.int64)
    want, _ = O.prefill_rows(q[None, :32768], k[None, :32768], v[None, :32768], rows, theta=1e6,
                             w_pretrained=w, w_local=w0)
    assert_close(to_f64(out)[rows[:, 2], rows[:, 1]], want, what="32K rows")


@pytest.mark.parametrize("g", [1, 4])
def test_varlen_freq_map_per_sequence(g):
    """jl_bifocal_prefill_varlen_map with the frequency map (Sec. 4.5): each
    sequence takes the map of its own length (factors 1 .. 5.2 here), its rows
    and LSE bit-identical to jl_bifocal_prefill_map on that sequence alone and
    matching the oracle's frequency map; the alias choice is the plain varlen
    call bit for bit."""
    Hkv, w, w0 = 2, 100, 30
    lens = [300, 1, 0, 64, 65, 517, 100, 129, 37]
    q, k, v, cu = _pack(lens, g * Hkv, Hkv, seed=20 + g)
    T = int(cu[-1])
    qd, kd, vd, cud = to_dev(q), to_dev(k), to_dev(v), torch.from_numpy(cu).cuda()
    say("varlen freq-map prefill g=%d T=%d" % (g, T))
    out = torch.full_like(qd, float("nan"))
    lse = torch.full((q.shape[1], T), float("nan"), device="cuda")
    api.prefill_varlen(qd, kd, vd, cud, max_seqlen=max(lens), w_pretrained=w, w_local=w0,
                       out=out, lse=lse, remote_map="freq")
    alias_map = api.prefill_varlen(qd, kd, vd, cud, max_seqlen=max(lens), w_pretrained=w,
                                   w_local=w0, remote_map="alias")
    alias = api.prefill_varlen(qd, kd, vd, cud, max_seqlen=max(lens), w_pretrained=w,
                               w_local=w0)
    torch.cuda.synchronize()
    assert torch.equal(alias_map.view(torch.int16), alias.view(torch.int16))
    o, ls = to_f64(out), lse.cpu().numpy()
    for s, L in enumerate(lens):
        if L == 0:
            continue
        a, b = cu[s], cu[s + 1]
        one, one_lse = api.bifocal_prefill(to_dev(q[None, a:b]), to_dev(k[None, a:b]),
                                           to_dev(v[None, a:b]), w_pretrained=w, w_local=w0,
                                           want_lse=True, remote_map="freq")
        torch.cuda.synchronize()
        assert torch.equal(out[a:b].view(torch.int16), one[0].view(torch.int16)), s
        assert torch.equal(lse[:, a:b], one_lse[0]), s
        want, _ = O.prefill(q[None, a:b], k[None, a:b], v[None, a:b], theta=1e6, w_pretrained=w,
                            w_local=w0, remote_map="freq")
        assert_close(o[a:b], want[0], what="freq seq %d L=%d" % (s, L))
