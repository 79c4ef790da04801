"""Decode parity on a raw cache: the HIP kernels through the C ABI against the oracle."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import assert_close, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _run(bifocal, q, kc, vc, lens, w, w0, theta=1e6, ws_fill=float("nan")):
    qd, kd, vd = to_dev(q), to_dev(kc), to_dev(vc)
    ld = torch.from_numpy(np.asarray(lens, dtype=np.int32)).cuda()
    out = torch.full_like(qd, float("nan"))
    B, Hq, _ = q.shape
    Hkv, max_len = kc.shape[2], kc.shape[1]
    nbytes = api.decode_workspace_bytes(B, Hq, Hkv, max_len)
    ws = torch.full((nbytes // 4,), ws_fill, dtype=torch.float32, device="cuda")
    if bifocal:
        api.bifocal_decode(qd, kd, vd, ld, w_pretrained=w, w_local=w0, rope_theta=theta, out=out,
                           workspace=ws)
    else:
        api.rope_attention_decode(qd, kd, vd, ld, rope_theta=theta, out=out, workspace=ws)
    torch.cuda.synchronize()
    return out


def test_decode_4b_128k_full():
    w = synth.WORKLOADS["qwen3_4b_decode_128k"]
    say("generating decode 4b 128k")
    q, kc, vc, lens = synth.make_inputs(w)
    for bif in (True, False):
        say("decode bifocal=%s B=%d Hq=%d Hkv=%d kv_len=%d" % (bif, w.B, w.Hq, w.Hkv, lens[0]))
        out = _run(bif, q, kc, vc, lens, w.w_pretrained, w.w_local)
        want, _, _ = O.decode(q, kc, vc, lens, theta=w.theta, w_pretrained=w.w_pretrained,
                              w_local=w.w_local, bifocal=bif)
        assert_close(to_f64(out), want, what="decode 128k bifocal=%s" % bif)


def test_decode_ragged_batch_with_nan_tails():
    w = synth.WORKLOADS["qwen3_4b_decode_b8_ragged"]
    say("generating decode ragged B=8")
    q, kc, vc, lens = synth.make_inputs(w)
    say("decode ragged lens", list(lens))
    out = _run(True, q, kc, vc, lens, w.w_pretrained, w.w_local)
    want, _, _ = O.decode(q, kc, vc, lens, theta=w.theta, w_pretrained=w.w_pretrained,
                          w_local=w.w_local)
    assert_close(to_f64(out), want, what="decode ragged")


@pytest.mark.parametrize("g", [1, 2, 4, 8])
def test_decode_small_shapes_and_g_transitions(g):
    """One untouched raw cache decoded at lengths across G changes (Sec. 3.2)."""
    Hkv, w_pre, w0 = 2, 96, 20
    max_len = 4 * w_pre + 5
    lens = [1, 2, w0, w0 + 1, w0 + 2, w_pre, w_pre + 1, 2 * w_pre, 2 * w_pre + 1, 3 * w_pre + 7,
            max_len]
    B = len(lens)
    q, kc, vc, lens = synth.decode_inputs(B, g * Hkv, Hkv, max_len, lens, seed=g, nan_tail=True,
                                          outlier_channels=8)
    say("decode small g=%d lens=%s" % (g, list(lens)))
    out = _run(True, q, kc, vc, lens, w_pre, w0)
    want, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=w_pre, w_local=w0)
    assert_close(to_f64(out), want, what="decode small g=%d" % g)
    van = _run(False, q, kc, vc, lens, w_pre, w0)
    want_v, _, _ = O.decode(q, kc, vc, lens, theta=1e6, bifocal=False)
    assert_close(to_f64(van), want_v, what="vanilla decode small g=%d" % g)


def test_decode_matches_prefill_last_row():
    Hq, Hkv, L, w_pre, w0 = 8, 2, 777, 200, 50
    qa, ka, va = synth.prefill_inputs(1, Hq, Hkv, L, 128, seed=77)
    say("prefill for decode comparison L=%d" % L)
    qd, kd, vd = to_dev(qa), to_dev(ka), to_dev(va)
    pre = api.bifocal_prefill(qd, kd, vd, w_pretrained=w_pre, w_local=w0)
    say("decode at the last position")
    dec = _run(True, qa[:, L - 1].copy(), ka, va, [L], w_pre, w0)
    a = to_f64(pre[:, L - 1])
    b = to_f64(dec)
    assert_close(b, a, max_abs=2e-2, mean_abs=2e-3, what="decode vs prefill last row")


def test_decode_deterministic_and_workspace_contents_irrelevant():
    Hq, Hkv, max_len = 16, 4, 5000
    lens = [4999, 1234, 5000]
    q, kc, vc, lens = synth.decode_inputs(3, Hq, Hkv, max_len, lens, seed=5)
    say("decode determinism")
    a = _run(True, q, kc, vc, lens, 1024, 100, ws_fill=float("nan"))
    b = _run(True, q, kc, vc, lens, 1024, 100, ws_fill=0.0)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("B", [2, 64, 65])
def test_decode_batch_split_plans(B):
    """Split counts balanced over the actual lengths (B <= 64: one short and
    long sequences side by side, so most workgroups go to the long ones) and
    the max_len-based split of larger batches (B = 65); NaN tails catch any
    read past a length."""
    Hq, Hkv, w_pre, w0, max_len = 8, 8, 512, 100, 4096
    rng = np.random.default_rng(B)
    lens = [int(x) for x in rng.integers(1, max_len + 1, size=B)]
    lens[0], lens[-1] = max_len, 1
    q, kc, vc, lens = synth.decode_inputs(B, Hq, Hkv, max_len, lens, seed=B, nan_tail=True)
    say("decode split plans B=%d" % B)
    for bif in (True, False):
        out = _run(bif, q, kc, vc, lens, w_pre, w0)
        want, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=w_pre, w_local=w0,
                              bifocal=bif)
        assert_close(to_f64(out), want, what="decode B=%d bifocal=%s" % (B, bif))


def test_decode_lengths_outside_range_are_clamped():
    """kv_lens lives on the device, so the host cannot check it: a length below
    1 reads as 1 and one past max_len as max_len, bit for bit, with no read
    outside the cache (NaN tails past every clamped length would show one)."""
    Hq, Hkv, w_pre, w0, max_len = 8, 2, 256, 64, 1000
    bad = [0, -7, max_len + 50, 2 ** 31 - 1, 700]
    good = [1, 1, max_len, max_len, 700]
    q, kc, vc, _ = synth.decode_inputs(len(bad), Hq, Hkv, max_len, good, seed=17, nan_tail=True)
    say("decode clamped lens", bad)
    for bif in (True, False):
        a = _run(bif, q, kc, vc, bad, w_pre, w0)
        b = _run(bif, q, kc, vc, good, w_pre, w0)
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
        want, _, _ = O.decode(q, kc, vc, good, theta=1e6, w_pretrained=w_pre, w_local=w0,
                              bifocal=bif)
        assert_close(to_f64(a), want, what="clamped lens bifocal=%s" % bif)


@pytest.mark.parametrize("Hkv,g", [(3, 2), (6, 1), (6, 4)])
def test_decode_partial_head_groups(Hkv, g):
    """A workgroup serves up to 4 kv heads: Hkv = 3 leaves one group of three,
    Hkv = 6 a full group beside a group of two, whose unused copy slots land
    in a slot nobody reads.  Ragged lengths with NaN tails, both kernels."""
    Hq, w_pre, w0, max_len = g * Hkv, 256, 40, 3000
    lens = [3000, 1, 1777, 257]
    q, kc, vc, lens = synth.decode_inputs(len(lens), Hq, Hkv, max_len, lens, seed=Hkv * 10 + g,
                                          nan_tail=True)
    say("decode partial head groups Hkv=%d g=%d" % (Hkv, g))
    for bif in (True, False):
        out = _run(bif, q, kc, vc, lens, w_pre, w0)
        want, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=w_pre, w_local=w0,
                              bifocal=bif)
        assert_close(to_f64(out), want, what="Hkv=%d g=%d bifocal=%s" % (Hkv, g, bif))


def test_decode_band_covering_every_key_is_vanilla():
    """w_local >= kv_len - 1 for every sequence: no key takes the remote view
    and the bifocal decode gives the vanilla decode's output bit for bit,
    whatever G each length gives (here 1 to 12)."""
    Hq, Hkv, w_pre, max_len = 8, 2, 256, 3000
    lens = [3000, 2999, 257, 1, 1500]
    q, kc, vc, lens = synth.decode_inputs(len(lens), Hq, Hkv, max_len, lens, seed=31, nan_tail=True)
    say("decode band over every key")
    a = _run(True, q, kc, vc, lens, w_pre, max_len - 1)
    b = _run(False, q, kc, vc, lens, w_pre, 0)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    c = _run(True, q, kc, vc, lens, w_pre, 2 ** 31 - 1)  # the largest w_local
    assert torch.equal(c.view(torch.int16), b.view(torch.int16))
    want, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=w_pre, w_local=max_len - 1)
    assert_close(to_f64(a), want, what="decode band over every key")


@pytest.mark.parametrize("w_pre,w0", [(1, 0), (1, 5), (7, 0)])
def test_decode_extreme_windows(w_pre, w0):
    """w_pretrained = 1 makes G the length itself, so every remote key sits
    at position f(k) = 0 (no rotation at all); w_local = 0 leaves only the
    query's own key in the band (Sec. 4's attention-to-self case)."""
    Hq, Hkv, max_len = 8, 2, 700
    lens = [700, 1, 2, 65, 333]
    q, kc, vc, lens = synth.decode_inputs(len(lens), Hq, Hkv, max_len, lens, seed=w_pre * 10 + w0,
                                          nan_tail=True)
    say("decode w_pre=%d w0=%d" % (w_pre, w0))
    out = _run(True, q, kc, vc, lens, w_pre, w0)
    want, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=w_pre, w_local=w0)
    assert_close(to_f64(out), want, what="decode w_pre=%d w0=%d" % (w_pre, w0))
