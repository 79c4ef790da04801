"""Continued (chunked) prefill over an existing raw cache: jl_bifocal_prefill_chunk
against the full prefill and the fp64 oracle."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import assert_close, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _cache(k, v, max_len):
    """Place [B, T, Hkv, d] keys/values in caches of max_len rows, NaN past T."""
    B, T, Hkv, d = k.shape
    nan = np.uint16(0x7FC0)
    kc = np.full((B, max_len, Hkv, d), nan, dtype=np.uint16)
    vc = np.full((B, max_len, Hkv, d), nan, dtype=np.uint16)
    kc[:, :T], vc[:, :T] = k, v
    return to_dev(kc), to_dev(vc)


@pytest.mark.parametrize("T,P,g,w_pre,w0", [(300, 200, 4, 70, 20), (517, 1, 2, 100, 128),
                                             (640, 0, 8, 128, 65), (700, 699, 2, 64, 30)])
def test_chunk_equals_full_prefill_rows(T, P, g, w_pre, w0):
    """The chunk's rows are bit-identical to rows P .. T-1 of the full prefill of
    length T, and match the oracle."""
    B, Hkv = 1, 2
    q, k, v = synth.prefill_inputs(B, g * Hkv, Hkv, T, 128, seed=T + P, outlier_channels=8)
    say("full prefill T=%d for chunk P=%d" % (T, P))
    full = api.bifocal_prefill(to_dev(q), to_dev(k), to_dev(v), w_pretrained=w_pre, w_local=w0)
    kc, vc = _cache(k, v, T + 37)
    say("chunk prefill T=%d P=%d g=%d" % (T, P, g))
    out, lse = api.prefill_chunk(to_dev(q[:, P:]), kc, vc, q_start=P, w_pretrained=w_pre,
                                 w_local=w0, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), full[:, P:].view(torch.int16))
    rows = np.array([[0, h, x] for h in range(g * Hkv) for x in range(P, T)], dtype=np.int64)
    want, want_lse, _ = O.prefill_rows(q, k, v, rows, theta=1e6, w_pretrained=w_pre, w_local=w0,
                                       want_lse=True)
    o = to_f64(out)
    got = o[0, rows[:, 2] - P, rows[:, 1]]
    assert_close(got, want, what="chunk T=%d P=%d" % (T, P))
    got_lse = lse.cpu().numpy()[0, rows[:, 1], rows[:, 2] - P]
    assert_close(got_lse, want_lse, max_abs=5e-2, mean_abs=5e-3, what="chunk lse")


def test_chunks_across_g_transitions():
    """A 2048-token sequence in four chunks of 512 over one untouched cache;
    G = 2, 4, 6, 8 from the growing length (w_pretrained = 256)."""
    B, Hq, Hkv, T, w_pre, w0 = 2, 8, 2, 2048, 256, 100
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, T, 128, seed=77, outlier_channels=8)
    kc, vc = _cache(k, v, T)
    for c in range(4):
        P, n = 512 * c, 512
        L = P + n
        say("chunk %d: P=%d L=%d G=%d" % (c, P, L, api.group_size(L, w_pre)))
        out = api.prefill_chunk(to_dev(q[:, P:L]), kc, vc, q_start=P, w_pretrained=w_pre,
                                w_local=w0)
        torch.cuda.synchronize()
        rows = np.array([[b, h, x] for b in range(B) for h in range(Hq) for x in range(P, L, 7)],
                        dtype=np.int64)
        want, _ = O.prefill_rows(q[:, :L], k[:, :L], v[:, :L], rows, theta=1e6,
                                 w_pretrained=w_pre, w_local=w0)
        o = to_f64(out)
        assert_close(o[rows[:, 0], rows[:, 2] - P, rows[:, 1]], want, what="chunk %d" % c)
        assert np.isfinite(o).all()


def test_vanilla_chunk_matches_rope_attention_rows():
    B, Hq, Hkv, T, P = 1, 4, 2, 400, 150
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, T, 128, seed=3)
    say("vanilla chunk")
    full = api.rope_attention(to_dev(q), to_dev(k), to_dev(v))
    kc, vc = _cache(k, v, 512)
    out = api.prefill_chunk(to_dev(q[:, P:]), kc, vc, q_start=P, bifocal=False)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), full[:, P:].view(torch.int16))


def test_chunk_rejects_cache_too_short():
    q = torch.zeros((1, 16, 4, 128), dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros((1, 100, 2, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(api.JetLongError) as e:
        api.prefill_chunk(q, kc, kc, q_start=90, w_pretrained=32, w_local=4)
    assert e.value.status == api.JL_ERR_INVALID_ARG
