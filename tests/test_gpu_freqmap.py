"""Frequency-interpolation remote map (Sec. 4.5, Table 6 ablation): the HIP
prefill through jl_bifocal_prefill_map against the fp64 oracle."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import (assert_close, prefill_block_q, rows_for, sample_positions, say, to_dev,
                         to_f64)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _run(q, k, v, w, w0, remote_map, theta=1e6, want_lse=False):
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    out = torch.full_like(qd, float("nan"))  # poison: every element must be written
    lse = None
    if want_lse:
        lse = torch.full((q.shape[0], q.shape[2], q.shape[1]), float("nan"), device="cuda")
    api.bifocal_prefill(qd, kd, vd, w_pretrained=w, w_local=w0, rope_theta=theta, out=out,
                        lse=lse, remote_map=remote_map)
    torch.cuda.synchronize()
    return (out, lse) if want_lse else out


@pytest.mark.parametrize("L,g,w_pre,w0", [(300, 4, 70, 20), (517, 2, 100, 128), (640, 8, 128, 65),
                                          (129, 1, 32, 0), (2048, 2, 512, 128)])
def test_freq_map_full_tensor(L, g, w_pre, w0):
    B, Hkv = 1, 2
    q, k, v = synth.prefill_inputs(B, g * Hkv, Hkv, L, 128, seed=L + g, outlier_channels=8)
    say("freq-map prefill L=%d g=%d w_pre=%d w0=%d" % (L, g, w_pre, w0))
    out, lse = _run(q, k, v, w_pre, w0, "freq", want_lse=True)
    want, want_lse = O.prefill(q, k, v, theta=1e6, w_pretrained=w_pre, w_local=w0,
                               remote_map="freq")
    assert_close(to_f64(out), want, what="freq map L=%d" % L)
    assert_close(lse.cpu().numpy(), want_lse, max_abs=5e-2, mean_abs=5e-3, what="freq lse")


def test_freq_map_differs_from_alias_and_alias_entry_matches():
    """The two remote maps give different outputs once L > w_pretrained, and
    jl_bifocal_prefill_map with JL_REMOTE_ALIAS equals jl_bifocal_prefill."""
    B, Hq, Hkv, L, w_pre, w0 = 1, 4, 2, 600, 100, 30
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=5)
    say("freq vs alias prefill")
    fr = to_f64(_run(q, k, v, w_pre, w0, "freq"))
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    al = api.bifocal_prefill(qd, kd, vd, w_pretrained=w_pre, w_local=w0)
    al2 = torch.empty_like(al)
    lib = api.lib()
    import ctypes
    rc = lib.jl_bifocal_prefill_map(ctypes.c_void_p(qd.data_ptr()), ctypes.c_void_p(kd.data_ptr()),
                                    ctypes.c_void_p(vd.data_ptr()), ctypes.c_void_p(al2.data_ptr()),
                                    None, B, Hq, Hkv, L, 128, 1e6, w_pre, w0, 0,
                                    ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert rc == api.JL_OK
    assert torch.equal(al.view(torch.int16), al2.view(torch.int16))
    diff = np.abs(fr - to_f64(al))
    say("freq vs alias max diff %.3e" % diff.max())
    assert diff.max() > 5e-2  # remote rows see really different rotations


def test_freq_map_within_window_is_vanilla():
    """L <= w_pretrained: s = 1, omega' = omega, and the call runs the vanilla
    kernel, bit for bit."""
    B, Hq, Hkv, L = 1, 4, 2, 400
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=11)
    say("freq map within window")
    fr = _run(q, k, v, 400, 50, "freq")
    van = api.rope_attention(to_dev(q), to_dev(k), to_dev(v))
    torch.cuda.synchronize()
    assert torch.equal(fr.view(torch.int16), van.view(torch.int16))


def test_freq_map_1p7b_128k_sampled_rows():
    w = synth.WORKLOADS["qwen3_1p7b_prefill_128k"]
    q, k, v = synth.make_inputs(w)
    G = api.group_size(w.L, w.w_pretrained)
    say("freq-map prefill %s" % w.name)
    out = _run(q, k, v, w.w_pretrained, w.w_local, "freq")
    pos = sample_positions(w.L, w.w_local, w.w_pretrained, G, prefill_block_q(w.Hq, w.Hkv), 16)
    rows = rows_for(w.B, w.Hq, pos)
    say("oracle rows", len(rows))
    want, _ = O.prefill_rows(q, k, v, rows, theta=w.theta, w_pretrained=w.w_pretrained,
                             w_local=w.w_local, remote_map="freq")
    o = out.float().cpu().numpy()
    got = o[rows[:, 0], rows[:, 2], rows[:, 1]].astype(np.float64)
    assert_close(got, want, what="freq map 128K rows")
    assert np.isfinite(o).all()


# ---------------------------------------------------------------- decode
def _decode_freq(q, kc, vc, lens, w, w0, remote_map="freq", theta=1e6):
    B, Hq, _ = q.shape
    Hkv, max_len = kc.shape[2], kc.shape[1]
    nbytes = api.decode_map_workspace_bytes(B, Hq, Hkv, max_len, 128, remote_map)
    ws = torch.full((nbytes // 4,), float("nan"), dtype=torch.float32, device="cuda")
    out = api.bifocal_decode(to_dev(q), to_dev(kc), to_dev(vc),
                             torch.from_numpy(np.asarray(lens, dtype=np.int32)).cuda(),
                             w_pretrained=w, w_local=w0, rope_theta=theta, workspace=ws,
                             remote_map=remote_map)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("g", [1, 4, 8])
def test_freq_map_decode_ragged_across_factors(g):
    """One cache, lengths inside and past the window: every sequence takes the
    frequencies of its own length (s = kv_len / w), NaN past each length."""
    Hkv, w_pre, w0 = 2, 96, 20
    max_len = 4 * w_pre + 40
    lens = [1, w0 + 1, w_pre, w_pre + 1, 2 * w_pre + 1, 3 * w_pre + 7, max_len]
    q, kc, vc, lens = synth.decode_inputs(len(lens), g * Hkv, Hkv, max_len, lens, seed=g,
                                          nan_tail=True, outlier_channels=8)
    say("freq-map decode g=%d" % g)
    out = _decode_freq(q, kc, vc, lens, w_pre, w0)
    want, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=w_pre, w_local=w0,
                          remote_map="freq")
    assert_close(to_f64(out), want, what="freq decode g=%d" % g)
    alias, _, _ = O.decode(q, kc, vc, lens, theta=1e6, w_pretrained=w_pre, w_local=w0)
    assert np.abs(want - alias).max() > 1e-2  # the two maps really differ here


def test_freq_map_decode_4b_128k():
    w = synth.WORKLOADS["qwen3_4b_decode_128k"]
    say("generating decode 4b 128k")
    q, kc, vc, lens = synth.make_inputs(w)
    say("freq-map decode 128k")
    out = _decode_freq(q, kc, vc, lens, w.w_pretrained, w.w_local)
    want, _, _ = O.decode(q, kc, vc, lens, theta=w.theta, w_pretrained=w.w_pretrained,
                          w_local=w.w_local, remote_map="freq")
    assert_close(to_f64(out), want, what="freq decode 128k")


def test_freq_map_decode_matches_prefill_last_row():
    """Decode at kv_len = L and the frequency-map prefill of length L agree on
    the last row (both take s = L / w)."""
    Hq, Hkv, L, w_pre, w0 = 8, 2, 700, 200, 64
    q, k, v = synth.prefill_inputs(1, Hq, Hkv, L, 128, seed=41, outlier_channels=8)
    say("freq-map prefill vs decode, L=%d" % L)
    pre = _run(q, k, v, w_pre, w0, "freq")
    dec = _decode_freq(q[:, L - 1].copy(), k, v, [L], w_pre, w0)
    assert_close(to_f64(dec)[0], to_f64(pre)[0, L - 1], max_abs=1e-2, mean_abs=1e-3,
                 what="decode vs prefill row")


def test_freq_map_decode_alias_entry_equals_plain_decode():
    """jl_bifocal_decode_map with JL_REMOTE_ALIAS is jl_bifocal_decode, bit for bit."""
    Hq, Hkv, w_pre, w0, max_len = 8, 2, 64, 16, 300
    lens = [300, 65, 129]
    q, kc, vc, lens = synth.decode_inputs(3, Hq, Hkv, max_len, lens, seed=43)
    say("decode map alias entry")
    a = _decode_freq(q, kc, vc, lens, w_pre, w0, remote_map="alias")
    b = api.bifocal_decode(to_dev(q), to_dev(kc), to_dev(vc),
                           torch.from_numpy(np.asarray(lens, dtype=np.int32)).cuda(),
                           w_pretrained=w_pre, w_local=w0)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
