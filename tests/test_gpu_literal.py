"""Literal Eq. (7) prefill (three window passes and a merge) against the oracle.

The oracle computes windows A, B and C separately in fp64 and merges them
literally (Sec. 3.3, Eq. (7)), so it checks both the merged output and each
window state the GPU leaves in the caller's workspace.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import assert_close, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _literal(q, k, v, w, w0, theta=1e6):
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    B, L, Hq, D = q.shape
    Hkv = k.shape[2]
    out = torch.full_like(qd, float("nan"))
    lse = torch.full((B, Hq, L), float("nan"), device="cuda")
    need = api.prefill_literal_workspace_bytes(B, Hq, Hkv, L)
    ws = torch.full((need // 4,), float("nan"), device="cuda").view(torch.uint8)
    api.bifocal_prefill_literal(qd, kd, vd, w_pretrained=w, w_local=w0, rope_theta=theta,
                                out=out, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    return out, lse, ws


@pytest.mark.parametrize("L,g,w_pre,w0", [
    (2, 2, 1, 0), (63, 4, 16, 5), (65, 2, 20, 0), (129, 1, 32, 64), (300, 4, 70, 20),
    (517, 2, 100, 128), (640, 8, 128, 65),
])
def test_literal_full_tensor(L, g, w_pre, w0):
    B, Hkv = 2, 2
    q, k, v = synth.prefill_inputs(B, g * Hkv, Hkv, L, 128, seed=7 * L + g, outlier_channels=8)
    say("literal prefill L=%d g=%d w_pre=%d w0=%d" % (L, g, w_pre, w0))
    out, lse, _ = _literal(q, k, v, w_pre, w0)
    want, want_lse = O.prefill(q, k, v, theta=1e6, w_pretrained=w_pre, w_local=w0)
    assert_close(to_f64(out), want, what="literal L=%d g=%d" % (L, g))
    assert_close(lse.cpu().numpy(), want_lse, max_abs=5e-2, mean_abs=5e-3, what="literal lse")


def test_literal_tiny_workload_and_window_states():
    """Tiny workload (L = 2048, G = 4): merged output on every row, and the
    three window states O_X, LSE_X on sampled rows of both heads."""
    w = synth.WORKLOADS["tiny_prefill"]
    q, k, v = synth.make_inputs(w)
    B, L, Hq, D = q.shape
    say("literal tiny prefill", q.shape)
    out, lse, ws = _literal(q, k, v, w.w_pretrained, w.w_local)
    want, want_lse = O.prefill(q, k, v, theta=w.theta, w_pretrained=w.w_pretrained,
                               w_local=w.w_local)
    assert_close(to_f64(out), want, what="literal tiny")
    assert_close(lse.cpu().numpy(), want_lse, max_abs=5e-2, mean_abs=5e-3, what="tiny lse")
    o3, l3 = api.literal_window_states(ws, B, Hq, L)
    o3, l3 = o3.cpu().numpy().astype(np.float64), l3.cpu().numpy().astype(np.float64)
    rows = [0, 1, 63, 64, 127, 128, 129, 130, 511, 512, 1000, 1023, 1024, 2046, 2047]
    for h in range(Hq):
        for qp in rows:
            wo, wl = O.window_states(q, k, v, 0, h, qp, theta=w.theta,
                                     w_pretrained=w.w_pretrained, w_local=w.w_local)
            for x in range(3):
                assert_close(o3[x, 0, qp, h], wo[x], max_abs=2e-2, mean_abs=2e-3,
                             what="O_%s h=%d q=%d" % ("ABC"[x], h, qp))
                assert abs(l3[x, 0, h, qp] - wl[x]) <= 5e-2, ("LSE", "ABC"[x], h, qp)


@pytest.mark.parametrize("L,g,w_pre,w0", [(300, 4, 70, 100), (517, 2, 100, 128)])
def test_windows_b_and_c_cancel_exactly_inside_the_band(L, g, w_pre, w0):
    """For q <= w0 the remote-only key set is empty: windows B and C cover the
    same keys with the same rotation, so the passes must agree bit for bit and
    the merged row must equal window A's."""
    B, Hkv = 1, 2
    q, k, v = synth.prefill_inputs(B, g * Hkv, Hkv, L, 128, seed=L + 11, outlier_channels=8)
    say("literal B == C for q <= w0, L=%d" % L)
    out, _, ws = _literal(q, k, v, w_pre, w0)
    o3, l3 = api.literal_window_states(ws, B, g * Hkv, L)
    n = w0 + 1
    assert torch.equal(o3[1, :, :n].view(torch.int32), o3[2, :, :n].view(torch.int32))
    assert torch.equal(l3[1, :, :, :n].view(torch.int32), l3[2, :, :, :n].view(torch.int32))
    # rows past the band do differ (the remote-only keys enter B only)
    assert not torch.equal(o3[1, :, n:], o3[2, :, n:])
    # merged = A there (up to the final bf16 rounding of W_A O_A / W_A)
    a_bf16 = o3[0, :, :n].to(torch.bfloat16).float()
    diff = (out[:, :n].float() - a_bf16).abs()
    assert bool((diff <= a_bf16.abs() * 2 ** -7 + 1e-30).all())  # at most one bf16 ulp


def test_literal_agrees_with_fused():
    B, Hq, Hkv, L, w_pre, w0 = 1, 8, 2, 700, 128, 96
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=5, outlier_channels=8)
    say("literal vs fused L=%d" % L)
    out, lse, _ = _literal(q, k, v, w_pre, w0)
    fused = torch.empty_like(out)
    flse = torch.empty_like(lse)
    api.bifocal_prefill(to_dev(q), to_dev(k), to_dev(v), w_pretrained=w_pre, w_local=w0,
                        out=fused, lse=flse)
    torch.cuda.synchronize()
    assert_close(to_f64(out), to_f64(fused), max_abs=2e-2, mean_abs=2e-3, what="literal-fused")
    assert (lse - flse).abs().max().item() <= 5e-2


def test_literal_windows_checked_rerun():
    """Each window pass runs a fast pass and reruns the blocks it lists with
    the checked kernel.  With the rescale bound lowered to 2^3 nearly every
    block of every window is listed; the merged output and the three window
    states must still match the oracle, and equal what the same call gives at
    the default bound to the tolerance."""
    B, Hq, Hkv, L, w_pre, w0 = 1, 8, 2, 517, 100, 40
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=91, outlier_channels=8)
    old = api.debug_prefill_rescale_log2(3.0)
    try:
        say("literal, windows rerun on every block, L=%d" % L)
        out, lse, ws = _literal(q, k, v, w_pre, w0)
    finally:
        api.debug_prefill_rescale_log2(old)
    want, want_lse = O.prefill(q, k, v, theta=1e6, w_pretrained=w_pre, w_local=w0)
    assert_close(to_f64(out), want, what="literal, windows rerun")
    assert_close(lse.cpu().numpy(), want_lse, max_abs=5e-2, mean_abs=5e-3, what="rerun lse")
    o3, l3 = api.literal_window_states(ws, B, Hq, L)
    o3, l3 = o3.cpu().numpy().astype(np.float64), l3.cpu().numpy().astype(np.float64)
    for h in (0, 5):
        for qp in (0, 40, 41, 200, 516):
            wo, wl = O.window_states(q, k, v, 0, h, qp, theta=1e6, w_pretrained=w_pre,
                                     w_local=w0)
            for x, name in enumerate("ABC"):
                assert_close(o3[x, 0, qp, h], wo[x], max_abs=2e-2, mean_abs=2e-3,
                             what="O_%s h=%d q=%d" % (name, h, qp))
                assert abs(l3[x, 0, h, qp] - wl[x]) <= 5e-2, ("LSE_" + name, h, qp)
    out_d, _, _ = _literal(q, k, v, w_pre, w0)
    assert_close(to_f64(out), to_f64(out_d), max_abs=2e-2, mean_abs=2e-3, what="rerun vs default")


def test_literal_within_window_is_vanilla():
    """G == 1: the literal entry runs the vanilla kernel, bit for bit."""
    B, Hq, Hkv, L = 1, 4, 2, 257
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=3)
    say("literal G == 1, L=%d" % L)
    out, _, _ = _literal(q, k, v, 512, 16)
    van = api.rope_attention(to_dev(q), to_dev(k), to_dev(v))
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), van.view(torch.int16))


def test_literal_within_window_allocates_nothing():
    """G == 1 at the 32K within-window shape: the vanilla kernel the literal
    entry runs stages its value tiles in the caller's workspace, so the call
    adds no device memory once the RoPE table covers L (a decode of the same
    length builds that table first), and it still equals the vanilla call."""
    B, Hq, Hkv, L = 1, 32, 8, 32768
    q, k, v = (to_dev(x) for x in synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=8))
    out = torch.empty_like(q)
    need = api.prefill_literal_workspace_bytes(B, Hq, Hkv, L)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    dq = q[:, L - 1].contiguous()
    lens = torch.full((B,), L, dtype=torch.int32, device="cuda")
    api.release_caches()
    api.bifocal_decode(dq, k, v, lens, w_pretrained=L, w_local=64)
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    say("literal G == 1 at L=%d, free %.1f GB" % (L, free0 / 1e9))
    api.bifocal_prefill_literal(q, k, v, w_pretrained=L, w_local=64, out=out, workspace=ws)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert free0 - free1 < (8 << 20), (free0, free1)
    van = api.rope_attention(q, k, v)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), van.view(torch.int16))


def test_literal_rejects_small_workspace():
    B, Hq, Hkv, L = 1, 4, 2, 128
    q, k, v = (to_dev(x) for x in synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=1))
    need = api.prefill_literal_workspace_bytes(B, Hq, Hkv, L)
    ws = torch.empty(need - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(api.JetLongError) as e:
        api.bifocal_prefill_literal(q, k, v, w_pretrained=32, w_local=8, workspace=ws)
    assert e.value.status == api.JL_ERR_WORKSPACE
