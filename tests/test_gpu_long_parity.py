"""Discriminating parity at the Qwen3-8B-like 128K shape (GPU).

The sampled-row tests compare the kernel with the oracle at tolerances that a
schedule or window bug confined to part of a long row could pass, because a
row of 1e5 keys averages to |O| ~ 5e-3.  These tests close that gap:

  * needles (Sec. 3.1, Eq. (3); the needle pin of the oracle): for chosen rows
    q* a remote key is planted as x_k* = c R(f(q*) - f(k*)) x_q*, which lines up
    with the query only under the aliasing map of Eq. (3), and a band key as
    x_k** = c R(q* - k**) x_q* at a distance between w0/2 and w0, which lines up
    only under the base rotation of the local window (Eq. (1)).  Each needle row
    holds one needle, whose score ~c |x_q|^2 / sqrt(d) ~ 45 lies ~30 above the
    rest, so the row's output is that key's value; a kernel with a wrong f, G,
    window or rotation misses it;
  * a margin: on the same rows the kernel's distance to the oracle must be at
    most a quarter of the distance between the oracle and the oracle of the
    neighbouring schedule G + 1 (max and mean), so the test can tell G from G+1.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import (assert_close, prefill_block_q, rows_for, sample_positions, say, to_dev,
                         to_f64)

pytestmark = [pytest.mark.gpu, pytest.mark.filterwarnings("ignore::DeprecationWarning")]

W = synth.WORKLOADS["qwen3_8b_prefill_128k"]
C = 4.0  # needle gain


def _plant(k, q, plan):
    """Plant needles into the raw key tensor (bf16 bits, modified in place):
    plan = [(b, h, q*, k*, shift)]; key k* of kv head h // g becomes
    C R(shift) x_q* (fp64 rotation, one bf16 rounding)."""
    g = W.Hq // W.Hkv
    for b, h, qs, ks, shift in plan:
        xq = synth.bf16_to_f32(q[b, qs, h]).astype(np.float64)
        k[b, ks, h // g] = synth.bf16_bits((C * O.rope_rotate(xq, shift, W.theta)).astype(np.float32))


@pytest.fixture(scope="module")
def needle_run():
    G = api.group_size(W.L, W.w_pretrained)
    assert G == 4
    say("generating", W.name)
    q, k, v = synth.make_inputs(W)
    w0 = W.w_local
    g = W.Hq // W.Hkv
    # (b, head, q*, k*, remote): remote needles in kv heads 0..3, band needles
    # (q* - k** in (w0/2, w0]) in kv heads 4..7, one needle per row
    picks = [(0, 0, W.L - 1, 1234, True), (0, 5, 100000, 77777, True),
             (0, 10, 40001, 30000, True), (0, 15, 60000, 2000, True),
             (0, 16, W.L - 1, W.L - 1 - 3000, False), (0, 21, 65536, 65536 - 4096, False),
             (0, 26, 100000, 100000 - 2049, False), (0, 31, 8191, 8191 - 4000, False)]
    plan = []
    for b, h, qs, ks, remote in picks:
        assert (qs - ks > w0) if remote else (w0 // 2 < qs - ks <= w0)
        # a remote needle sits far (>= 7500 positions) from where base
        # positions would put it, so the unmodified rotation cannot line it up
        assert not remote or (qs - ks) - (qs // G - ks // G) >= 7500
        assert (h // g < 4) == remote
        plan.append((b, h, qs, ks, qs // G - ks // G if remote else qs - ks))
    _plant(k, q, plan)
    say("needle prefill at 128K")
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    out = api.bifocal_prefill(qd, kd, vd, w_pretrained=W.w_pretrained, w_local=w0,
                              rope_theta=W.theta)
    van = api.rope_attention(qd, kd, vd, rope_theta=W.theta)
    torch.cuda.synchronize()
    o = out.float().cpu().numpy()
    ov = van.float().cpu().numpy()
    del qd, kd, vd, out, van
    return q, k, v, o, ov, picks, G


def test_needles_route_through_both_views_at_128k(needle_run):
    q, k, v, o, ov, picks, G = needle_run
    g = W.Hq // W.Hkv
    vf = synth.bf16_to_f32(v).astype(np.float64)
    rows = np.array([[b, h, qs] for b, h, qs, _, _ in picks], dtype=np.int64)
    want, _ = O.prefill_rows(q, k, v, rows, theta=W.theta, w_pretrained=W.w_pretrained,
                             w_local=W.w_local)
    got = o[rows[:, 0], rows[:, 2], rows[:, 1]].astype(np.float64)
    assert_close(got, want, what="needle rows")
    for i, (b, h, qs, ks, remote) in enumerate(picks):
        target = vf[b, ks, h // g]
        e_or = np.abs(want[i] - target).max()
        e_gpu = np.abs(got[i] - target).max()
        e_van = np.abs(ov[b, qs, h].astype(np.float64) - target).max()
        say("%s needle q*=%d k*=%d head %d: oracle %.2e, gpu %.2e, vanilla %.2e from V[k*]" %
            ("remote" if remote else "band", qs, ks, h, e_or, e_gpu, e_van))
        assert e_or < 1e-2 and e_gpu < 2e-2
        if remote:  # the unmodified model does not see the remote needle
            assert e_van > 0.2, e_van
        else:       # ... and sees the band needle as the method does
            assert e_van < 2e-2, e_van


def test_margin_against_neighbouring_schedule(needle_run):
    q, k, v, o, ov, picks, G = needle_run
    block_q = prefill_block_q(W.Hq, W.Hkv)
    pos = sample_positions(W.L, W.w_local, W.w_pretrained, G, block_q, 8, seed=3)
    pos = sorted(set(pos) | {qs for _, _, qs, _, _ in picks})
    rows = rows_for(W.B, W.Hq, pos)[:: 3]  # every third (b, head, q) keeps the oracle brief
    say("oracle rows", len(rows), "at G, G+1 and w0/2")
    want, _ = O.prefill_rows(q, k, v, rows, theta=W.theta, w_pretrained=W.w_pretrained,
                             w_local=W.w_local)
    w_next = -(-W.L // (G + 1))
    assert O.group_size(W.L, w_next) == G + 1
    alt_g, _ = O.prefill_rows(q, k, v, rows, theta=W.theta, w_pretrained=w_next,
                              w_local=W.w_local)
    alt_w, _ = O.prefill_rows(q, k, v, rows, theta=W.theta, w_pretrained=W.w_pretrained,
                              w_local=W.w_local // 2)
    got = o[rows[:, 0], rows[:, 2], rows[:, 1]].astype(np.float64)
    err = np.abs(got - want)
    dg = np.abs(alt_g - want)
    dw = np.abs(alt_w - want)
    say("128K margin: gpu err max %.3e mean %.3e | G+1 moves max %.3e mean %.3e | "
        "w0/2 moves max %.3e mean %.3e" % (err.max(), err.mean(), dg.max(), dg.mean(),
                                            dw.max(), dw.mean()))
    assert_close(got, want, what="128K margin rows")
    assert err.max() <= 0.25 * dg.max() and err.mean() <= 0.25 * dg.mean()
    assert err.max() <= 0.25 * dw.max() and err.mean() <= 0.25 * dw.mean()
    # the same without the needle rows, whose planted keys move by O(1)
    plain = ~np.isin(rows[:, 2], [qs for _, _, qs, _, _ in picks])
    e, a1, a2 = err[plain], dg[plain], dw[plain]
    say("128K margin without needle rows: gpu max %.3e mean %.3e | G+1 max %.3e mean %.3e | "
        "w0/2 max %.3e mean %.3e" % (e.max(), e.mean(), a1.max(), a1.mean(), a2.max(), a2.mean()))
    assert e.mean() <= 0.25 * a1.mean() and e.mean() <= 0.25 * a2.mean()
    assert e.max() <= 0.25 * a1.max()
