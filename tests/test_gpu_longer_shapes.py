"""Lengths past the benchmark's 128K: 256K and 1M prefills (G = 8, 32) and a
512K decode (G = 16) with few heads, against the fp64 oracle on sampled rows,
each with a planted remote needle that lines up only under the aliasing map of
Eq. (3); and the decode at its largest accepted length, 2^23."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import (assert_close, prefill_block_q, rows_for, sample_positions, say, to_dev,
                         to_f64)

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

THETA = 1e6


def _needle(q, k, b, h, g, qs, ks, G, gain=4.0):
    """Key ks of kv head h // g becomes gain R(f(qs) - f(ks)) x_q[qs] (bf16)."""
    xq = synth.bf16_to_f32(q[b, qs, h]).astype(np.float64)
    shift = qs // G - ks // G
    k[b, ks, h // g] = synth.bf16_bits((gain * O.rope_rotate(xq, shift, THETA)).astype(np.float32))


@pytest.mark.parametrize("L,G_want", [(262144, 8), (1048576, 32)])
def test_prefill_long_sampled_rows_and_needle(L, G_want):
    B, Hq, Hkv, w_pre, w0 = 1, 4, 1, 32768, 4096
    G = api.group_size(L, w_pre)
    assert G == G_want
    say("generating %dK prefill inputs" % (L // 1024))
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=L // 1024)
    qs, ks = L - 1, 12345  # a remote needle for head 2
    _needle(q, k, 0, 2, Hq // Hkv, qs, ks, G)
    say("prefill L=%d G=%d" % (L, G))
    out = api.bifocal_prefill(to_dev(q), to_dev(k), to_dev(v), w_pretrained=w_pre, w_local=w0)
    torch.cuda.synchronize()
    o = to_f64(out)
    assert np.isfinite(o).all()
    pos = sample_positions(L, w0, w_pre, G, prefill_block_q(Hq, Hkv), 24, seed=3)
    rows = rows_for(B, Hq, pos)
    say("oracle on %d rows" % len(rows))
    want, _ = O.prefill_rows(q, k, v, rows, theta=THETA, w_pretrained=w_pre, w_local=w0)
    assert_close(o[rows[:, 0], rows[:, 2], rows[:, 1]], want, what="prefill %dK G=%d" % (L // 1024, G))
    # the needle row is the needle's value row: the oracle's exactly, the kernel's too
    vk = synth.bf16_to_f32(v[0, ks, 0]).astype(np.float64)
    got = o[0, qs, 2]
    ref, _ = O.prefill_rows(q, k, v, np.array([[0, 2, qs]], dtype=np.int64), theta=THETA,
                            w_pretrained=w_pre, w_local=w0)
    say("needle: oracle %.2e, gpu %.2e from V[k*]" % (np.abs(ref[0] - vk).max(),
                                                      np.abs(got - vk).max()))
    assert np.abs(ref[0] - vk).max() < 1e-6
    assert np.abs(got - vk).max() < 2e-2


def test_decode_512k_g16():
    B, Hq, Hkv, max_len, w_pre, w0 = 2, 8, 1, 524288, 32768, 4096
    lens = [max_len, 300001]
    assert api.group_size(max_len, w_pre) == 16
    say("generating 512K decode inputs")
    q, kc, vc, ln = synth.decode_inputs(B, Hq, Hkv, max_len, lens, seed=512, nan_tail=True)
    # a remote needle for head 3 of sequence 0 (its query sits at max_len - 1)
    xq = synth.bf16_to_f32(q[0, 3]).astype(np.float64)
    shift = (max_len - 1) // 16 - 4567 // 16
    kc[0, 4567, 0] = synth.bf16_bits((4.0 * O.rope_rotate(xq, shift, THETA)).astype(np.float32))
    say("decode B=%d max_len=%d" % (B, max_len))
    out = api.bifocal_decode(to_dev(q), to_dev(kc), to_dev(vc), torch.from_numpy(ln).cuda(),
                             w_pretrained=w_pre, w_local=w0)
    torch.cuda.synchronize()
    want, _, _ = O.decode(q, kc, vc, ln, theta=THETA, w_pretrained=w_pre, w_local=w0)
    assert_close(to_f64(out), want, what="decode 512K G=16")
    vk = synth.bf16_to_f32(vc[0, 4567, 0]).astype(np.float64)
    assert np.abs(want[0, 3] - vk).max() < 1e-6
    assert np.abs(to_f64(out)[0, 3] - vk).max() < 2e-2


def test_decode_at_the_maximum_length():
    """max_len = 2^23, the largest length the decode accepts (G = 256): the
    query's cos/sin rows reach the last table row and byte offset 2^32 - 512.
    The fp64 oracle would rotate 2^23 keys per view, so the check is by
    construction instead: every key is zero but two planted ones, a remote
    key that lines up with head 0's query only under Eq. (3) with G = 256
    and a band key that lines up with head 1's under the base rotation.
    Each needle scores about 34 against 0 for the 2^23 others, so each head's
    output is its needle's value row to within 1e-8 before bf16 rounding; the
    vanilla decode, which rotates the remote key to its own position, is not."""
    B, Hq, Hkv, max_len, w_pre, w0 = 1, 2, 1, 1 << 23, 32768, 4096
    G = api.group_size(max_len, w_pre)
    assert G == 256
    qpos = max_len - 1
    rng = np.random.default_rng(23)
    q = synth.bf16_bits(rng.standard_normal((B, Hq, 128), dtype=np.float32))
    say("building 2^23-key caches")
    kc = np.zeros((B, max_len, Hkv, 128), dtype=np.uint16)
    pool = synth.bf16_bits(rng.standard_normal((1 << 16, 128), dtype=np.float32))
    vc = np.tile(pool, (max_len >> 16, 1)).reshape(B, max_len, Hkv, 128)
    ks_r, ks_l, gain = 1234567, qpos - 1000, 3.0
    xq = synth.bf16_to_f32(q[0]).astype(np.float64)
    kc[0, ks_r, 0] = synth.bf16_bits(
        (gain * O.rope_rotate(xq[0], qpos // G - ks_r // G, THETA)).astype(np.float32))
    kc[0, ks_l, 0] = synth.bf16_bits((gain * O.rope_rotate(xq[1], qpos - ks_l, THETA)).astype(np.float32))
    vc[0, ks_r, 0] = synth.bf16_bits(rng.standard_normal(128, dtype=np.float32))
    vc[0, ks_l, 0] = synth.bf16_bits(rng.standard_normal(128, dtype=np.float32))
    qd, kd, vd = to_dev(q), to_dev(kc), to_dev(vc)
    ld = torch.full((B,), max_len, dtype=torch.int32, device="cuda")
    say("decode max_len=%d G=%d" % (max_len, G))
    out = to_f64(api.bifocal_decode(qd, kd, vd, ld, w_pretrained=w_pre, w_local=w0))
    van = to_f64(api.rope_attention_decode(qd, kd, vd, ld))
    torch.cuda.synchronize()
    want = synth.bf16_to_f32(vc[0, [ks_r, ks_l], 0]).astype(np.float64)
    err = np.abs(out[0] - want)
    say("needle rows: max err %.2e, mean %.2e; vanilla head 0 off by %.2f" %
        (err.max(), err.mean(), np.abs(van[0, 0] - want[0]).max()))
    assert np.isfinite(out).all()
    assert err.max() < 2e-2 and err.mean() < 1e-3
    assert np.abs(van[0, 0] - want[0]).max() > 0.5
