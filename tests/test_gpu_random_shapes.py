"""Seeded random small configurations against the fp64 oracle: full-tensor
prefill (with LSE) and a ragged decode batch per configuration, under the
Eq. (3) map and the Sec. 4.5 frequency map, so corner
combinations of length, GQA group, pretraining window and local window that
the hand-picked cases miss are covered too.  The draw is fixed (seed 2607),
so every run checks the same configurations."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api, synth
from parity_util import assert_close, say, to_dev, to_f64

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _configs(n=16, seed=2607):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        L = int(rng.integers(1, 700))
        g = int(rng.choice([1, 2, 4, 8]))
        Hkv = int(rng.choice([1, 2, 3]))
        # mostly G >= 2 and a band shorter than the sequence; a quarter with
        # G = 1 and an eighth with a band over every key
        w_pre = int(rng.integers(L, 2 * L + 1)) if rng.random() < 0.25 else \
            int(rng.integers(1, max(2, L // 2 + 1)))
        w0 = int(rng.integers(L - 1, 2 * L)) if rng.random() < 0.125 else \
            int(rng.integers(0, max(1, L // 2)))
        B = int(rng.integers(1, 3))
        out.append((i, B, Hkv, g, L, w_pre, w0))
    return out


@pytest.mark.parametrize("remote_map", ["alias", "freq"])
@pytest.mark.parametrize("i,B,Hkv,g,L,w_pre,w0", _configs())
def test_random_prefill_and_decode(i, B, Hkv, g, L, w_pre, w0, remote_map):
    Hq = g * Hkv
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=1000 + i, outlier_channels=8)
    say("random config %d (%s): B=%d Hkv=%d g=%d L=%d w_pre=%d w0=%d G=%d"
        % (i, remote_map, B, Hkv, g, L, w_pre, w0, api.group_size(L, w_pre)))
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    out = torch.full_like(qd, float("nan"))
    lse = torch.full((B, Hq, L), float("nan"), device="cuda")
    api.bifocal_prefill(qd, kd, vd, w_pretrained=w_pre, w_local=w0, out=out, lse=lse,
                        remote_map=remote_map)
    torch.cuda.synchronize()
    want, want_lse = O.prefill(q, k, v, theta=1e6, w_pretrained=w_pre, w_local=w0,
                               remote_map=remote_map)
    assert_close(to_f64(out), want, what="prefill config %d" % i)
    assert_close(lse.cpu().numpy(), want_lse, max_abs=5e-2, mean_abs=5e-3, what="lse")

    # decode over the same keys: sequence b's query is its last prefill row's
    # query, at a seeded length of its own (G follows that length)
    rng = np.random.default_rng(2000 + i)
    lens = np.array([int(rng.integers(1, L + 1)) for _ in range(B)], dtype=np.int32)
    dq = np.stack([q[b, lens[b] - 1] for b in range(B)])
    dout = api.bifocal_decode(to_dev(dq), kd, vd, torch.from_numpy(lens).cuda(),
                              w_pretrained=w_pre, w_local=w0, remote_map=remote_map)
    torch.cuda.synchronize()
    dwant, _, _ = O.decode(dq, k, v, lens, theta=1e6, w_pretrained=w_pre, w_local=w0,
                           remote_map=remote_map)
    assert_close(to_f64(dout), dwant, what="decode config %d lens %s" % (i, [int(x) for x in lens]))


@pytest.mark.parametrize("i,B,Hkv,g,L,w_pre,w0", _configs())
def test_random_chunk_paged_and_packed_entries_agree(i, B, Hkv, g, L, w_pre, w0):
    """On the same configurations, each serving entry point against the full
    prefill of the same keys, bit for bit: a chunk of rows P .. L-1 over a
    NaN-padded cache (G from its length L), the same chunk over shuffled
    pages, and the batch packed into one varlen call (each sequence its own L)."""
    Hq = g * Hkv
    rng = np.random.default_rng(3000 + i)
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=1000 + i, outlier_channels=8)
    qd, kd, vd = to_dev(q), to_dev(k), to_dev(v)
    full = api.bifocal_prefill(qd, kd, vd, w_pretrained=w_pre, w_local=w0)

    P = int(rng.integers(0, L))
    pad = int(rng.integers(0, 100))
    nan = np.uint16(0x7FC0)
    kc = np.full((B, L + pad, Hkv, 128), nan, dtype=np.uint16)
    vc = np.full_like(kc, nan)
    kc[:, :L], vc[:, :L] = k, v
    say("random config %d: chunk P=%d of L=%d, pad %d" % (i, P, L, pad))
    chunk = api.prefill_chunk(to_dev(q[:, P:]), to_dev(kc), to_dev(vc), q_start=P,
                              w_pretrained=w_pre, w_local=w0)
    torch.cuda.synchronize()
    assert torch.equal(chunk.view(torch.int16), full[:, P:].view(torch.int16))

    page = int(rng.choice([64, 128, 256]))
    per_seq = (L + page - 1) // page
    n_pages = B * per_seq + 2
    order = rng.permutation(n_pages)
    kp = np.full((n_pages, page, Hkv, 128), nan, dtype=np.uint16)
    vp = np.full_like(kp, nan)
    table = np.zeros((B, per_seq), dtype=np.int32)
    for b in range(B):
        for j in range(per_seq):
            pg = int(order[b * per_seq + j])
            table[b, j] = pg
            lo, hi = j * page, min((j + 1) * page, L)
            kp[pg, :hi - lo], vp[pg, :hi - lo] = k[b, lo:hi], v[b, lo:hi]
    say("random config %d: paged chunk, page %d" % (i, page))
    paged = api.prefill_chunk_paged(to_dev(q[:, P:]), to_dev(kp), to_dev(vp),
                                    torch.from_numpy(table).cuda(), q_start=P,
                                    w_pretrained=w_pre, w_local=w0)
    torch.cuda.synchronize()
    assert torch.equal(paged.view(torch.int16), chunk.view(torch.int16))

    # the batch packed with a second, shorter copy of each sequence
    cut = [L] + [int(rng.integers(1, L + 1)) for _ in range(B)]
    seqs = [(0, cut[0])] + [(b, cut[1 + b]) for b in range(B)]
    cu = np.cumsum([0] + [n for _, n in seqs]).astype(np.int32)
    qp = np.concatenate([q[b, :n] for b, n in seqs])
    kpk = np.concatenate([k[b, :n] for b, n in seqs])
    vpk = np.concatenate([v[b, :n] for b, n in seqs])
    say("random config %d: packed lengths %s" % (i, [n for _, n in seqs]))
    packed = api.prefill_varlen(to_dev(qp), to_dev(kpk), to_dev(vpk), torch.from_numpy(cu).cuda(),
                                max_seqlen=L, w_pretrained=w_pre, w_local=w0)
    torch.cuda.synchronize()
    for s_, (b, n) in enumerate(seqs):
        alone = api.bifocal_prefill(to_dev(q[b:b + 1, :n]), to_dev(k[b:b + 1, :n]),
                                    to_dev(v[b:b + 1, :n]), w_pretrained=w_pre, w_local=w0)
        torch.cuda.synchronize()
        assert torch.equal(packed[cu[s_]:cu[s_ + 1]].view(torch.int16), alone[0].view(torch.int16))


@pytest.mark.parametrize("i,B,Hkv,g,L,w_pre,w0", _configs())
def test_random_paged_and_noalloc_decode_agree(i, B, Hkv, g, L, w_pre, w0):
    """On the same configurations, the paged decode (shuffled pages, both remote
    maps) and the no-alloc decode against the dense decode over the same keys, bit for bit,
    with ragged lengths; the dense cache is padded to the pool's capacity so
    all three take the same split plan."""
    Hq = g * Hkv
    rng = np.random.default_rng(4000 + i)
    page = int(rng.choice([16, 32, 64]))
    per_seq = (L + page - 1) // page
    max_len = per_seq * page
    lens = [int(rng.integers(1, L + 1)) for _ in range(B)]
    q, kc, vc, lens = synth.decode_inputs(B, Hq, Hkv, max_len, lens, seed=5000 + i, nan_tail=True)
    ld = torch.from_numpy(lens).cuda()
    say("random config %d: decode lens %s, page %d" % (i, [int(x) for x in lens], page))
    dense = api.bifocal_decode(to_dev(q), to_dev(kc), to_dev(vc), ld, w_pretrained=w_pre,
                               w_local=w0)
    noalloc = api.bifocal_decode_noalloc(to_dev(q), to_dev(kc), to_dev(vc), ld,
                                         w_pretrained=w_pre, w_local=w0)
    n_pages = B * per_seq + 3
    order = rng.permutation(n_pages)
    nan = np.uint16(0x7FC0)
    kp = np.full((n_pages, page, Hkv, 128), nan, dtype=np.uint16)
    vp = np.full_like(kp, nan)
    table = np.zeros((B, per_seq), dtype=np.int32)
    for b in range(B):
        for j in range(per_seq):
            pg = int(order[b * per_seq + j])
            table[b, j] = pg
            kp[pg], vp[pg] = kc[b, j * page:(j + 1) * page], vc[b, j * page:(j + 1) * page]
    paged = api.decode_paged(to_dev(q), to_dev(kp), to_dev(vp), torch.from_numpy(table).cuda(),
                             ld, w_pretrained=w_pre, w_local=w0)
    # the same pages under the frequency map
    dense_f = api.bifocal_decode(to_dev(q), to_dev(kc), to_dev(vc), ld, w_pretrained=w_pre,
                                 w_local=w0, remote_map="freq")
    paged_f = api.decode_paged(to_dev(q), to_dev(kp), to_dev(vp), torch.from_numpy(table).cuda(),
                               ld, w_pretrained=w_pre, w_local=w0, remote_map="freq")
    torch.cuda.synchronize()
    assert torch.equal(noalloc.view(torch.int16), dense.view(torch.int16))
    assert torch.equal(paged.view(torch.int16), dense.view(torch.int16))
    assert torch.equal(paged_f.view(torch.int16), dense_f.view(torch.int16))


@pytest.mark.parametrize("i,B,Hkv,g,L,w_pre,w0", _configs())
def test_random_literal_mode(i, B, Hkv, g, L, w_pre, w0):
    """The literal Eq. (7) prefill (three window passes and the merge) on the
    same configurations, against the oracle's output and LSE."""
    Hq = g * Hkv
    q, k, v = synth.prefill_inputs(B, Hq, Hkv, L, 128, seed=1000 + i, outlier_channels=8)
    say("random config %d: literal mode, G=%d" % (i, api.group_size(L, w_pre)))
    out, lse = api.bifocal_prefill_literal(to_dev(q), to_dev(k), to_dev(v), w_pretrained=w_pre,
                                           w_local=w0, want_lse=True)
    torch.cuda.synchronize()
    want, want_lse = O.prefill(q, k, v, theta=1e6, w_pretrained=w_pre, w_local=w0)
    assert_close(to_f64(out), want, what="literal config %d" % i)
    assert_close(lse.cpu().numpy(), want_lse, max_abs=5e-2, mean_abs=5e-3, what="literal lse")
