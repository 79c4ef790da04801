"""The C ABI without a GPU: symbols, status strings, host schedule, argument checks.

Every invalid call below must be rejected on the host before anything touches
the HIP runtime, so these run on a machine without a GPU.  Fake device
addresses are never dereferenced because validation fails first.
"""
import ctypes

import pytest

from oracle import oracle as O
from paper_2607_07740_amd import api

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")

P = ctypes.c_void_p
A = P(0x1000)  # aligned fake device address
A2 = P(0x2000)
MIS = P(0x1002)  # misaligned


def test_library_exports_every_declared_symbol():
    L = api.lib()
    names = api.declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(L, n), n


def test_status_strings_and_version():
    L = api.lib()
    for code, name in [(0, "JL_OK"), (1, "JL_ERR_INVALID_ARG"), (2, "JL_ERR_UNSUPPORTED"),
                       (3, "JL_ERR_WORKSPACE"), (4, "JL_ERR_HIP")]:
        assert L.jl_status_string(code).decode() == name
    assert L.jl_status_string(99).decode() == "JL_ERR_UNKNOWN"
    assert L.jl_version() >= 100


def test_host_group_size_matches_oracle():
    for w in (1, 2, 3, 7, 512, 32768):
        for Lx in list(range(1, 3 * w + 2, max(1, w // 7))) + [131072, 2 ** 31 - 1]:
            assert api.group_size(Lx, w) == O.group_size(Lx, w), (Lx, w)
    assert api.group_size(0, 5) == -1 and api.group_size(5, 0) == -1


def _prefill(q=A, k=A, v=A, o=A, lse=None, B=1, Hq=4, Hkv=2, L=64, d=128, theta=1e6, w=16,
             w0=4):
    return api.lib().jl_bifocal_prefill(q, k, v, o, lse, B, Hq, Hkv, L, d, theta, w, w0, None)


@pytest.mark.parametrize("kw,code", [
    (dict(Hq=3, Hkv=2), api.JL_ERR_INVALID_ARG),
    (dict(B=0), api.JL_ERR_INVALID_ARG),
    (dict(Hkv=0), api.JL_ERR_INVALID_ARG),
    (dict(L=0), api.JL_ERR_INVALID_ARG),
    (dict(d=64), api.JL_ERR_UNSUPPORTED),
    (dict(d=127), api.JL_ERR_INVALID_ARG),
    (dict(theta=0.0), api.JL_ERR_INVALID_ARG),
    (dict(theta=float("nan")), api.JL_ERR_INVALID_ARG),
    (dict(w=0), api.JL_ERR_INVALID_ARG),
    (dict(w0=-1), api.JL_ERR_INVALID_ARG),
    (dict(q=None), api.JL_ERR_INVALID_ARG),
    (dict(k=MIS), api.JL_ERR_INVALID_ARG),
    (dict(o=None), api.JL_ERR_INVALID_ARG),
    (dict(lse=P(0x1001)), api.JL_ERR_INVALID_ARG),
    (dict(Hq=6, Hkv=2), api.JL_ERR_UNSUPPORTED),  # GQA group 3 does not divide 256
])
def test_prefill_rejects_before_launch(kw, code):
    assert _prefill(**kw) == code
    assert api.lib().jl_last_error().decode() != ""


@pytest.mark.parametrize("remote_map", [-1, 2, 7])
def test_prefill_map_rejects_unknown_remote_map(remote_map):
    L = api.lib()
    assert L.jl_bifocal_prefill_map(A, A, A, A, None, 1, 4, 2, 64, 128, 1e6, 16, 4, remote_map,
                                    None) == api.JL_ERR_INVALID_ARG
    assert "remote_map" in L.jl_last_error().decode()
    # the usual checks still apply to a valid map
    assert L.jl_bifocal_prefill_map(A, A, A, A, None, 1, 4, 2, 0, 128, 1e6, 16, 4, 1,
                                    None) == api.JL_ERR_INVALID_ARG


@pytest.mark.parametrize("q_start,n,max_len", [(-1, 16, 64), (0, 0, 64), (60, 16, 64),
                                                (0, 65, 64)])
def test_prefill_chunk_rejects_bad_ranges(q_start, n, max_len):
    L = api.lib()
    for rc in (L.jl_bifocal_prefill_chunk(A, A, A, A, None, 1, 4, 2, q_start, n, max_len, 128,
                                          1e6, 16, 4, None),
               L.jl_rope_attention_chunk(A, A, A, A, None, 1, 4, 2, q_start, n, max_len, 128, 1e6,
                                         None)):
        assert rc == api.JL_ERR_INVALID_ARG
        assert L.jl_last_error().decode() != ""


def _chunk_paged(bifocal=True, **kw):
    a = dict(table=A2, max_pages=8, page_size=64, n_pages=20, B=1, Hq=8, Hkv=2, q_start=100,
             n=60, d=128)
    a.update(kw)
    args = [A, A, A, a["table"], a["max_pages"], a["page_size"], a["n_pages"], A, None, a["B"],
            a["Hq"], a["Hkv"], a["q_start"], a["n"], a["d"], 1e6]
    L = api.lib()
    if bifocal:
        return L.jl_bifocal_prefill_chunk_paged(*args, 64, 8, None)
    return L.jl_rope_attention_chunk_paged(*args, None)


@pytest.mark.parametrize("kw,code", [
    (dict(table=None), api.JL_ERR_INVALID_ARG),
    (dict(table=MIS), api.JL_ERR_INVALID_ARG),
    (dict(page_size=0), api.JL_ERR_INVALID_ARG),
    (dict(page_size=96), api.JL_ERR_INVALID_ARG),
    (dict(page_size=1 << 21), api.JL_ERR_INVALID_ARG),
    (dict(page_size=32), api.JL_ERR_UNSUPPORTED),  # a page must hold whole 64-key tiles
    (dict(max_pages=0), api.JL_ERR_INVALID_ARG),
    (dict(n_pages=0), api.JL_ERR_INVALID_ARG),
    (dict(q_start=-1), api.JL_ERR_INVALID_ARG),
    (dict(n=0), api.JL_ERR_INVALID_ARG),
    (dict(q_start=500, n=13), api.JL_ERR_INVALID_ARG),  # 513 keys > 8 pages of 64
    (dict(B=0), api.JL_ERR_INVALID_ARG),
    (dict(d=64), api.JL_ERR_UNSUPPORTED),
])
def test_prefill_chunk_paged_rejects_before_launch(kw, code):
    for bif in (True, False):
        assert _chunk_paged(bif, **kw) == code, kw
        assert api.lib().jl_last_error().decode() != ""


def test_prefill_chunk_paged_page_count_limit_is_exact():
    # one sequence's page list must fit the attention kernel's 4096-entry LDS
    # table; B = 0 makes a call that passes the page checks fail just after
    big = dict(max_pages=5000, page_size=64, q_start=0, B=0)
    assert _chunk_paged(n=4096 * 64, **big) == api.JL_ERR_INVALID_ARG
    assert _chunk_paged(n=4096 * 64 + 1, **big) == api.JL_ERR_UNSUPPORTED
    assert "4096" in api.lib().jl_last_error().decode()


@pytest.mark.parametrize("kw,code", [
    (dict(T=0), api.JL_ERR_INVALID_ARG),
    (dict(max_seqlen=0), api.JL_ERR_INVALID_ARG),
    (dict(cu=None), api.JL_ERR_INVALID_ARG),
    (dict(cu=P(0x1002)), api.JL_ERR_INVALID_ARG),
    (dict(B=0), api.JL_ERR_INVALID_ARG),
    (dict(Hq=12, Hkv=1), api.JL_ERR_UNSUPPORTED),
    (dict(q=MIS), api.JL_ERR_INVALID_ARG),
    (dict(lse=P(0x1001)), api.JL_ERR_INVALID_ARG),
    (dict(w=0), api.JL_ERR_INVALID_ARG),
    (dict(w0=-1), api.JL_ERR_INVALID_ARG),
    (dict(T=2 ** 31 - 1, Hkv=1024, Hq=1024), api.JL_ERR_INVALID_ARG),
])
def test_prefill_varlen_rejects_before_launch(kw, code):
    a = dict(q=A, lse=None, cu=A2, B=3, T=300, max_seqlen=200, Hq=8, Hkv=2, w=64, w0=8)
    a.update(kw)
    L = api.lib()
    rc = L.jl_bifocal_prefill_varlen(a["q"], A, A, A, a["lse"], a["cu"], a["B"], a["T"],
                                     a["max_seqlen"], a["Hq"], a["Hkv"], 128, 1e6, a["w"],
                                     a["w0"], None)
    assert rc == code, L.jl_last_error()
    assert L.jl_last_error().decode() != ""
    if "w" not in kw and "w0" not in kw:
        rc = L.jl_rope_attention_varlen(a["q"], A, A, A, a["lse"], a["cu"], a["B"], a["T"],
                                        a["max_seqlen"], a["Hq"], a["Hkv"], 128, 1e6, None)
        assert rc == code


@pytest.mark.parametrize("kw", [dict(page_size=8), dict(page_size=48), dict(page_size=0),
                                dict(max_pages=0), dict(n_pages=0), dict(table=None),
                                dict(table=P(0x1002))])
def test_decode_paged_rejects_bad_pages(kw):
    a = dict(table=A2, max_pages=4, page_size=64, n_pages=10)
    a.update(kw)
    L = api.lib()
    rc = L.jl_bifocal_decode_paged(A, A, A, a["table"], a["max_pages"], a["page_size"],
                                   a["n_pages"], A2, A, 1, 8, 2, 128, 1e6, 64, 8, A, 1 << 20, None)
    assert rc == api.JL_ERR_INVALID_ARG
    rc = L.jl_rope_attention_decode_paged(A, A, A, a["table"], a["max_pages"], a["page_size"],
                                          a["n_pages"], A2, A, 1, 8, 2, 128, 1e6, A, 1 << 20,
                                          None)
    assert rc == api.JL_ERR_INVALID_ARG


def test_decode_map_rejects_bad_map_and_small_workspace():
    L = api.lib()
    for rm in (-1, 2):
        assert L.jl_bifocal_decode_map(A, A, A, A2, 1024, A, 1, 8, 2, 128, 1e6, 64, 8, rm, A,
                                       1 << 30, None) == api.JL_ERR_INVALID_ARG
        assert L.jl_decode_map_workspace_bytes(1, 8, 2, 1024, 128, rm) == 0
    alias = L.jl_decode_map_workspace_bytes(1, 8, 2, 1024, 128, 0)
    freq = L.jl_decode_map_workspace_bytes(1, 8, 2, 1024, 128, 1)
    assert alias == api.decode_workspace_bytes(1, 8, 2, 1024)
    assert freq == alias
    rc = L.jl_bifocal_decode_map(A, A, A, A2, 1024, A, 1, 8, 2, 128, 1e6, 64, 8, 1, A, freq - 1,
                                 None)
    assert rc == api.JL_ERR_WORKSPACE


def test_rope_attention_rejects_before_launch():
    L = api.lib()
    assert L.jl_rope_attention(A, A, A, A, None, 1, 4, 2, 0, 128, 1e6, None) == api.JL_ERR_INVALID_ARG
    assert L.jl_rope_attention(A, A, A, A, None, 1, 4, 2, 8, 96, 1e6, None) == api.JL_ERR_UNSUPPORTED


def _decode(q=A, kc=A, vc=A, lens=A2, max_len=1024, o=A, B=2, Hq=8, Hkv=2, d=128, theta=1e6,
            w=256, w0=16, ws=A, ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = api.decode_workspace_bytes(B, Hq, Hkv, max_len) if Hkv and Hq % max(Hkv, 1) == 0 else 0
    return api.lib().jl_bifocal_decode(q, kc, vc, lens, max_len, o, B, Hq, Hkv, d, theta, w, w0,
                                       ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(max_len=0), api.JL_ERR_INVALID_ARG),
    (dict(Hq=7, Hkv=2), api.JL_ERR_INVALID_ARG),
    (dict(d=256), api.JL_ERR_UNSUPPORTED),
    (dict(Hq=32, Hkv=2), api.JL_ERR_UNSUPPORTED),  # group 16 > 8
    (dict(w=0), api.JL_ERR_INVALID_ARG),
    (dict(w0=-5), api.JL_ERR_INVALID_ARG),
    (dict(lens=None), api.JL_ERR_INVALID_ARG),
    (dict(q=MIS), api.JL_ERR_INVALID_ARG),
    (dict(ws=None), api.JL_ERR_WORKSPACE),
    (dict(ws_bytes=16), api.JL_ERR_WORKSPACE),
    (dict(max_len=(1 << 23) + 16), api.JL_ERR_UNSUPPORTED),  # table rows past 32-bit offsets
])
def test_decode_rejects_before_launch(kw, code):
    assert _decode(**kw) == code


def test_decode_length_limit_is_exact():
    # 2^23 positions is the last length the split kernel's 32-bit table
    # offsets cover; the check rejects one step past it on the host, for the
    # dense, paged and frequency-map forms alike
    L = api.lib()
    assert _decode(max_len=(1 << 23) + 1) == api.JL_ERR_UNSUPPORTED
    assert "8388608" in L.jl_last_error().decode()
    ws = 1 << 40  # any size: the length check comes first
    rc = L.jl_bifocal_decode_paged(A, A, A, A2, (1 << 23) // 64 + 1, 64, 10, A2, A, 1, 8, 2, 128,
                                   1e6, 64, 8, A, ws, None)
    assert rc == api.JL_ERR_UNSUPPORTED
    rc = L.jl_bifocal_decode_map(A, A, A, A2, (1 << 23) + 1, A, 1, 8, 2, 128, 1e6, 64, 8, 1, A,
                                 ws, None)
    assert rc == api.JL_ERR_UNSUPPORTED


@pytest.mark.parametrize("remote_map", [-1, 2])
def test_varlen_map_rejects_unknown_remote_map(remote_map):
    L = api.lib()
    rc = L.jl_bifocal_prefill_varlen_map(A, A, A, A, None, A2, 3, 300, 200, 8, 2, 128, 1e6, 64, 8,
                                         remote_map, None)
    assert rc == api.JL_ERR_INVALID_ARG
    assert "remote_map" in L.jl_last_error().decode()


@pytest.mark.parametrize("remote_map", [-1, 2])
def test_paged_decode_map_rejects_unknown_remote_map(remote_map):
    L = api.lib()
    rc = L.jl_bifocal_decode_paged_map(A, A, A, A2, 4, 64, 10, A2, A, 1, 8, 2, 128, 1e6, 64, 8,
                                       remote_map, A, 1 << 30, None)
    assert rc == api.JL_ERR_INVALID_ARG
    assert "remote_map" in L.jl_last_error().decode()
    assert L.jl_bifocal_decode_paged_map(A, A, A, None, 4, 64, 10, A2, A, 1, 8, 2, 128, 1e6, 64,
                                         8, 1, A, 1 << 30, None) == api.JL_ERR_INVALID_ARG


def test_noalloc_decode_bounds_are_checked_on_the_host():
    # the fixed array holds the table of 131072 positions and 24 MiB of split
    # states; larger calls are refused before any device work
    L = api.lib()
    args = lambda B, Hq, Hkv, n: (A, A, A, A2, n, A, B, Hq, Hkv, 128, 1e6, 64, 8, None)
    assert L.jl_bifocal_decode_noalloc(*args(1, 8, 2, 131073)) == api.JL_ERR_UNSUPPORTED
    assert "131072" in L.jl_last_error().decode()
    big = api.decode_workspace_bytes(64, 64, 8, 131072)
    assert big > 24 << 20
    assert L.jl_bifocal_decode_noalloc(*args(64, 64, 8, 131072)) == api.JL_ERR_UNSUPPORTED
    assert "states" in L.jl_last_error().decode()
    # the usual checks come first
    assert L.jl_bifocal_decode_noalloc(*args(0, 8, 2, 1024)) == api.JL_ERR_INVALID_ARG
    assert L.jl_bifocal_decode_noalloc(A, A, A, None, 1024, A, 1, 8, 2, 128, 1e6, 64, 8,
                                       None) == api.JL_ERR_INVALID_ARG


def test_workspace_size_is_positive_and_monotone():
    a = api.decode_workspace_bytes(1, 32, 8, 131072)
    b = api.decode_workspace_bytes(8, 32, 8, 131072)
    assert 0 < a <= b
    assert api.decode_workspace_bytes(1, 32, 8, 0) == 0
    assert api.decode_workspace_bytes(1, 32, 8, 1024, 64) == 0


def test_debug_entry_points_reject_bad_arguments():
    L = api.lib()
    assert L.jl_debug_schedule(A, 4, A, 4, 0, A, A, A, None) == api.JL_ERR_INVALID_ARG
    assert L.jl_debug_schedule(A, -1, A, 4, 8, A, A, A, None) == api.JL_ERR_INVALID_ARG
    bq, bk, nq, nk = (ctypes.c_int(), ctypes.c_int(), ctypes.c_int(), ctypes.c_int())
    rc = L.jl_debug_prefill_tiles(2048, 2, 1, 128, None, 0, ctypes.byref(bq), ctypes.byref(bk),
                                  ctypes.byref(nq), ctypes.byref(nk), None)
    assert rc == api.JL_ERR_INVALID_ARG  # no buffer, but the geometry is reported
    assert (bq.value, bk.value) == (128, 64)  # 256 rows = 128 positions x 2 heads
    assert (nq.value, nk.value) == (16, 32)


def _literal(ws=A, ws_bytes=None, B=1, Hq=4, Hkv=2, L=64, w=16, w0=4, o=A):
    if ws_bytes is None:
        ws_bytes = api.prefill_literal_workspace_bytes(B, Hq, Hkv, L)
    return api.lib().jl_bifocal_prefill_literal(A, A, A, o, None, B, Hq, Hkv, L, 128, 1e6, w, w0,
                                                ws, ws_bytes, None)


def test_literal_workspace_size_and_rejections():
    B, Hq, Hkv, L = 2, 8, 2, 1000
    n = api.prefill_literal_workspace_bytes(B, Hq, Hkv, L)
    o_bytes = 3 * B * L * Hq * 128 * 4
    lse_bytes = -(-3 * B * Hq * L * 4 // 256) * 256
    img = B * Hkv * (-(-L // 64)) * 16384  # V^T tile images only: K is read raw
    retry = 256 + 4 * B * Hkv * L  # the windows' counters and list of blocks for the checked rerun
    assert n == o_bytes + lse_bytes + img + retry
    assert api.prefill_literal_workspace_bytes(B, 7, Hkv, L) == 0
    assert api.prefill_literal_workspace_bytes(B, Hq, Hkv, L, 64) == 0
    assert _literal(ws=None) == api.JL_ERR_WORKSPACE
    assert _literal(ws_bytes=1024) == api.JL_ERR_WORKSPACE
    assert _literal(ws=P(0x1010)) == api.JL_ERR_INVALID_ARG  # not 256-byte aligned
    assert _literal(o=None) == api.JL_ERR_INVALID_ARG
    assert _literal(w=0) == api.JL_ERR_INVALID_ARG
