"""ctypes binding of the fp64 CPU oracle (``jl_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP implementation.  Every function follows Jet-Long (arXiv
2607.07740): Eq. (2) group size, Eq. (3) remote map, Eq. (1) two-window score,
Sec. 3.3 three windows merged by Eq. (7), Sec. 3.2 decode on a raw cache, and
the frequency-interpolation remote map of the Sec. 4.5 ablation.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "jl_oracle.c")
_LIB = os.path.join(_HERE, "libjloracle.so")
# JETLONG_ORACLE_LIB may name a prebuilt variant (the sanitizer build); it is loaded as is
_LIB_OVERRIDE = os.environ.get("JETLONG_ORACLE_LIB")

_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with the host C compiler (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            lib = ctypes.CDLL(_LIB_OVERRIDE)
        else:
            build()  # compiles when the library is missing or older than the source
            lib = ctypes.CDLL(_LIB)
        i64, i32, dbl, vp = ctypes.c_int64, ctypes.c_int, ctypes.c_double, ctypes.c_void_p
        lib.jlo_group_size.restype = i64
        lib.jlo_group_size.argtypes = [i64, i64]
        lib.jlo_remote_position.restype = i64
        lib.jlo_remote_position.argtypes = [i64, i64]
        lib.jlo_position_offset.restype = i64
        lib.jlo_position_offset.argtypes = [i64, i64]
        lib.jlo_rope_rotate.restype = None
        lib.jlo_rope_rotate.argtypes = [vp, i32, dbl, dbl, vp]
        lib.jlo_rope_rotate_freqs.restype = None
        lib.jlo_rope_rotate_freqs.argtypes = [vp, i32, dbl, vp, vp]
        lib.jlo_yarn_frequencies.restype = None
        lib.jlo_yarn_frequencies.argtypes = [i32, dbl, dbl, dbl, dbl, dbl, vp]
        lib.jlo_prefill_rows_map.restype = i32
        lib.jlo_prefill_rows_map.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, dbl, i64, i64,
                                             i32, i32, vp, i64, vp, vp]
        lib.jlo_prefill_rows.restype = i32
        lib.jlo_prefill_rows.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, dbl, i64, i64, i32,
                                         vp, i64, vp, vp]
        lib.jlo_decode_map.restype = i32
        lib.jlo_decode_map.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, dbl, i64, i64,
                                       i32, i32, vp, vp]
        lib.jlo_decode.restype = i32
        lib.jlo_decode.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, dbl, i64, i64, i32,
                                   vp, vp]
        lib.jlo_window_states.restype = i32
        lib.jlo_window_states.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, dbl, i64, i64,
                                          i64, i64, i64, vp, vp]
        lib.jlo_max_threads.restype = i32
        lib.jlo_max_threads.argtypes = []
        _lib = lib
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def _bf16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("oracle inputs are bf16 bit patterns (uint16), got %s" % a.dtype)
    return a


def group_size(L: int, w_pretrained: int) -> int:
    """Eq. (2): G = max(1, ceil(L / w_pretrained)); -1 for invalid arguments."""
    return int(_load().jlo_group_size(L, w_pretrained))


def remote_position(x: int, G: int) -> int:
    """Eq. (3): f(x) = floor(x / G)."""
    return int(_load().jlo_remote_position(x, G))


def position_offset(x: int, G: int) -> int:
    """Eq. (5): Delta(x) = f(x) - x."""
    return int(_load().jlo_position_offset(x, G))


def rope_rotate(x: np.ndarray, pos: float, theta: float) -> np.ndarray:
    """Explicit rotate-half RoPE of one fp64 vector to position ``pos``."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty_like(x)
    _load().jlo_rope_rotate(_ptr(x), x.shape[0], float(pos), float(theta), _ptr(y))
    return y


def rope_rotate_freqs(x: np.ndarray, pos: float, omega: np.ndarray) -> np.ndarray:
    """Rotate-half rotation of one fp64 vector with explicit frequencies omega [d/2]."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    omega = np.ascontiguousarray(omega, dtype=np.float64)
    assert omega.shape == (x.shape[0] // 2,)
    y = np.empty_like(x)
    _load().jlo_rope_rotate_freqs(_ptr(x), x.shape[0], float(pos), _ptr(omega), _ptr(y))
    return y


def yarn_frequencies(d: int, theta: float, L: float, w_pretrained: float, alpha: float = 1.0,
                     beta: float = 32.0) -> np.ndarray:
    """Remote-view frequencies of the frequency-interpolation map (Sec. 4.5,
    Table 6): YaRN's per-pair ramp with s = max(1, L / w_pretrained)."""
    out = np.empty(d // 2, dtype=np.float64)
    _load().jlo_yarn_frequencies(int(d), float(theta), float(L), float(w_pretrained),
                                 float(alpha), float(beta), _ptr(out))
    return out


REMOTE_MAPS = {"alias": 0, "freq": 1}


def max_threads() -> int:
    return int(_load().jlo_max_threads())


def prefill_rows(q, k, v, rows, *, theta: float, w_pretrained: int = 1, w_local: int = 0,
                 bifocal: bool = True, want_lse: bool = False, remote_map: str = "alias"):
    """Oracle output rows of a prefill call.

    q: uint16 [B, L, Hq, d]; k, v: uint16 [B, L, Hkv, d] (bf16 bits, raw pre-RoPE).
    rows: int64 [n, 3] of (b, h, q).  remote_map: "alias" (Eq. (3)) or "freq"
    (frequency interpolation, Sec. 4.5).  Returns fp64 [n, d] (and fp64 [n]
    LSE), plus the number of host threads the oracle used.
    """
    q, k, v = _bf16(q), _bf16(k), _bf16(v)
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    assert k.shape == (B, L, Hkv, d) and v.shape == k.shape
    rows = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1, 3)
    out = np.empty((rows.shape[0], d), dtype=np.float64)
    lse = np.empty(rows.shape[0], dtype=np.float64) if want_lse else None
    rc = _load().jlo_prefill_rows_map(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, L, d,
                                      float(theta), int(w_pretrained), int(w_local),
                                      1 if bifocal else 0, REMOTE_MAPS[remote_map], _ptr(rows),
                                      rows.shape[0], _ptr(out),
                                      _ptr(lse) if lse is not None else None)
    if rc < 0:
        raise ValueError("oracle prefill_rows failed with status %d" % -rc)
    return (out, lse, rc) if want_lse else (out, rc)


def all_rows(B: int, Hq: int, L: int) -> np.ndarray:
    b, h, qq = np.meshgrid(np.arange(B), np.arange(Hq), np.arange(L), indexing="ij")
    return np.stack([b.ravel(), h.ravel(), qq.ravel()], axis=1).astype(np.int64)


def prefill(q, k, v, *, theta: float, w_pretrained: int = 1, w_local: int = 0,
            bifocal: bool = True, remote_map: str = "alias"):
    """Full-tensor oracle prefill: fp64 [B, L, Hq, d] and LSE fp64 [B, Hq, L]."""
    B, L, Hq, d = q.shape
    rows = all_rows(B, Hq, L)
    out, lse, _ = prefill_rows(q, k, v, rows, theta=theta, w_pretrained=w_pretrained,
                               w_local=w_local, bifocal=bifocal, want_lse=True,
                               remote_map=remote_map)
    o = out.reshape(B, Hq, L, d).transpose(0, 2, 1, 3).copy()
    return o, lse.reshape(B, Hq, L)


def decode(q, k_cache, v_cache, kv_lens, *, theta: float, w_pretrained: int = 1,
           w_local: int = 0, bifocal: bool = True, remote_map: str = "alias"):
    """Oracle decode: q uint16 [B, Hq, d]; caches uint16 [B, max_len, Hkv, d];
    kv_lens int32 [B].  remote_map "alias" (Eq. (3)) or "freq" (Sec. 4.5, with
    the factor from each sequence's own length).  Returns fp64 [B, Hq, d], LSE
    fp64 [B, Hq], threads used."""
    q, k_cache, v_cache = _bf16(q), _bf16(k_cache), _bf16(v_cache)
    B, Hq, d = q.shape
    _, max_len, Hkv, _ = k_cache.shape
    kv_lens = np.ascontiguousarray(kv_lens, dtype=np.int32)
    out = np.empty((B, Hq, d), dtype=np.float64)
    lse = np.empty((B, Hq), dtype=np.float64)
    rc = _load().jlo_decode_map(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(kv_lens), max_len,
                                B, Hq, Hkv, d, float(theta), int(w_pretrained), int(w_local),
                                1 if bifocal else 0, REMOTE_MAPS[remote_map], _ptr(out),
                                _ptr(lse))
    if rc < 0:
        raise ValueError("oracle decode failed with status %d" % -rc)
    return out, lse, rc


def window_states(q, k, v, b: int, h: int, qpos: int, *, theta: float, w_pretrained: int,
                  w_local: int):
    """The three Sec. 3.3 window states for one row: (O [3, d], lse [3]) for A, B, C."""
    q, k, v = _bf16(q), _bf16(k), _bf16(v)
    B, L, Hq, d = q.shape
    Hkv = k.shape[2]
    o3 = np.empty((3, d), dtype=np.float64)
    l3 = np.empty(3, dtype=np.float64)
    rc = _load().jlo_window_states(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, L, d, float(theta),
                                   int(w_pretrained), int(w_local), b, h, qpos, _ptr(o3),
                                   _ptr(l3))
    if rc != 0:
        raise ValueError("oracle window_states failed with status %d" % -rc)
    return o3, l3
