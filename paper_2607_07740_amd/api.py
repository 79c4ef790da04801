"""Thin ctypes binding of libjetlong.so (C ABI in include/jetlong.h).

Argument marshalling only: every step of the attention runs in the library's
HIP kernels.  PyTorch supplies device memory and the current stream.  If the
library is not built this module raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
# JETLONG_LIB may name another build of the same library (the host-sanitizer build)
LIB_PATH = os.environ.get("JETLONG_LIB") or os.path.join(HERE, "libjetlong.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "jetlong.h")

JL_OK, JL_ERR_INVALID_ARG, JL_ERR_UNSUPPORTED, JL_ERR_WORKSPACE, JL_ERR_HIP = range(5)
REMOTE_MAPS = {"alias": 0, "freq": 1}  # JL_REMOTE_ALIAS, JL_REMOTE_FREQ
TILE_SKIP, TILE_LOCAL, TILE_REMOTE, TILE_MIXED = range(4)

_lib = None


class JetLongError(RuntimeError):
    def __init__(self, status: int, name: str, detail: str):
        super().__init__("%s (%d): %s" % (name, status, detail))
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libjetlong.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libjetlong.so is not built (run __graft_entry__.build()); "
                               "the HIP library is the only implementation")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, dbl, sz = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double,
                                 ctypes.c_size_t)
        L.jl_status_string.restype = ctypes.c_char_p
        L.jl_status_string.argtypes = [i32]
        L.jl_last_error.restype = ctypes.c_char_p
        L.jl_last_error.argtypes = []
        L.jl_version.restype = i32
        L.jl_version.argtypes = []
        L.jl_group_size.restype = i64
        L.jl_group_size.argtypes = [i64, i64]
        L.jl_bifocal_prefill.restype = i32
        L.jl_bifocal_prefill.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, dbl, i32,
                                         i32, vp]
        L.jl_bifocal_prefill_map.restype = i32
        L.jl_bifocal_prefill_map.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, dbl,
                                             i32, i32, i32, vp]
        L.jl_bifocal_prefill_chunk.restype = i32
        L.jl_bifocal_prefill_chunk.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                               i32, dbl, i32, i32, vp]
        L.jl_rope_attention_chunk.restype = i32
        L.jl_rope_attention_chunk.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                              i32, dbl, vp]
        L.jl_bifocal_prefill_chunk_paged.restype = i32
        L.jl_bifocal_prefill_chunk_paged.argtypes = [vp, vp, vp, vp, i32, i32, i32, vp, vp, i32,
                                                     i32, i32, i32, i32, i32, dbl, i32, i32, vp]
        L.jl_rope_attention_chunk_paged.restype = i32
        L.jl_rope_attention_chunk_paged.argtypes = [vp, vp, vp, vp, i32, i32, i32, vp, vp, i32,
                                                    i32, i32, i32, i32, i32, dbl, vp]
        L.jl_bifocal_prefill_varlen.restype = i32
        L.jl_bifocal_prefill_varlen.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32,
                                                i32, dbl, i32, i32, vp]
        L.jl_bifocal_prefill_varlen_map.restype = i32
        L.jl_bifocal_prefill_varlen_map.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32,
                                                    i32, i32, dbl, i32, i32, i32, vp]
        L.jl_rope_attention_varlen.restype = i32
        L.jl_rope_attention_varlen.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32,
                                               i32, dbl, vp]
        L.jl_decode_map_workspace_bytes.restype = sz
        L.jl_decode_map_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32]
        L.jl_bifocal_decode_map.restype = i32
        L.jl_bifocal_decode_map.argtypes = [vp, vp, vp, vp, i32, vp, i32, i32, i32, i32, dbl,
                                            i32, i32, i32, vp, sz, vp]
        L.jl_rope_attention.restype = i32
        L.jl_rope_attention.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, dbl, vp]
        L.jl_prefill_literal_workspace_bytes.restype = sz
        L.jl_prefill_literal_workspace_bytes.argtypes = [i32, i32, i32, i32, i32]
        L.jl_bifocal_prefill_literal.restype = i32
        L.jl_bifocal_prefill_literal.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, dbl,
                                                 i32, i32, vp, sz, vp]
        L.jl_decode_workspace_bytes.restype = sz
        L.jl_decode_workspace_bytes.argtypes = [i32, i32, i32, i32, i32]
        L.jl_bifocal_decode.restype = i32
        L.jl_bifocal_decode.argtypes = [vp, vp, vp, vp, i32, vp, i32, i32, i32, i32, dbl, i32, i32,
                                        vp, sz, vp]
        L.jl_bifocal_decode_noalloc.restype = i32
        L.jl_bifocal_decode_noalloc.argtypes = [vp, vp, vp, vp, i32, vp, i32, i32, i32, i32, dbl,
                                                i32, i32, vp]
        L.jl_rope_attention_decode.restype = i32
        L.jl_rope_attention_decode.argtypes = [vp, vp, vp, vp, i32, vp, i32, i32, i32, i32, dbl,
                                               vp, sz, vp]
        L.jl_bifocal_decode_paged.restype = i32
        L.jl_bifocal_decode_paged.argtypes = [vp, vp, vp, vp, i32, i32, i32, vp, vp, i32, i32, i32,
                                              i32, dbl, i32, i32, vp, sz, vp]
        L.jl_bifocal_decode_paged_map.restype = i32
        L.jl_bifocal_decode_paged_map.argtypes = [vp, vp, vp, vp, i32, i32, i32, vp, vp, i32,
                                                  i32, i32, i32, dbl, i32, i32, i32, vp, sz, vp]
        L.jl_rope_attention_decode_paged.restype = i32
        L.jl_rope_attention_decode_paged.argtypes = [vp, vp, vp, vp, i32, i32, i32, vp, vp, i32,
                                                     i32, i32, i32, dbl, vp, sz, vp]
        L.jl_debug_schedule.restype = i32
        L.jl_debug_schedule.argtypes = [vp, i32, vp, i32, i32, vp, vp, vp, vp]
        L.jl_debug_prefill_tiles.restype = i32
        L.jl_debug_prefill_tiles.argtypes = [i32, i32, i32, i32, vp, i64,
                                             ctypes.POINTER(i32), ctypes.POINTER(i32),
                                             ctypes.POINTER(i32), ctypes.POINTER(i32), vp]
        L.jl_debug_prefill_rescale_log2.restype = dbl
        L.jl_debug_prefill_rescale_log2.argtypes = [dbl]
        L.jl_debug_kernel_events.restype = i32
        L.jl_debug_kernel_events.argtypes = [i32, vp, vp]
        L.jl_release_caches.restype = None
        L.jl_release_caches.argtypes = []
        _lib = L
    return _lib


def declared_functions() -> list:
    """Function names declared in include/jetlong.h."""
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(jl_[a-z0-9_]+)\s*\(", src)))


def _check(status: int) -> None:
    if status != JL_OK:
        L = lib()
        raise JetLongError(status, L.jl_status_string(status).decode(),
                           L.jl_last_error().decode())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t, name, dtype=None, shape=None, device=None):
    """Device pointer of a contiguous CUDA tensor.  The library reads and writes
    through raw pointers, so a caller-supplied output must have exactly the
    shape the call writes (shape), and every tensor must sit on the query's
    device (device)."""
    import torch
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError("%s must be a CUDA (HIP) tensor" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, the query on %s" % (name, t.device, device))
    return ctypes.c_void_p(t.data_ptr())


def _bf16(t, name, q, shape=None):
    """A bf16 tensor of the call, on q's device."""
    import torch
    return _dev(t, name, torch.bfloat16, shape, q.device)


def _f32(t, name, q, shape):
    """An optional fp32 output (None passes a null pointer), on q's device."""
    import torch
    return None if t is None else _dev(t, name, torch.float32, shape, q.device)


def _i32(t, name, q):
    import torch
    return _dev(t, name, torch.int32, None, q.device)


def group_size(L: int, w_pretrained: int) -> int:
    return int(lib().jl_group_size(L, w_pretrained))


def _prefill(bifocal, q, k, v, w_pretrained, w_local, rope_theta, out, lse, want_lse, stream,
             remote_map="alias"):
    import torch
    B, L, Hq, D = q.shape
    Hkv = k.shape[2]
    if k.shape != (B, L, Hkv, D) or v.shape != k.shape:
        raise ValueError("k and v must be [B, L, Hkv, D] matching q [B, L, Hq, D]")
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, L), dtype=torch.float32, device=q.device)
    args = [_bf16(q, "q", q), _bf16(k, "k", q), _bf16(v, "v", q),
            _bf16(out, "out", q, q.shape), _f32(lse, "lse", q, (B, Hq, L)), B, Hq, Hkv, L, D,
            float(rope_theta)]
    if bifocal and remote_map != "alias":
        _check(lib().jl_bifocal_prefill_map(*args, int(w_pretrained), int(w_local),
                                            REMOTE_MAPS[remote_map], _stream(stream)))
    elif bifocal:
        _check(lib().jl_bifocal_prefill(*args, int(w_pretrained), int(w_local), _stream(stream)))
    else:
        _check(lib().jl_rope_attention(*args, _stream(stream)))
    return (out, lse) if want_lse else out


def bifocal_prefill(q, k, v, *, w_pretrained: int, w_local: int, rope_theta: float = 1e6,
                    out=None, lse=None, want_lse: bool = False, stream=None,
                    remote_map: str = "alias"):
    """jl_bifocal_prefill: q [B, L, Hq, 128], k/v [B, L, Hkv, 128] raw bf16 -> out bf16.
    remote_map "freq" calls jl_bifocal_prefill_map with JL_REMOTE_FREQ (Sec. 4.5)."""
    if remote_map not in REMOTE_MAPS:
        raise ValueError("remote_map must be one of %s" % sorted(REMOTE_MAPS))
    return _prefill(True, q, k, v, w_pretrained, w_local, rope_theta, out, lse,
                    want_lse or lse is not None, stream, remote_map)


def rope_attention(q, k, v, *, rope_theta: float = 1e6, out=None, lse=None,
                   want_lse: bool = False, stream=None):
    """jl_rope_attention: vanilla causal RoPE attention with the same kernel."""
    return _prefill(False, q, k, v, 1, 0, rope_theta, out, lse, want_lse or lse is not None,
                    stream)


def prefill_chunk(q, k_cache, v_cache, *, q_start: int, w_pretrained: int = 1, w_local: int = 0,
                  rope_theta: float = 1e6, bifocal: bool = True, out=None, lse=None,
                  want_lse: bool = False, stream=None):
    """jl_bifocal_prefill_chunk / jl_rope_attention_chunk: q [B, n, Hq, 128] raw queries at
    positions q_start .. q_start + n - 1 over the raw caches [B, max_len, Hkv, 128]."""
    import torch
    B, n, Hq, D = q.shape
    _, max_len, Hkv, _ = k_cache.shape
    if k_cache.shape != (B, max_len, Hkv, D) or v_cache.shape != k_cache.shape:
        raise ValueError("caches must be [B, max_len, Hkv, D] matching q [B, n, Hq, D]")
    if out is None:
        out = torch.empty_like(q)
    want_lse = want_lse or lse is not None
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, n), dtype=torch.float32, device=q.device)
    args = [_bf16(q, "q", q), _bf16(k_cache, "k_cache", q), _bf16(v_cache, "v_cache", q),
            _bf16(out, "out", q, q.shape), _f32(lse, "lse", q, (B, Hq, n)), B, Hq, Hkv,
            int(q_start), n, max_len, D, float(rope_theta)]
    if bifocal:
        _check(lib().jl_bifocal_prefill_chunk(*args, int(w_pretrained), int(w_local),
                                              _stream(stream)))
    else:
        _check(lib().jl_rope_attention_chunk(*args, _stream(stream)))
    return (out, lse) if want_lse else out


def prefill_chunk_paged(q, k_pages, v_pages, block_table, *, q_start: int,
                        w_pretrained: int = 1, w_local: int = 0, rope_theta: float = 1e6,
                        bifocal: bool = True, out=None, lse=None, want_lse: bool = False,
                        stream=None):
    """jl_bifocal_prefill_chunk_paged / jl_rope_attention_chunk_paged: q [B, n, Hq, 128] raw
    queries at positions q_start .. q_start + n - 1, pools [n_pages, page_size, Hkv, 128] raw,
    block_table int32 [B, max_pages] on the device."""
    import torch
    B, n, Hq, D = q.shape
    n_pages, page_size, Hkv, _ = k_pages.shape
    if k_pages.shape != (n_pages, page_size, Hkv, D) or v_pages.shape != k_pages.shape:
        raise ValueError("page pools must be [n_pages, page_size, Hkv, D]")
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("block_table must be [B, max_pages]")
    max_pages = block_table.shape[1]
    if out is None:
        out = torch.empty_like(q)
    want_lse = want_lse or lse is not None
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, n), dtype=torch.float32, device=q.device)
    args = [_bf16(q, "q", q), _bf16(k_pages, "k_pages", q), _bf16(v_pages, "v_pages", q),
            _i32(block_table, "block_table", q), max_pages, page_size, n_pages,
            _bf16(out, "out", q, q.shape), _f32(lse, "lse", q, (B, Hq, n)), B, Hq, Hkv,
            int(q_start), n, D, float(rope_theta)]
    if bifocal:
        _check(lib().jl_bifocal_prefill_chunk_paged(*args, int(w_pretrained), int(w_local),
                                                    _stream(stream)))
    else:
        _check(lib().jl_rope_attention_chunk_paged(*args, _stream(stream)))
    return (out, lse) if want_lse else out


def prefill_varlen(q, k, v, cu_seqlens, *, max_seqlen: int, w_pretrained: int = 1,
                   w_local: int = 0, rope_theta: float = 1e6, bifocal: bool = True, out=None,
                   lse=None, want_lse: bool = False, stream=None, remote_map: str = "alias"):
    """jl_bifocal_prefill_varlen / jl_rope_attention_varlen: packed sequences, q [T, Hq, 128],
    k, v [T, Hkv, 128], cu_seqlens int32 [B + 1] on the device; lse is [Hq, T].
    remote_map "freq" calls jl_bifocal_prefill_varlen_map with JL_REMOTE_FREQ (Sec. 4.5)."""
    if remote_map not in REMOTE_MAPS:
        raise ValueError("remote_map must be one of %s" % sorted(REMOTE_MAPS))
    import torch
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    if k.shape != (T, Hkv, D) or v.shape != k.shape:
        raise ValueError("k and v must be [T, Hkv, D] matching q [T, Hq, D]")
    if cu_seqlens.dim() != 1 or cu_seqlens.numel() < 2:
        raise ValueError("cu_seqlens must be [B + 1] with B >= 1")
    B = cu_seqlens.numel() - 1
    if out is None:
        out = torch.empty_like(q)
    want_lse = want_lse or lse is not None
    if lse is None and want_lse:
        lse = torch.empty((Hq, T), dtype=torch.float32, device=q.device)
    args = [_bf16(q, "q", q), _bf16(k, "k", q), _bf16(v, "v", q),
            _bf16(out, "out", q, q.shape), _f32(lse, "lse", q, (Hq, T)),
            _i32(cu_seqlens, "cu_seqlens", q), B, T, int(max_seqlen), Hq, Hkv, D,
            float(rope_theta)]
    if bifocal and remote_map != "alias":
        _check(lib().jl_bifocal_prefill_varlen_map(*args, int(w_pretrained), int(w_local),
                                                   REMOTE_MAPS[remote_map], _stream(stream)))
    elif bifocal:
        _check(lib().jl_bifocal_prefill_varlen(*args, int(w_pretrained), int(w_local),
                                               _stream(stream)))
    else:
        _check(lib().jl_rope_attention_varlen(*args, _stream(stream)))
    return (out, lse) if want_lse else out


def prefill_literal_workspace_bytes(B: int, Hq: int, Hkv: int, L: int,
                                    head_dim: int = 128) -> int:
    return int(lib().jl_prefill_literal_workspace_bytes(B, Hq, Hkv, L, head_dim))


def bifocal_prefill_literal(q, k, v, *, w_pretrained: int, w_local: int, rope_theta: float = 1e6,
                            out=None, lse=None, want_lse: bool = False, workspace=None,
                            stream=None):
    """jl_bifocal_prefill_literal: Eq. (7) as three window passes and a merge.

    Returns out (and lse when asked).  workspace, if given, is a uint8 CUDA
    tensor of at least prefill_literal_workspace_bytes(...) bytes; after the
    call literal_window_states(workspace, ...) views the per-window results.
    """
    import torch
    B, L, Hq, D = q.shape
    Hkv = k.shape[2]
    if k.shape != (B, L, Hkv, D) or v.shape != k.shape:
        raise ValueError("k and v must be [B, L, Hkv, D] matching q [B, L, Hq, D]")
    want_lse = want_lse or lse is not None
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, L), dtype=torch.float32, device=q.device)
    need = prefill_literal_workspace_bytes(B, Hq, Hkv, L, D)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    _check(lib().jl_bifocal_prefill_literal(
        _bf16(q, "q", q), _bf16(k, "k", q), _bf16(v, "v", q), _bf16(out, "out", q, q.shape),
        _f32(lse, "lse", q, (B, Hq, L)), B, Hq, Hkv, L, D, float(rope_theta), int(w_pretrained),
        int(w_local), _dev(workspace, "workspace", device=q.device),
        workspace.numel() * workspace.element_size(), _stream(stream)))
    return (out, lse) if want_lse else out


def literal_window_states(workspace, B: int, Hq: int, L: int, head_dim: int = 128):
    """Views of a literal-prefill workspace: (O [3, B, L, Hq, D] fp32, LSE [3, B, Hq, L] fp32)."""
    import torch
    n_o = 3 * B * L * Hq * head_dim
    f = workspace[: 4 * (n_o + 3 * B * Hq * L)].view(torch.float32)
    return (f[:n_o].view(3, B, L, Hq, head_dim), f[n_o:].view(3, B, Hq, L))


def decode_workspace_bytes(B: int, Hq: int, Hkv: int, max_len: int, head_dim: int = 128) -> int:
    return int(lib().jl_decode_workspace_bytes(B, Hq, Hkv, max_len, head_dim))


def _decode(bifocal, q, k_cache, v_cache, kv_lens, w_pretrained, w_local, rope_theta, out,
            workspace, stream):
    import torch
    B, Hq, D = q.shape
    _, max_len, Hkv, _ = k_cache.shape
    if k_cache.shape != (B, max_len, Hkv, D) or v_cache.shape != k_cache.shape:
        raise ValueError("caches must be [B, max_len, Hkv, D]")
    if kv_lens.shape != (B,):
        raise ValueError("kv_lens must be [B]")
    if out is None:
        out = torch.empty_like(q)
    need = decode_workspace_bytes(B, Hq, Hkv, max_len, D)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    args = [_bf16(q, "q", q), _bf16(k_cache, "k_cache", q), _bf16(v_cache, "v_cache", q),
            _i32(kv_lens, "kv_lens", q), max_len, _bf16(out, "out", q, q.shape), B, Hq, Hkv, D,
            float(rope_theta)]
    ws = [_dev(workspace, "workspace", device=q.device),
          workspace.numel() * workspace.element_size()]
    if bifocal:
        _check(lib().jl_bifocal_decode(*args, int(w_pretrained), int(w_local), *ws,
                                       _stream(stream)))
    else:
        _check(lib().jl_rope_attention_decode(*args, *ws, _stream(stream)))
    return out


def bifocal_decode_noalloc(q, k_cache, v_cache, kv_lens, *, w_pretrained: int, w_local: int,
                           rope_theta: float = 1e6, out=None, stream=None):
    """jl_bifocal_decode_noalloc: jl_bifocal_decode without a workspace; the library's
    fixed per-device array holds the split states and the cos/sin table."""
    import torch
    B, Hq, D = q.shape
    _, max_len, Hkv, _ = k_cache.shape
    if k_cache.shape != (B, max_len, Hkv, D) or v_cache.shape != k_cache.shape:
        raise ValueError("caches must be [B, max_len, Hkv, D]")
    if kv_lens.shape != (B,):
        raise ValueError("kv_lens must be [B]")
    if out is None:
        out = torch.empty_like(q)
    _check(lib().jl_bifocal_decode_noalloc(
        _bf16(q, "q", q), _bf16(k_cache, "k_cache", q), _bf16(v_cache, "v_cache", q),
        _i32(kv_lens, "kv_lens", q), max_len, _bf16(out, "out", q, q.shape), B, Hq, Hkv, D,
        float(rope_theta),
        int(w_pretrained), int(w_local), _stream(stream)))
    return out


def bifocal_decode(q, k_cache, v_cache, kv_lens, *, w_pretrained: int, w_local: int,
                   rope_theta: float = 1e6, out=None, workspace=None, stream=None,
                   remote_map: str = "alias"):
    """jl_bifocal_decode: q [B, Hq, 128] raw, caches [B, max_len, Hkv, 128] raw, kv_lens int32.
    remote_map "freq" calls jl_bifocal_decode_map with JL_REMOTE_FREQ (Sec. 4.5)."""
    if remote_map == "alias":
        return _decode(True, q, k_cache, v_cache, kv_lens, w_pretrained, w_local, rope_theta,
                       out, workspace, stream)
    import torch
    if remote_map not in REMOTE_MAPS:
        raise ValueError("remote_map must be one of %s" % sorted(REMOTE_MAPS))
    B, Hq, D = q.shape
    _, max_len, Hkv, _ = k_cache.shape
    if k_cache.shape != (B, max_len, Hkv, D) or v_cache.shape != k_cache.shape:
        raise ValueError("caches must be [B, max_len, Hkv, D]")
    if kv_lens.shape != (B,):
        raise ValueError("kv_lens must be [B]")
    if out is None:
        out = torch.empty_like(q)
    need = decode_map_workspace_bytes(B, Hq, Hkv, max_len, D, remote_map)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    _check(lib().jl_bifocal_decode_map(
        _bf16(q, "q", q), _bf16(k_cache, "k_cache", q), _bf16(v_cache, "v_cache", q),
        _i32(kv_lens, "kv_lens", q), max_len, _bf16(out, "out", q, q.shape), B, Hq, Hkv, D,
        float(rope_theta), int(w_pretrained), int(w_local), REMOTE_MAPS[remote_map],
        _dev(workspace, "workspace", device=q.device),
        workspace.numel() * workspace.element_size(), _stream(stream)))
    return out


def decode_map_workspace_bytes(B: int, Hq: int, Hkv: int, max_len: int, head_dim: int = 128,
                               remote_map: str = "alias") -> int:
    return int(lib().jl_decode_map_workspace_bytes(B, Hq, Hkv, max_len, head_dim,
                                                   REMOTE_MAPS[remote_map]))


def rope_attention_decode(q, k_cache, v_cache, kv_lens, *, rope_theta: float = 1e6, out=None,
                          workspace=None, stream=None):
    """jl_rope_attention_decode: vanilla RoPE decode with the same kernels."""
    return _decode(False, q, k_cache, v_cache, kv_lens, 1, 0, rope_theta, out, workspace, stream)


def decode_paged(q, k_pages, v_pages, block_table, kv_lens, *, w_pretrained: int = 1,
                 w_local: int = 0, rope_theta: float = 1e6, bifocal: bool = True, out=None,
                 workspace=None, stream=None, remote_map: str = "alias"):
    """jl_bifocal_decode_paged / jl_rope_attention_decode_paged: q [B, Hq, 128] raw,
    pools [n_pages, page_size, Hkv, 128] raw, block_table int32 [B, max_pages],
    kv_lens int32 [B].  remote_map "freq" calls jl_bifocal_decode_paged_map with
    JL_REMOTE_FREQ (Sec. 4.5)."""
    import torch
    B, Hq, D = q.shape
    n_pages, page_size, Hkv, _ = k_pages.shape
    if k_pages.shape != (n_pages, page_size, Hkv, D) or v_pages.shape != k_pages.shape:
        raise ValueError("page pools must be [n_pages, page_size, Hkv, D]")
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("block_table must be [B, max_pages]")
    if kv_lens.shape != (B,):
        raise ValueError("kv_lens must be [B]")
    max_pages = block_table.shape[1]
    if remote_map not in REMOTE_MAPS:
        raise ValueError("remote_map must be one of %s" % sorted(REMOTE_MAPS))
    if out is None:
        out = torch.empty_like(q)
    if remote_map != "alias" and bifocal:
        need = decode_map_workspace_bytes(B, Hq, Hkv, max_pages * page_size, D, remote_map)
    else:
        need = decode_workspace_bytes(B, Hq, Hkv, max_pages * page_size, D)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    args = [_bf16(q, "q", q), _bf16(k_pages, "k_pages", q), _bf16(v_pages, "v_pages", q),
            _i32(block_table, "block_table", q), max_pages, page_size, n_pages,
            _i32(kv_lens, "kv_lens", q), _bf16(out, "out", q, q.shape), B, Hq, Hkv, D,
            float(rope_theta)]
    ws = [_dev(workspace, "workspace", device=q.device),
          workspace.numel() * workspace.element_size()]
    if bifocal and remote_map != "alias":
        _check(lib().jl_bifocal_decode_paged_map(*args, int(w_pretrained), int(w_local),
                                                 REMOTE_MAPS[remote_map], *ws, _stream(stream)))
    elif bifocal:
        _check(lib().jl_bifocal_decode_paged(*args, int(w_pretrained), int(w_local), *ws,
                                             _stream(stream)))
    else:
        _check(lib().jl_rope_attention_decode_paged(*args, *ws, _stream(stream)))
    return out


def debug_schedule(lengths, positions, w_pretrained: int, stream=None):
    """jl_debug_schedule: device-computed G(L), f(x), Delta(x) (int32 CUDA tensors)."""
    import torch
    nl, npos = lengths.numel(), positions.numel()
    g = torch.empty(nl, dtype=torch.int32, device=lengths.device)
    f = torch.empty((nl, npos), dtype=torch.int32, device=lengths.device)
    dlt = torch.empty((nl, npos), dtype=torch.int32, device=lengths.device)
    _check(lib().jl_debug_schedule(_dev(lengths, "lengths", torch.int32), nl,
                                   _dev(positions, "positions", torch.int32), npos,
                                   int(w_pretrained), _dev(g, "g"), _dev(f, "f"), _dev(dlt, "d"),
                                   _stream(stream)))
    return g, f, dlt


def debug_prefill_tiles(L: int, Hq: int, Hkv: int, w_local: int, device="cuda", stream=None):
    """jl_debug_prefill_tiles: (classes int8 [n_qblocks, n_ktiles], block_q, block_k)."""
    import torch
    bq, bk, nq, nk = (ctypes.c_int(), ctypes.c_int(), ctypes.c_int(), ctypes.c_int())
    # first call with no buffer reports the geometry
    lib().jl_debug_prefill_tiles(L, Hq, Hkv, w_local, None, 0, ctypes.byref(bq),
                                 ctypes.byref(bk), ctypes.byref(nq), ctypes.byref(nk), None)
    if nq.value <= 0:
        _check(JL_ERR_INVALID_ARG)
    out = torch.empty((nq.value, nk.value), dtype=torch.int8, device=device)
    _check(lib().jl_debug_prefill_tiles(L, Hq, Hkv, w_local, _dev(out, "classes"), out.numel(),
                                        ctypes.byref(bq), ctypes.byref(bk), ctypes.byref(nq),
                                        ctypes.byref(nk), _stream(stream)))
    return out, bq.value, bk.value


def release_caches() -> None:
    lib().jl_release_caches()


def debug_prefill_rescale_log2(log2_bound: float) -> float:
    """jl_debug_prefill_rescale_log2: set the prefill rescale bound, return the old one."""
    return float(lib().jl_debug_prefill_rescale_log2(float(log2_bound)))


def debug_kernel_events(which: int, start=None, stop=None) -> None:
    """jl_debug_kernel_events: record torch.cuda.Event pair (start, stop) around
    the prefill attention kernel (which = 0) or the decode split kernel
    (which = 1) of every later call; no events clears the hook."""
    def ev(e):
        if e is None:
            return None
        if e.cuda_event == 0:  # torch creates the HIP event at its first record
            e.record()
        return ctypes.c_void_p(e.cuda_event)
    _check(lib().jl_debug_kernel_events(int(which), ev(start), ev(stop)))
