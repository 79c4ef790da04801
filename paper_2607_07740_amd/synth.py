"""Seeded synthetic inputs for bifocal-RoPE attention.

This module only draws random numbers and rounds them to bf16; it contains no
attention, rotation or schedule arithmetic.  Both the HIP path's tests and the
oracle's tests take their inputs from here.

Recipe: numpy ``default_rng(seed)`` (PCG64), ``standard_normal`` float32 drawn
in the order Q, K, V; where a workload asks for outlier channels,
``rng.choice(d, n, replace=False)`` picks them and K is multiplied by 1.5 on
those channels (this makes attention peaky); finally round-to-nearest-even to
bf16.  Shapes follow the Qwen3 family the paper evaluates (Sec. 4.1): head
dim 128, grouped-query heads, RoPE base 1e6, a 32768-token pretraining window.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np

BF16_NAN = 0x7FC0


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even.

    The sum u + 0x7FFF + lsb is formed in uint32; where it wraps (NaN
    patterns only) the kept bits 16..31 are those the exact sum would give,
    as the result is 16 bits wide either way."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    out = np.empty(u.shape, dtype=np.uint16)
    step = 1 << 24  # chunked to bound temporaries on very large inputs
    flat_u, flat_o = u.reshape(-1), out.reshape(-1)
    for s in range(0, flat_u.size, step):
        c = flat_u[s:s + step]
        r = (c >> 16) & 1
        r += 0x7FFF
        r += c
        r >>= 16
        flat_o[s:s + step] = r
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def prefill_inputs(B: int, Hq: int, Hkv: int, L: int, d: int = 128, *, seed: int = 0,
                   outlier_channels: int = 0):
    """Raw (pre-RoPE) Q [B, L, Hq, d], K and V [B, L, Hkv, d] as bf16 bits."""
    rng = np.random.default_rng(seed)
    q = rng.standard_normal(size=(B, L, Hq, d), dtype=np.float32)
    k = rng.standard_normal(size=(B, L, Hkv, d), dtype=np.float32)
    v = rng.standard_normal(size=(B, L, Hkv, d), dtype=np.float32)
    if outlier_channels:
        ch = rng.choice(d, outlier_channels, replace=False)
        k[..., ch] *= np.float32(1.5)
    return bf16_bits(q), bf16_bits(k), bf16_bits(v)


def decode_inputs(B: int, Hq: int, Hkv: int, max_len: int, kv_lens: Sequence[int], d: int = 128,
                  *, seed: int = 0, nan_tail: bool = False, outlier_channels: int = 0):
    """Raw query [B, Hq, d] and raw caches [B, max_len, Hkv, d] (bf16 bits).

    With ``nan_tail`` every cache slot at or past kv_lens[b] holds bf16 NaN, so
    a kernel that reads past a sequence's length poisons its output.
    """
    rng = np.random.default_rng(seed)
    q = rng.standard_normal(size=(B, Hq, d), dtype=np.float32)
    k = rng.standard_normal(size=(B, max_len, Hkv, d), dtype=np.float32)
    v = rng.standard_normal(size=(B, max_len, Hkv, d), dtype=np.float32)
    if outlier_channels:
        ch = rng.choice(d, outlier_channels, replace=False)
        k[..., ch] *= np.float32(1.5)
    qb, kb, vb = bf16_bits(q), bf16_bits(k), bf16_bits(v)
    lens = np.asarray(kv_lens, dtype=np.int32)
    if nan_tail:
        for b in range(B):
            kb[b, lens[b]:] = BF16_NAN
            vb[b, lens[b]:] = BF16_NAN
    return qb, kb, vb, lens


def ragged_lengths(B: int, lo: int, hi: int, *, seed: int = 0) -> np.ndarray:
    """Seeded uniform integer lengths in [lo, hi]."""
    rng = np.random.default_rng(seed)
    return rng.integers(lo, hi + 1, size=B).astype(np.int32)


def device_inputs(w: "Workload", torch, kv_lens: Optional[Sequence[int]] = None):
    """Timing inputs drawn on the device: torch's seeded CUDA generator
    (``manual_seed(w.seed)``), ``randn`` float32 in the order Q, K, V, the same
    outlier-channel scaling of K, then bf16 (torch's round-to-nearest-even).
    A different random stream from ``make_inputs`` (same distribution and
    shapes); used where a workload is too large to draw on the host quickly.
    Prefill: Q [B, L, Hq, d], K, V [B, L, Hkv, d].  Decode: Q [B, Hq, d], caches
    [B, L, Hkv, d] and the int32 lengths (``kv_lens`` overrides the workload's)."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(w.seed)
    qshape = (w.B, w.L, w.Hq, w.d) if w.kind == "prefill" else (w.B, w.Hq, w.d)
    kshape = (w.B, w.L, w.Hkv, w.d)
    q = torch.randn(qshape, generator=gen, device="cuda").to(torch.bfloat16)
    k = torch.randn(kshape, generator=gen, device="cuda")
    if w.outlier_channels:
        ch = np.random.default_rng(w.seed).choice(w.d, w.outlier_channels, replace=False)
        k[..., torch.from_numpy(ch).cuda()] *= 1.5
    k = k.to(torch.bfloat16)
    v = torch.randn(kshape, generator=gen, device="cuda").to(torch.bfloat16)
    if w.kind == "prefill":
        return q, k, v
    lens = np.asarray(kv_lens if kv_lens is not None else w.kv_lens, dtype=np.int32)
    return q, k, v, lens


@dataclass(frozen=True)
class Workload:
    """One synthetic attention-layer workload (shapes of a Qwen3-like layer)."""
    name: str
    kind: str  # "prefill" or "decode"
    B: int
    Hq: int
    Hkv: int
    L: int  # prefill length, or the cache capacity (max_len) for decode
    w_pretrained: int
    w_local: int
    d: int = 128
    theta: float = 1e6
    outlier_channels: int = 0
    kv_lens: Optional[tuple] = None
    nan_tail: bool = False
    seed: int = 0
    note: str = field(default="", compare=False)


WORKLOADS = {
    w.name: w for w in [
        Workload("tiny_prefill", "prefill", 1, 2, 1, 2048, 512, 128, outlier_channels=8,
                 note="GQA 2:1, G=4; full-tensor parity case"),
        Workload("qwen3_1p7b_within_32k", "prefill", 1, 16, 8, 32768, 32768, 4096,
                 note="L equals the pretraining window: G=1, must equal vanilla"),
        Workload("qwen3_1p7b_prefill_128k", "prefill", 1, 16, 8, 131072, 32768, 4096,
                 outlier_channels=8, note="G=4"),
        Workload("qwen3_8b_prefill_128k", "prefill", 1, 32, 8, 131072, 32768, 4096,
                 note="G=4"),
        Workload("qwen3_8b_prefill_64k", "prefill", 1, 32, 8, 65536, 32768, 4096,
                 note="G=2"),
        Workload("qwen3_4b_decode_128k", "decode", 1, 32, 8, 131072, 32768, 4096,
                 kv_lens=(131072,), note="one query at position 131071, G=4"),
        Workload("qwen3_4b_decode_b8_ragged", "decode", 8, 32, 8, 131072, 32768, 4096,
                 kv_lens=(32768, 32769, 65536, 65537, 98304, 98305, 131071, 131072),
                 nan_tail=True, note="G=1..4 across every boundary; NaN past each length"),
    ]
}


def make_inputs(w: Workload):
    """Inputs of a named workload, as bf16 bit arrays."""
    if w.kind == "prefill":
        return prefill_inputs(w.B, w.Hq, w.Hkv, w.L, w.d, seed=w.seed,
                              outlier_channels=w.outlier_channels)
    return decode_inputs(w.B, w.Hq, w.Hkv, w.L, w.kv_lens, w.d, seed=w.seed,
                         nan_tail=w.nan_tail, outlier_channels=w.outlier_channels)
