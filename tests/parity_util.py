"""Helpers shared by the GPU parity tests (marshalling and comparison only)."""
import sys

import numpy as np

# Output tolerance of the bf16 result against the fp64 oracle.
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def say(*args):
    """Progress line, flushed before each GPU step so a failing step is named."""
    print("[gpu-test]", *args, flush=True)
    sys.stdout.flush()


def to_dev(bits):
    import torch
    a = np.ascontiguousarray(bits)
    return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to("cuda")


def to_f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def assert_close(got, want, max_abs=MAX_ABS, mean_abs=MEAN_ABS, what=""):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    assert np.isfinite(got).all(), "%s: non-finite output" % what
    err = np.abs(got - want)
    mx, mn = float(err.max()), float(err.mean())
    say("%s max_abs=%.3e mean_abs=%.3e n=%d" % (what, mx, mn, err.size))
    assert mx <= max_abs, "%s: max abs err %.4e > %.1e" % (what, mx, max_abs)
    assert mn <= mean_abs, "%s: mean abs err %.4e > %.1e" % (what, mn, mean_abs)
    return mx, mn


def prefill_block_q(Hq, Hkv):
    """Query positions per prefill workgroup, as the library reports it
    (jl_debug_prefill_tiles fills the geometry even without a buffer)."""
    import ctypes
    from paper_2607_07740_amd import api
    bq, bk, nq, nk = (ctypes.c_int() for _ in range(4))
    api.lib().jl_debug_prefill_tiles(64, Hq, Hkv, 0, None, 0, ctypes.byref(bq), ctypes.byref(bk),
                                     ctypes.byref(nq), ctypes.byref(nk), None)
    assert bq.value > 0
    return bq.value


def sample_positions(L, w0, w_pre, G, block_q, n_random, seed=0):
    """Stratified query positions: window edges, block edges, G-group edges,
    multiples of the pretraining window, the middle and the end, plus seeded
    uniform positions."""
    qs = {0, 1, w0 - 1, w0, w0 + 1, w0 + 2, w0 + block_q, w0 + block_q + 1, L // 2, L - 2, L - 1,
          block_q - 1, block_q, 63, 64, 65}
    for m in (1, 2, 3):
        for dlt in (-1, 0, 1):
            qs.add(m * w_pre + dlt)
    t = (L // 2) // max(G, 1)
    for dlt in (-1, 0, 1):
        qs.add(G * t + dlt)
    rng = np.random.default_rng(seed)
    qs.update(int(x) for x in rng.integers(0, L, size=n_random))
    return sorted(q for q in qs if 0 <= q < L)


def rows_for(B, Hq, positions):
    return np.array([[b, h, q] for b in range(B) for h in range(Hq) for q in positions],
                    dtype=np.int64)
