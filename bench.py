#!/usr/bin/env python3
"""Benchmark of the fused bifocal-RoPE attention hot path on one MI355X.

One step = one bifocal prefill of a Qwen3-8B-like attention layer at
L = 131072 (B=1, Hq=32, Hkv=8, d=128, G=4, w0=4096) followed by one bifocal
decode of a Qwen3-4B-like layer against a 131072-token raw KV cache.  Inputs
are synthetic and seeded (paper_2607_07740_amd.synth) and resident in HBM
before timing starts.  Prints ONE JSON line.

  value       prefill TFLOP/s (algorithmic: 4 d B Hq L(L+1)/2 per call)
  roofline    prefill kernel vs dense bf16 MFMA peak (HIP events, launch stream)
  decode_*    decode us per call (split + reduce; calls back to back on the
              stream, two caches alternating) and HBM GB/s vs 8 TB/s
  overhead_*  bifocal / same-build vanilla RoPE attention - 1
  cpu_baseline  the fp64 oracle on a bounded row sample, on the host cores
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "bifocal prefill TFLOP/s & MFMA util at 128K; decode us/token and HBM GB/s at 128K"
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0     # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "prefill_traffic_qwen3_8b_128k.txt")
KERNEL_SOURCES = ["paper_2607_07740_amd/csrc/prefill.hip", "paper_2607_07740_amd/csrc/jl_device.h"]


def _kernel_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def _traffic_from_profile():
    """HBM bytes per prefill launch from the committed rocprofv3 counter summary,
    or None when it is missing or was taken on a different kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.lstrip().startswith("#"):
            key, val = line.split(":", 1)
            vals[key.strip()] = val.strip()
    if vals.get("kernel_source_sha256") != _kernel_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _dev(bits, torch, np):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(q, k, v, w, target_s: float, dec=None):
    """Time the oracle (as it stands) on a seeded sample of prefill rows; also
    its full wall time on the tiny prefill and on the decode workload."""
    import numpy as np
    from oracle import oracle as O
    from paper_2607_07740_amd import synth
    rng = np.random.default_rng(1234)
    g = w.Hq // w.Hkv

    def rows_of(n):
        pos = rng.integers(0, w.L, size=n)
        return np.stack([np.zeros(n, np.int64), rng.integers(0, g, size=n),  # kv head 0's group
                         pos], axis=1).astype(np.int64)

    def run(rows):
        t0 = time.perf_counter()
        _, thr = O.prefill_rows(q, k, v, rows, theta=w.theta, w_pretrained=w.w_pretrained,
                                w_local=w.w_local)
        return time.perf_counter() - t0, thr

    # two probes separate the per-call cost (rotating the kv head's keys) from
    # the per-row cost, so the timed sample lands near target_s
    t_a, _ = run(rows_of(16))
    t_b, _ = run(rows_of(256))
    per_row = max((t_b - t_a) / 240.0, 1e-5)
    fixed = max(t_a - 16 * per_row, 0.0)
    n = int(max(16, min(200000, (target_s - fixed) / per_row)))
    rows = rows_of(n)
    dt, threads = run(rows)
    flops = float(np.sum(4.0 * w.d * (rows[:, 2] + 1)))
    full_s = float(np.sum(4.0 * w.d * w.B * w.Hq * (np.arange(w.L) + 1.0))) / (flops / dt)
    res = {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(threads),
           "kind": "oracle",
           "sample": "%d rows (b=0, heads of kv head 0, uniform positions) of %s, %.1f s wall, "
                     "includes rotating that kv head's keys" % (n, w.name, dt),
           "cpu_model": _cpu_model(),
           "full_prefill_s_extrapolated": round(full_s, 1)}
    tw = synth.WORKLOADS["tiny_prefill"]
    tq, tk, tv = synth.make_inputs(tw)
    t0 = time.perf_counter()
    O.prefill(tq, tk, tv, theta=tw.theta, w_pretrained=tw.w_pretrained, w_local=tw.w_local)
    res["tiny_prefill_s"] = round(time.perf_counter() - t0, 3)
    if dec is not None:
        dq, dk, dv, lens, wd = dec
        t0 = time.perf_counter()
        O.decode(dq, dk, dv, lens, theta=wd.theta, w_pretrained=wd.w_pretrained,
                 w_local=wd.w_local)
        res["decode_ms"] = round((time.perf_counter() - t0) * 1e3, 1)
        res["decode_kv_lens"] = [int(x) for x in lens]
    # the B = 8 ragged decode: inputs drawn on the device and copied to the host
    try:
        import torch
        w8 = synth.WORKLOADS["qwen3_4b_decode_b8_ragged"]
        host = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
        q8, k8, v8, l8 = synth.device_inputs(w8, torch)
        q8, k8, v8 = host(q8), host(k8), host(v8)
        torch.cuda.empty_cache()
        t0 = time.perf_counter()
        O.decode(q8, k8, v8, l8, theta=w8.theta, w_pretrained=w8.w_pretrained,
                 w_local=w8.w_local)
        res["decode_b8_ragged_ms"] = round((time.perf_counter() - t0) * 1e3, 1)
        del q8, k8, v8
    except (ImportError, RuntimeError) as e:  # no device for the inputs
        res["decode_b8_ragged_ms"] = "skipped: %s" % e
    return res


def config_block(wp, wd, dlens, G):
    """The bench line's `config`: the timed prefill and decode workloads, with
    the decode batch's own kv lengths."""
    return {
        "workload": "%s + %s" % (wp.name, wd.name),
        "prefill": {"B": wp.B, "Hq": wp.Hq, "Hkv": wp.Hkv, "L": wp.L, "head_dim": wp.d,
                    "w_pretrained": wp.w_pretrained, "w_local": wp.w_local,
                    "rope_theta": wp.theta, "G": int(G)},
        "decode": {"B": wd.B, "Hq": wd.Hq, "Hkv": wd.Hkv, "kv_lens": [int(x) for x in dlens],
                   "head_dim": wd.d, "w_pretrained": wd.w_pretrained,
                   "w_local": wd.w_local, "rope_theta": wd.theta},
    }


EXTRA_PREFILL = ["qwen3_8b_prefill_64k", "qwen3_1p7b_prefill_128k", "qwen3_1p7b_within_32k"]


def measure_configs(api, synth, torch, np, stream, reps, decode_batch):
    """The workload list's other configurations, each timed bifocal against the
    same-build vanilla kernel (interleaved, medians): the 8B-like layer at 64K
    (G = 2), the 1.7B-like layer at 128K (G = 4), the within-window case
    (G = 1), and B = 8 decode at the ragged boundary lengths and at seeded
    uniform lengths in [32768, 131072].  Inputs are drawn on the device."""
    med = lambda x: sorted(x)[len(x) // 2]

    def timed(fn, n=1):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    res = {}
    for name in EXTRA_PREFILL:
        w = synth.WORKLOADS[name]
        q, k, v = synth.device_inputs(w, torch)
        out = torch.empty_like(q)
        bif = lambda: api.bifocal_prefill(q, k, v, w_pretrained=w.w_pretrained, w_local=w.w_local,
                                          rope_theta=w.theta, out=out, stream=stream)
        van = lambda: api.rope_attention(q, k, v, rope_theta=w.theta, out=out, stream=stream)
        bif()
        van()
        tb, tv = [], []
        for _ in range(reps):
            tv.append(timed(van))
            tb.append(timed(bif))
        flops = 4.0 * w.d * w.B * w.Hq * w.L * (w.L + 1) / 2.0
        res[name] = {"B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "L": w.L,
                     "G": api.group_size(w.L, w.w_pretrained),
                     "bifocal_ms": round(med(tb), 3), "vanilla_ms": round(med(tv), 3),
                     "TFLOPs": round(flops / (med(tb) * 1e-3) / 1e12, 1),
                     "mfma_frac": round(flops / (med(tb) * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                     "overhead_vs_vanilla": round(med(tb) / med(tv) - 1.0, 4)}
        del q, k, v, out
    wd = synth.WORKLOADS["qwen3_4b_decode_b8_ragged"]
    variants = {"qwen3_4b_decode_b8_ragged": list(wd.kv_lens),
                "qwen3_4b_decode_b8_uniform": [int(x) for x in
                                               synth.ragged_lengths(8, 32768, 131072, seed=0)]}
    for name, lens in variants.items():
        q, kc, vc, ln = synth.device_inputs(wd, torch, kv_lens=lens)
        lens_d = torch.from_numpy(ln).cuda()
        out = torch.empty_like(q)
        ws = torch.empty(api.decode_workspace_bytes(wd.B, wd.Hq, wd.Hkv, wd.L), dtype=torch.uint8,
                         device="cuda")
        bif = lambda: api.bifocal_decode(q, kc, vc, lens_d, w_pretrained=wd.w_pretrained,
                                         w_local=wd.w_local, rope_theta=wd.theta, out=out,
                                         workspace=ws, stream=stream)
        van = lambda: api.rope_attention_decode(q, kc, vc, lens_d, rope_theta=wd.theta, out=out,
                                                workspace=ws, stream=stream)
        bif()
        van()
        tb, tv = [], []
        for _ in range(max(reps, 5)):
            tv.append(timed(van, decode_batch))
            tb.append(timed(bif, decode_batch))
        nbytes = 2.0 * float(np.sum(ln)) * wd.Hkv * wd.d * 2.0 + 2.0 * wd.B * wd.Hq * wd.d * 2.0
        gbps = nbytes / (med(tb) * 1e-3) / 1e9
        res[name] = {"B": wd.B, "kv_lens": lens, "bifocal_us": round(med(tb) * 1e3, 1),
                     "vanilla_us": round(med(tv) * 1e3, 1), "GBps": round(gbps, 1),
                     "hbm_frac": round(gbps / PEAK_HBM_GBPS, 4),
                     "overhead_vs_vanilla": round(med(tb) / med(tv) - 1.0, 4)}
        del q, kc, vc, out, ws
    return res


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--prefill", default="qwen3_8b_prefill_128k")
    ap.add_argument("--decode", default="qwen3_4b_decode_128k")
    ap.add_argument("--overhead-reps", type=int, default=3,
                    help="interleaved vanilla/bifocal prefill pairs for the overhead figure")
    ap.add_argument("--decode-reps", type=int, default=20,
                    help="interleaved vanilla/bifocal batches of back-to-back decode calls "
                         "(decode median and overhead)")
    ap.add_argument("--decode-batch", type=int, default=10,
                    help="decode calls per timed batch")
    ap.add_argument("--literal-reps", type=int, default=2,
                    help="timed calls of the literal three-pass prefill (0 skips it)")
    ap.add_argument("--paged-reps", type=int, default=8,
                    help="timed batches of decode calls on a paged copy of the cache (0 skips)")
    ap.add_argument("--sweep-reps", type=int, default=2,
                    help="timed vanilla/bifocal pairs per length of the 8B-like prefill sweep "
                         "4K .. 128K (0 skips)")
    ap.add_argument("--varlen-reps", type=int, default=3,
                    help="timed packed prefills of 131072 tokens in seven sequences (0 skips)")
    ap.add_argument("--freq-reps", type=int, default=1,
                    help="timed calls of the prefill with the frequency-interpolation remote map "
                         "(0 skips it)")
    ap.add_argument("--config-reps", type=int, default=3,
                    help="timed vanilla/bifocal pairs for each of the other workload "
                         "configurations (64K, 1.7B-like 128K, within-window, B=8 decode; 0 skips)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--zero-inputs", action="store_true",
                    help="diagnostic: time the main workloads on all-zero Q, K, V (the matrix "
                         "cores then draw far less power); not a benchmark result")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB three times (the "
                         "reference for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE) and exit")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (each GPU would take "
              "its own kv heads with no exchange); run with --gpus 1", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2607_07740_amd import api, synth

    torch.cuda.set_device(0)
    if args.copy_calibration:
        nbytes = args.copy_calibration << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": nbytes, "reps": 3}), flush=True)
        return 0
    wp = synth.WORKLOADS[args.prefill]
    wd = synth.WORKLOADS[args.decode]
    assert wp.kind == "prefill" and wd.kind == "decode"

    # ---- inputs resident in HBM
    qh, kh, vh = synth.make_inputs(wp)
    q, k, v = _dev(qh, torch, np), _dev(kh, torch, np), _dev(vh, torch, np)
    out = torch.empty_like(q)
    dq, dk, dv, dlens = synth.make_inputs(wd)
    dqd = _dev(dq, torch, np)
    caches = [(_dev(dk, torch, np), _dev(dv, torch, np))]
    # a second cache with the same contents, alternated so consecutive decode
    # calls cannot be served from the 256 MB Infinity Cache
    caches.append((caches[0][0].clone(), caches[0][1].clone()))
    if args.zero_inputs:
        for t in (q, k, v, dqd) + caches[0] + caches[1]:
            t.zero_()
    lens_d = torch.from_numpy(dlens).cuda()
    dout = torch.empty_like(dqd)
    ws = torch.empty(api.decode_workspace_bytes(wd.B, wd.Hq, wd.Hkv, wd.L), dtype=torch.uint8,
                     device="cuda")

    stream = torch.cuda.current_stream()

    def prefill(bifocal=True):
        if bifocal:
            api.bifocal_prefill(q, k, v, w_pretrained=wp.w_pretrained, w_local=wp.w_local,
                                rope_theta=wp.theta, out=out, stream=stream)
        else:
            api.rope_attention(q, k, v, rope_theta=wp.theta, out=out, stream=stream)

    def decode(i, bifocal=True):
        kc, vc = caches[i % 2]
        if bifocal:
            api.bifocal_decode(dqd, kc, vc, lens_d, w_pretrained=wd.w_pretrained,
                               w_local=wd.w_local, rope_theta=wd.theta, out=dout, workspace=ws,
                               stream=stream)
        else:
            api.rope_attention_decode(dqd, kc, vc, lens_d, rope_theta=wd.theta, out=dout,
                                      workspace=ws, stream=stream)

    for i in range(args.warmup):
        prefill()
        decode(i)
    torch.cuda.synchronize()

    # e[0..3]: whole prefill and decode calls; e[4..7]: the attention kernel
    # and the decode split kernel alone, recorded by the library on the same
    # stream right around those launches -- on even steps only: the records
    # inside a call add gaps of their own, so the whole-call decode time after
    # a prefill comes from the odd steps (every step when there is only one)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(8)] for _ in range(args.steps)]
    inner = [i % 2 == 0 for i in range(args.steps)]
    for e in ev:
        for x in e:
            x.record(stream)  # creates the HIP events before they are handed over
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        e = ev[i]
        if inner[i]:
            api.debug_kernel_events(0, e[4], e[5])
            api.debug_kernel_events(1, e[6], e[7])
        else:
            api.debug_kernel_events(0)
            api.debug_kernel_events(1)
        e[0].record(stream)
        prefill()
        e[1].record(stream)
        e[2].record(stream)
        decode(i)
        e[3].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    api.debug_kernel_events(0)
    api.debug_kernel_events(1)

    pre_ms = [e[0].elapsed_time(e[1]) for e in ev]
    plain = [e for e, x in zip(ev, inner) if not x] or ev
    dec_ms = [e[2].elapsed_time(e[3]) for e in plain]
    attn_ms = [e[4].elapsed_time(e[5]) for e, x in zip(ev, inner) if x]
    split_ms = [e[6].elapsed_time(e[7]) for e, x in zip(ev, inner) if x]
    pre_avg = sum(pre_ms) / len(pre_ms)
    dec_avg = sum(dec_ms) / len(dec_ms)
    attn_avg = sum(attn_ms) / len(attn_ms)
    split_avg = sum(split_ms) / len(split_ms)

    flops = 4.0 * wp.d * wp.B * wp.Hq * wp.L * (wp.L + 1) / 2.0
    tflops = flops / (pre_avg * 1e-3) / 1e12
    attn_tflops = flops / (attn_avg * 1e-3) / 1e12
    kv_bytes = 2.0 * float(np.sum(dlens)) * wd.Hkv * wd.d * 2.0
    io_bytes = 2.0 * wd.B * wd.Hq * wd.d * 2.0
    dec_gbps = (kv_bytes + io_bytes) / (dec_avg * 1e-3) / 1e9

    # ---- overhead against the same-build vanilla kernel, interleaved
    def timed(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b)

    pb, pv, db_, dv_ = [], [], [], []
    for r in range(args.overhead_reps):
        pv.append(timed(lambda: prefill(False)))
        pb.append(timed(lambda: prefill(True)))

    # decode per call as a model issues it: one layer's call after another on
    # the stream with no host synchronisation in between (alternating the two
    # caches, so no call finds the previous one's K/V in the Infinity Cache);
    # batches of vanilla and bifocal calls interleave.  A third batch per
    # repetition, not part of the call timings, times the split kernel of its
    # middle call with events the library records on the stream right around it
    sev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.decode_reps)]
    for x, y in sev:
        x.record(stream)
        y.record(stream)

    def decode_batch(bifocal, evs=None):
        for i in range(args.decode_batch):
            mid = evs is not None and i == args.decode_batch // 2
            if mid:
                api.debug_kernel_events(1, evs[0], evs[1])
            decode(i, bifocal)
            if mid:
                api.debug_kernel_events(1)

    torch.cuda.synchronize()
    for r in range(args.decode_reps):
        dv_.append(timed(lambda: decode_batch(False)) / args.decode_batch)
        db_.append(timed(lambda: decode_batch(True)) / args.decode_batch)
        decode_batch(True, sev[r])  # the split kernel timed alone, outside the call timings
    torch.cuda.synchronize()
    med = lambda x: sorted(x)[len(x) // 2] if x else float("nan")
    dec_med = med(db_)
    dec_gbps = (kv_bytes + io_bytes) / (dec_med * 1e-3) / 1e9
    split_steady = med([x.elapsed_time(y) for x, y in sev])
    split_gbps = kv_bytes / (split_steady * 1e-3) / 1e9

    # ---- Eq. (7) taken literally: three window passes plus the merge
    lit = {}
    if args.literal_reps > 0:
        lws = torch.empty(api.prefill_literal_workspace_bytes(wp.B, wp.Hq, wp.Hkv, wp.L),
                          dtype=torch.uint8, device="cuda")

        def literal():
            api.bifocal_prefill_literal(q, k, v, w_pretrained=wp.w_pretrained,
                                        w_local=wp.w_local, rope_theta=wp.theta, out=out,
                                        workspace=lws, stream=stream)
        literal()
        lt = [timed(literal) for _ in range(args.literal_reps)]
        del lws
        lit = {"literal_prefill_ms": round(med(lt), 3),
               "literal_throughput_vs_vanilla": round(med(pv) / med(lt), 4),
               "fused_speedup_vs_literal": round(med(lt) / med(pb), 4)}

    # ---- the same decode on a paged cache: 256-key pages in shuffled order
    pg = {}
    if args.paged_reps > 0:
        page = 256
        n_pg = (wd.L + page - 1) // page
        perm = torch.randperm(wd.B * n_pg, generator=torch.Generator().manual_seed(0))
        kc0, vc0 = caches[0]
        kpool = torch.empty((wd.B * n_pg, page, wd.Hkv, wd.d), dtype=torch.bfloat16, device="cuda")
        vpool = torch.empty_like(kpool)
        kpool[perm] = kc0[:, :n_pg * page].reshape(wd.B * n_pg, page, wd.Hkv, wd.d)
        vpool[perm] = vc0[:, :n_pg * page].reshape(wd.B * n_pg, page, wd.Hkv, wd.d)
        table = perm.to(torch.int32).reshape(wd.B, n_pg).cuda()
        # two pools alternate, as the two dense caches do, so no call is served
        # from the Infinity Cache
        pools = [(kpool, vpool), (kpool.clone(), vpool.clone())]

        def paged_batch():
            for i in range(args.decode_batch):
                kp, vp = pools[i % 2]
                api.decode_paged(dqd, kp, vp, table, lens_d, w_pretrained=wd.w_pretrained,
                                 w_local=wd.w_local, rope_theta=wd.theta, out=dout, workspace=ws,
                                 stream=stream)
        paged_batch()
        # interleaved with dense batches, so the ratio compares like with like
        pt, pd = [], []
        for _ in range(args.paged_reps):
            pt.append(timed(paged_batch) / args.decode_batch)
            pd.append(timed(lambda: decode_batch(True)) / args.decode_batch)
        pg = {"decode_paged_us": round(med(pt) * 1e3, 2),
              "decode_paged_vs_dense": round(med(pt) / med(pd), 4)}
        del kpool, vpool, pools

    # ---- the Sec. 4.5 ablation's remote view: frequency interpolation
    fm = {}
    if args.freq_reps > 0:
        def freq_map():
            api.bifocal_prefill(q, k, v, w_pretrained=wp.w_pretrained, w_local=wp.w_local,
                                rope_theta=wp.theta, out=out, stream=stream, remote_map="freq")
        freq_map()
        ft = [timed(freq_map) for _ in range(args.freq_reps)]
        fm = {"freq_map_prefill_ms": round(med(ft), 3)}
        # decode with the frequency map: the kernel forms its rows from the
        # device lengths, interleaved with the Eq. (3) decode
        fws = torch.empty(api.decode_map_workspace_bytes(wd.B, wd.Hq, wd.Hkv, wd.L, wd.d, "freq"),
                          dtype=torch.uint8, device="cuda")

        def freq_decode_batch():
            for i in range(args.decode_batch):
                kc, vc = caches[i % 2]
                api.bifocal_decode(dqd, kc, vc, lens_d, w_pretrained=wd.w_pretrained,
                                   w_local=wd.w_local, rope_theta=wd.theta, out=dout,
                                   workspace=fws, stream=stream, remote_map="freq")
        freq_decode_batch()
        fdt, adt = [], []
        for _ in range(max(3, args.decode_reps // 4)):
            fdt.append(timed(freq_decode_batch) / args.decode_batch)
            adt.append(timed(lambda: decode_batch(True)) / args.decode_batch)
        fm["freq_map_decode_us"] = round(med(fdt) * 1e3, 2)
        fm["freq_map_decode_vs_alias"] = round(med(fdt) / med(adt), 4)
        del fws

    # ---- packed variable-length prefill: the prefill layer's 131072 tokens as
    # seven sequences of 64K .. 1K in one call, against one call per sequence
    vl = {}
    if args.varlen_reps > 0:
        vlens = [65536, 32768, 16384, 8192, 4096, 3072, 1024]
        cu = torch.tensor([0] + list(np.cumsum(vlens)), dtype=torch.int32, device="cuda")
        qv, kv_, vv = q[0], k[0], v[0]  # [T, H, 128] views of the resident inputs
        ov = out[0]

        def varlen():
            api.prefill_varlen(qv, kv_, vv, cu, max_seqlen=max(vlens), w_pretrained=wp.w_pretrained,
                               w_local=wp.w_local, rope_theta=wp.theta, out=ov, stream=stream)
        parts = []
        for a, b in zip(cu[:-1].tolist(), cu[1:].tolist()):
            parts.append((q[:, a:b].contiguous(), k[:, a:b].contiguous(), v[:, a:b].contiguous()))

        def separate():
            for qs, ks, vs in parts:
                api.bifocal_prefill(qs, ks, vs, w_pretrained=wp.w_pretrained, w_local=wp.w_local,
                                    rope_theta=wp.theta, stream=stream)
        varlen()
        separate()
        tv_, ts_ = [], []
        for _ in range(args.varlen_reps):
            tv_.append(timed(varlen))
            ts_.append(timed(separate))
        vfl = sum(4.0 * wp.d * wp.Hq * n * (n + 1) / 2.0 for n in vlens)
        vl = {"varlen_prefill": {"lens": vlens, "ms": round(med(tv_), 3),
                                 "TFLOPs": round(vfl / (med(tv_) * 1e-3) / 1e12, 1),
                                 "mfma_frac": round(vfl / (med(tv_) * 1e-3) / 1e12 /
                                                    PEAK_BF16_TFLOPS, 4),
                                 "separate_calls_ms": round(med(ts_), 3)}}
        del parts

    # ---- decode served warm: the same cache call after call (the Infinity
    # Cache then holds part of K/V); the primary decode figure above is cold
    warm = [timed(lambda: [decode(0) for _ in range(args.decode_batch)]) / args.decode_batch
            for _ in range(max(1, args.decode_reps // 4))]

    # ---- the paper's length sweep (Tab. 7 lengths) on the 8B-like layer: the
    # G = 1 plateau below the window, then G = 2, 3, 4
    sweep = []
    if args.sweep_reps > 0:
        for Lx in (4096, 8192, 16384, 32768, 65536, 98304, 131072):
            qx, kx, vx = q[:, :Lx], k[:, :Lx].contiguous(), v[:, :Lx].contiguous()
            qx = qx.contiguous()
            ox = torch.empty_like(qx)
            fb = lambda: api.bifocal_prefill(qx, kx, vx, w_pretrained=wp.w_pretrained,
                                             w_local=wp.w_local, rope_theta=wp.theta, out=ox,
                                             stream=stream)
            fv = lambda: api.rope_attention(qx, kx, vx, rope_theta=wp.theta, out=ox,
                                            stream=stream)
            fb()
            fv()
            tb, tv = [], []
            for _ in range(args.sweep_reps):
                tv.append(timed(fv))
                tb.append(timed(fb))
            fl = 4.0 * wp.d * wp.B * wp.Hq * Lx * (Lx + 1) / 2.0
            sweep.append({"L": Lx, "G": api.group_size(Lx, wp.w_pretrained),
                          "bifocal_ms": round(med(tb), 3), "vanilla_ms": round(med(tv), 3),
                          "TFLOPs": round(fl / (med(tb) * 1e-3) / 1e12, 1),
                          "bifocal_vs_vanilla_throughput": round(med(tv) / med(tb), 4)})
            del qx, kx, vx, ox

    cfg = {}
    if args.config_reps > 0:
        cfg = measure_configs(api, synth, torch, np, stream, args.config_reps, args.decode_batch)

    traffic = _traffic_from_profile()
    line = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "zeros (diagnostic)" if args.zero_inputs else "synthetic",
        "config": config_block(wp, wd, dlens, api.group_size(wp.L, wp.w_pretrained)),
        "prefill_ms": round(pre_avg, 3),
        "prefill_mfma_frac": round(tflops / PEAK_BF16_TFLOPS, 4),
        "decode_us": round(dec_med * 1e3, 2),
        "decode_us_after_prefill": round(med(dec_ms) * 1e3, 2),
        "decode_GBps": round(dec_gbps, 1),
        "decode_hbm_frac": round(dec_gbps / PEAK_HBM_GBPS, 4),
        "overhead_prefill_vs_vanilla": round(med(pb) / med(pv) - 1.0, 4),
        "overhead_decode_vs_vanilla": round(med(db_) / med(dv_) - 1.0, 4),
        "vanilla_prefill_ms": round(med(pv), 3),
        "vanilla_decode_us": round(med(dv_) * 1e3, 2),
        "decode_warm_us": round(med(warm) * 1e3, 2),
        **lit,
        **fm,
        **pg,
        **vl,
        "roofline": {
            "bound": "mfma",
            "kernel": "prefill_kernel<fused>",
            "achieved": round(attn_tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "kernel_ms": round(attn_avg, 3),
        },
        "decode_roofline": {
            "bound": "hbm", "kernel": "decode_split_kernel<bifocal>",
            "achieved": round(split_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
            "frac": round(split_gbps / PEAK_HBM_GBPS, 4), "kernel_us": round(split_steady * 1e3, 2),
            "kernel_us_after_prefill": round(split_avg * 1e3, 2),
        },
    }
    if cfg:
        line["configs"] = cfg
    if sweep:
        line["length_sweep"] = sweep
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(qh, kh, vh, wp, args.cpu_seconds,
                                            (dq, dk, dv, dlens, wd))
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
