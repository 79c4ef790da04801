"""Host-side checks of bench.py's reported configuration (no GPU)."""
import importlib.util
import os

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_config_block_reports_the_decode_workloads_own_lengths():
    from paper_2607_07740_amd import synth
    bench = _bench()
    wp = synth.WORKLOADS["qwen3_8b_prefill_128k"]
    wd = synth.WORKLOADS["qwen3_4b_decode_128k"]
    dlens = np.asarray(wd.kv_lens, dtype=np.int32)
    cfg = bench.config_block(wp, wd, dlens, 4)
    assert cfg["decode"]["kv_lens"] == [131072]
    assert cfg["decode"]["B"] == 1 and cfg["decode"]["Hq"] == 32 and cfg["decode"]["Hkv"] == 8
    assert cfg["prefill"]["L"] == 131072 and cfg["prefill"]["G"] == 4
    assert cfg["workload"] == "qwen3_8b_prefill_128k + qwen3_4b_decode_128k"


def test_bench_main_keeps_decode_and_varlen_lengths_apart():
    # the varlen leg's sequence list must not rebind the decode workload's
    # lengths, which the config block and the oracle's decode timing use
    src = open(os.path.join(ROOT, "bench.py")).read()
    main = src[src.index("def main()"):]
    assert "dq, dk, dv, dlens = synth.make_inputs(wd)" in main
    assert "config_block(wp, wd, dlens," in main
    assert "(dq, dk, dv, dlens, wd)" in main
    assert "\n        lens = " not in main and "\n    lens = " not in main


def test_traffic_is_reported_only_for_the_profiled_kernel_source(tmp_path, monkeypatch):
    """bench.py reads the HBM traffic from the committed counter summary only
    while that summary's source hash matches the kernel sources it runs."""
    bench = _bench()
    good = tmp_path / "good.txt"
    good.write_text("# comment: ignored\nkernel_source_sha256: %s\nhbm_bytes_per_launch: 1.5e+10\n"
                    % bench._kernel_hash())
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(good))
    assert bench._traffic_from_profile() == 1.5e10
    stale = tmp_path / "stale.txt"
    stale.write_text("kernel_source_sha256: %s\nhbm_bytes_per_launch: 1.5e+10\n" % ("0" * 64))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(stale))
    assert bench._traffic_from_profile() is None
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "missing.txt"))
    assert bench._traffic_from_profile() is None


def test_more_than_one_gpu_is_refused():
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0
    assert "--gpus 1" in r.stderr
