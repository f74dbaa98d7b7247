"""bench.py's command-line contract that holds without a GPU."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "single MI355X" in r.stderr and "--gpus 2" in r.stderr
    assert r.stdout.strip() == ""  # no JSON line for a run that did not happen


def test_bench_lists_its_workloads():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--help"], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0
    for wl in ("layer", "ln_qkv", "causal_softmax_pv", "ffn_decode_t1", "causal_attention", "decode_attention"):
        assert wl in r.stdout


def test_bench_weight_copies_cover_the_last_level_cache():
    # HBM-bound LN shapes rotate through about 1 GB of prepared weights (four times the
    # 256 MB last-level cache); MFMA-bound shapes use one copy
    sys.path.insert(0, ROOT)
    import bench
    from paper_2502_17728_amd import inputs as I
    assert bench.weight_copies(I.ln_ffn_decode(1)) == 3      # 470 MB of W'
    assert bench.weight_copies(I.ln_ffn_decode(16)) == 3
    assert bench.weight_copies(I.ln_qkv_tokens(32)) == 10    # 100.7 MB of W'
    assert bench.weight_copies(I.LN_QKV) == 1
    assert bench.weight_copies(I.LN_FFN_PREFILL) == 1
    assert bench.weight_copies(I.LN_F32_SMALL) == 1          # above the fp32 ridge point


def test_bench_paths_and_traffic_table():
    # the timed step can run the deferred kernels, the unfused comparators or (for profiling)
    # the vendor library's plain product; every stored traffic figure names the sources it
    # was counted on, and a figure taken on other sources reads as unknown
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--help"], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0 and "library" in r.stdout and "unfused" in r.stdout
    sys.path.insert(0, ROOT)
    import bench
    for (kernel, workload), t in bench.TRAFFIC.items():
        assert kernel in bench.KERNEL_SOURCES
        assert len(t["sha256"]) == len(bench.KERNEL_SOURCES[kernel])
        assert t["fetch_kib"] > 0 and 1.9 < t["fetch_scale"] < 2.1 and t["write_scale"] == 1.0
    saved = dict(bench.TRAFFIC)
    try:
        key = next(iter(bench.TRAFFIC))
        bench.TRAFFIC[key] = dict(bench.TRAFFIC[key], sha256=("0" * 64,) * len(bench.TRAFFIC[key]["sha256"]))
        assert bench.measured_traffic(*key) is None
    finally:
        bench.TRAFFIC.clear()
        bench.TRAFFIC.update(saved)
