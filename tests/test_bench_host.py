"""bench.py's host-side contract (CPU): one GPU only, one JSON line."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_traffic_figures_belong_to_the_profiled_workload():
    sys.path.insert(0, ROOT)
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    with open(b.TRAFFIC_FILE) as f:
        t = json.load(f)
    # HBM bytes from the counters cover at least the algorithmic bytes, and
    # never apply to another workload
    assert t["bytes_per_launch"] >= t["algorithmic_bytes_per_launch"]
    assert b.measured_traffic("qwen3-32b-decode") is None


def _bench_module():
    sys.path.insert(0, ROOT)
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    return b


def test_attention_flops_count_every_visible_position():
    from paper_2607_03333_amd import synth
    b = _bench_module()
    for wl in (synth.make(synth.config_index("tiny-fork-f32")),
               synth.make(synth.config_index("qwen3-32b-verify"), sessions=2, prefix=40, vocab=256)):
        for i, st in enumerate(wl.steps):
            # brute force: row j of a thread with n positions and r rows sees
            # the positions 0 .. n - r + j
            visible = 0
            for seq, r in zip(st.seqs, st.n_rows):
                n = wl.thread_len(seq, i)
                for j in range(r):
                    visible += sum(1 for p in range(n) if p <= n - r + j)
            assert b.attention_flops(wl, i, st) == visible * wl.hq * 4 * wl.d
            assert visible > 0


def test_mfma_ridge_points():
    b = _bench_module()
    # bf16: 2.5 PFLOP/s over 8 TB/s; fp32 MFMA: 157.3 TFLOP/s over 8 TB/s
    assert abs(b.MFMA_PEAK_TFLOPS["bf16"] * 1e12 / (b.HBM_PEAK_GBPS * 1e9) - 312.5) < 1e-9
    assert abs(b.MFMA_PEAK_TFLOPS["f32"] * 1e12 / (b.HBM_PEAK_GBPS * 1e9) - 19.6625) < 1e-9


def test_kernel_hash_follows_the_code_not_its_comments(tmp_path):
    # the counters in profiles/ stay matched across comment and layout edits
    # of the kernel sources and stop matching once a line of code changes
    b = _bench_module()
    srcs = []
    for i, path in enumerate(b.KERNEL_SOURCES):
        with open(path) as f:
            text = f.read()
        p = tmp_path / f"src{i}"
        p.write_text(text)
        srcs.append((p, text))
    b.KERNEL_SOURCES = [str(p) for p, _ in srcs]
    h0 = b.kernel_source_hash()
    p0, t0 = srcs[0]
    p0.write_text("// a note\n" + t0.replace("\n", "\n  ", 3) + "\n/* another\n note */\n")
    assert b.kernel_source_hash() == h0
    p0.write_text(t0 + "\nconstexpr int kNotInTheKernel = 1;\n")
    assert b.kernel_source_hash() != h0
